"""Parity of the bf16 storage mode (PMLP_BF16_STORE: the bf16 operand mode
with the hidden pre-activation Z also kept in bfloat16 between the kernels)
with the oracle's `rounding="bf16_store"`.

A stored Z has two correct values where the fp32 accumulator lies within
rounding of a bfloat16 midpoint, and such pairs are common (half an ulp of
bfloat16 is 2^-9 relative), so the one-step comparisons hand the GPU's
stored Z (read back with pmlp_hidden on the same weights and batch) to the
oracle, which takes it only where it is one of the two correct values and
counts every other difference as a conflict; the tests assert none.  "Within
rounding" is the bound of an fp32 sum of K products in any order, gamma_K =
K u / (1 - K u) of the sum of their magnitudes (u = 2^-24, K = F + 1
counting a bias), since the matrix cores fix no summation order.  With
that, the bar is the fp32 path's: per-model normwise 1e-5 for one step
(dW1 after the kink and dZ rounding-tie allowances, dW2 relative to the size
of its terms).  Over an epoch the two sides take different sides of some
ties at every step, so the losses are held to 1e-3 of the oracle's storage
mode and 2e-2 of the exact oracle (the bf16 operand mode's bars), the
weights to 2e-2.
"""
import zlib

import numpy as np
import pytest

import pmlp_workloads as wl
from parity import (cross_entropy, dw2_terms, err_cols, err_dw2, err_logits, err_losses,
                    err_rows)

pytestmark = pytest.mark.gpu

TOL_STEP = 1e-5
TOL_EPOCH = 1e-3
TOL_VS_EXACT = 2e-2
MODE = "bf16_store"


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    torch.cuda.set_device(0)
    return torch


@pytest.fixture(scope="module")
def pm(torch):
    import paper_2206_08369_amd as pm
    pm.load_library()
    return pm


def dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def store_net(pm, F, O, hs, acts, seed=0):
    return pm.PackedMLP(F, O, hs, acts, seed=seed, precision=pm.PMLP_BF16_STORE)


# shapes of the bf16 product's tiling (ragged p tiles, q <= 64 and > 64,
# k tails) and of both M3 forwards (O <= 4 and the matrix-core one) and the
# M3 backward, with one- to 1100-sample batches
CASES = {
    "tiny_b1": dict(hs=[1, 2, 3, 1], F=3, O=2, B=1),
    "ragged": dict(M=37, hmax=40, F=13, O=3, B=7),
    "tile_spanning": dict(hs=[1300, 513, 512, 1, 700, 3, 1024], F=10, O=2, B=33),
    "f100_b250": dict(M=30, hmax=300, F=100, O=2, B=250),
    "f1000_b300": dict(M=6, hmax=80, F=1000, O=2, B=300),
    "f64_b64_o10": dict(M=25, hmax=200, F=64, O=10, B=64),
    "o16_b16": dict(M=10, hmax=20, F=37, O=16, B=16),
    "o8_b32": dict(M=12, hmax=30, F=20, O=8, B=29),
    "b1100": dict(M=6, hmax=20, F=20, O=2, B=1100),
}


def case_inputs(name, seed=0):
    c = CASES[name]
    rng = np.random.default_rng(zlib.crc32(name.encode()) + seed)
    if "hs" in c:
        hs = np.asarray(c["hs"], np.int32)
        acts = rng.integers(0, 13, len(hs)).astype(np.int32)
    else:
        hs, acts = wl.random_models(rng, c["M"], c["hmax"])
    X, y = wl.make_dataset(c["F"], c["O"], c["B"], seed=int(rng.integers(1 << 30)))
    return hs, acts, c["F"], c["O"], c["B"], X, y


def zband(F):
    """The tie band of a stored Z: gamma_K for K = F + 1 terms."""
    k = (F + 1) * 2.0 ** -24
    return k / (1.0 - k)


def stored_z(net, torch, Xd):
    """The GPU's stored Z [B, N] (fp32 copies of bfloat16 values)."""
    Z, _ = net.hidden(Xd)
    z = Z.cpu().numpy()
    assert not np.any(z.view(np.uint32) & 0xFFFF), "stored Z must be bfloat16 values"
    return z


@pytest.mark.parametrize("name", sorted(CASES))
def test_store_hidden_layer(pm, orc, torch, name):
    hs, acts, F, O, B, X, y = case_inputs(name)
    net = store_net(pm, F, O, hs, acts, seed=31)
    W1, _ = net.get_params()
    Z, H = net.hidden(dev(torch, X))
    Z, H = Z.cpu().numpy(), H.cpu().numpy()
    RZ, RH = orc.hidden(hs, acts, W1, X, rounding=MODE, stored_z=Z, zband=zband(F))
    assert orc.stored_z_conflicts() == 0
    assert np.array_equal(Z, RZ.astype(np.float32))
    assert err_cols(H, RH, hs).max() <= TOL_STEP
    # the stored values are the operand mode's Z rounded (to within ties)
    RZb, _ = orc.hidden(hs, acts, W1, X, rounding="bf16")
    assert err_cols(Z, RZb, hs).max() <= 2.0 ** -8
    net.close()


@pytest.mark.parametrize("name", sorted(CASES))
def test_store_forward_logits(pm, orc, torch, name):
    hs, acts, F, O, B, X, y = case_inputs(name)
    net = store_net(pm, F, O, hs, acts, seed=32)
    W1, W2 = net.get_params()
    Xd = dev(torch, X)
    zs = stored_z(net, torch, Xd)
    got = net.forward(Xd).cpu().numpy()
    want = orc.forward(hs, acts, W1, W2, X, rounding=MODE, stored_z=zs, zband=zband(F))
    assert orc.stored_z_conflicts() == 0
    assert err_logits(got, want).max() <= TOL_STEP
    net.close()


@pytest.mark.parametrize("name", sorted(CASES))
def test_store_gradients_and_losses(pm, orc, torch, name):
    hs, acts, F, O, B, X, y = case_inputs(name)
    net = store_net(pm, F, O, hs, acts, seed=33)
    W1, W2 = net.get_params()
    Xd, yd = dev(torch, X), dev(torch, y)
    zs = stored_z(net, torch, Xd)
    dW1, dW2 = net.gradients(Xd, yd)
    loss = net.losses()
    r1, r2, rl, allow = orc.gradients(hs, acts, W1, W2, X, y, rounding=MODE, stored_z=zs, zband=zband(F))
    assert orc.stored_z_conflicts() == 0
    assert err_rows(dW1.cpu().numpy(), r1, hs, allow).max() <= TOL_STEP
    terms = dw2_terms(orc, hs, acts, W1, W2, X, y, rounding=MODE, stored_z=zs, zband=zband(F))
    assert err_dw2(dW2.cpu().numpy(), r2, hs, terms).max() <= TOL_STEP
    assert err_losses(loss, rl).max() <= TOL_STEP
    net.close()


@pytest.mark.parametrize("name", ["ragged", "f100_b250", "f1000_b300", "f64_b64_o10"])
def test_store_train_step_is_sgd_on_the_same_gradients(pm, orc, torch, name):
    hs, acts, F, O, B, X, y = case_inputs(name)
    lr = 0.05
    net = store_net(pm, F, O, hs, acts, seed=34)
    W1, W2 = net.get_params()
    Xd, yd = dev(torch, X), dev(torch, y)
    zs = stored_z(net, torch, Xd)
    dW1, dW2 = [t.cpu().numpy() for t in net.gradients(Xd, yd)]
    net.train_step(Xd, yd, lr)
    loss = net.losses()
    T1, T2 = net.get_params()
    assert np.all(np.abs(T1 - (W1 - lr * dW1)) <= 2 * np.spacing(np.maximum(np.abs(W1), np.abs(T1))))
    assert np.all(np.abs(T2 - (W2 - lr * dW2)) <= 2 * np.spacing(np.maximum(np.abs(W2), np.abs(T2))))
    O1, O2, ol = orc.train(hs, acts, W1, W2, X, y, [(0, B)], lr, rounding=MODE, stored_z=zs, zband=zband(F))
    allow = orc.gradients(hs, acts, W1, W2, X, y, rounding=MODE, stored_z=zs, zband=zband(F))[3]
    assert orc.stored_z_conflicts() == 0
    assert err_losses(loss, ol).max() <= TOL_STEP
    assert err_rows(T1, O1, hs, lr * allow).max() <= TOL_STEP
    assert err_cols(T2, O2, hs).max() <= TOL_STEP
    net.close()


def test_modes_share_a_handle(pm, orc, torch):
    """Switching between the three modes on one handle: each step computes
    in the mode set for it (the stored Z of one mode is never read by the
    next), and the operand mode's Z is not rounded."""
    hs, acts, F, O, B, X, y = case_inputs("ragged")
    net = pm.PackedMLP(F, O, hs, acts, seed=35)
    W1, W2 = net.get_params()
    Xd = dev(torch, X)
    for mode, rounding in ((pm.PMLP_BF16_STORE, MODE), (pm.PMLP_BF16_GEMM, "bf16"),
                           (pm.PMLP_FP32, "exact"), (pm.PMLP_BF16_STORE, MODE)):
        net.set_precision(mode)
        Z, _ = net.hidden(Xd)
        z = Z.cpu().numpy()
        got = net.forward(Xd).cpu().numpy()
        kw = dict(stored_z=z, zband=zband(F)) if rounding == MODE else {}
        want = orc.forward(hs, acts, W1, W2, X, rounding=rounding, **kw)
        assert err_logits(got, want).max() <= TOL_STEP
        if rounding == "bf16":
            assert np.any(z.view(np.uint32) & 0xFFFF)
    net.close()


@pytest.mark.parametrize("wname", ["w60_f10", "w1k_f50"])
def test_store_one_epoch(pm, orc, torch, wname):
    w = wl.WORKLOADS[wname]
    hs, acts = w.model_grid()
    X, y = wl.workload_dataset(w)
    net = store_net(pm, w.F, w.O, hs, acts, seed=w.init_seed)
    W1, W2 = net.get_params()
    Xd, yd = dev(torch, X), dev(torch, y)
    batches = w.batches()
    for s, n in batches:
        net.train_step(Xd[s:s + n], yd[s:s + n], w.lr)
    last = net.losses()
    T1, T2 = net.get_params()
    logits = np.concatenate([net.forward(Xd[s:s + 1024]).cpu().numpy()
                             for s in range(0, w.S, 1024)])
    got = cross_entropy(logits, y)
    R1, R2, rl = orc.train(hs, acts, W1, W2, X, y, batches, w.lr, rounding=MODE)
    assert err_losses(last, rl).max() <= TOL_EPOCH
    assert err_losses(got, orc.dataset_loss(hs, acts, R1, R2, X, y, rounding=MODE)).max() \
        <= TOL_EPOCH
    assert err_rows(T1, R1, hs).max() <= TOL_VS_EXACT
    assert err_cols(T2, R2, hs).max() <= TOL_VS_EXACT
    E1, E2, el = orc.train(hs, acts, W1, W2, X, y, batches, w.lr)
    assert err_losses(last, el).max() <= TOL_VS_EXACT
    assert err_losses(got, orc.dataset_loss(hs, acts, E1, E2, X, y)).max() <= TOL_VS_EXACT
    net.close()
