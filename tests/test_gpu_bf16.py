"""Parity of the bf16-in / fp32-accumulate mode (PMLP_BF16_GEMM) with the
oracle.

Against the oracle's bf16 operand mode (X, W1 and dZ rounded to bfloat16
before the two input-layer products, everything else fp64) the bar is the
fp32 path's: per-model normwise 1e-5 for one step (dW1 after the kink and
rounding-tie allowances), 1e-3 for losses after one epoch.  Against the
exact fp64 oracle, per-model losses after one epoch stay within 2e-2.
Shapes span the bf16 GEMM's tiling: p tiles of 128 or 256 rows with ragged
ends, q tiles of 64 or 128, k stages of 32 with tails of 4 to 28, and the
small-q instance (q <= 64).
"""
import zlib

import numpy as np
import pytest

import pmlp_workloads as wl
from parity import offsets, cross_entropy, err_cols, err_logits, err_losses, err_rows, submodel

pytestmark = pytest.mark.gpu

TOL_STEP = 1e-5
TOL_EPOCH = 1e-3
TOL_EPOCH_VS_EXACT = 2e-2


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


def bf16_net(pm, F, O, hs, acts, seed=0):
    return pm.PackedMLP(F, O, hs, acts, seed=seed, precision=pm.PMLP_BF16_GEMM)


CASES = {
    "tiny_b1": dict(hs=[1, 2, 3, 1], F=3, O=2, B=1),            # K = 4: one masked stage
    "ragged": dict(M=37, hmax=40, F=13, O=3, B=7),
    "tile_spanning": dict(hs=[1300, 513, 512, 1, 700, 3, 1024], F=10, O=2, B=33),
    "f100_b250": dict(M=30, hmax=300, F=100, O=2, B=250),         # K1: 3 stages + tail 4
    "f1000_b300": dict(M=6, hmax=80, F=1000, O=2, B=300),         # K6: K = 304, tail 16
    "f64_b64_o10": dict(M=25, hmax=200, F=64, O=10, B=64),        # both GEMMs q <= 64
    "b1100": dict(M=6, hmax=20, F=20, O=2, B=1100),
    "o16_f37": dict(M=10, hmax=20, F=37, O=16, B=48),
}


def case_inputs(name, seed=0):
    c = CASES[name]
    rng = np.random.default_rng(zlib.crc32(name.encode()) + seed)
    if "hs" in c:
        hs = np.asarray(c["hs"], np.int32)
        acts = rng.integers(0, 10, len(hs)).astype(np.int32)
    else:
        hs, acts = wl.random_models(rng, c["M"], c["hmax"])
    X, y = wl.make_dataset(c["F"], c["O"], c["B"], seed=int(rng.integers(1 << 30)))
    return hs, acts, c["F"], c["O"], c["B"], X, y


@pytest.mark.parametrize("name", sorted(CASES))
def test_bf16_hidden_layer(pm, orc, torch, name):
    hs, acts, F, O, B, X, y = case_inputs(name)
    net = bf16_net(pm, F, O, hs, acts, seed=21)
    W1, _ = net.get_params()
    Z, H = net.hidden(dev(torch, X))
    RZ, RH = orc.hidden(hs, acts, W1, X, rounding="bf16")
    assert err_cols(Z.cpu().numpy(), RZ, hs).max() <= TOL_STEP
    assert err_cols(H.cpu().numpy(), RH, hs).max() <= TOL_STEP
    net.close()


@pytest.mark.parametrize("name", sorted(CASES))
def test_bf16_forward_logits(pm, orc, torch, name):
    hs, acts, F, O, B, X, y = case_inputs(name)
    net = bf16_net(pm, F, O, hs, acts, seed=22)
    W1, W2 = net.get_params()
    got = net.forward(dev(torch, X)).cpu().numpy()
    want = orc.forward(hs, acts, W1, W2, X, rounding="bf16")
    assert err_logits(got, want).max() <= TOL_STEP
    net.close()


@pytest.mark.parametrize("name", sorted(CASES))
def test_bf16_gradients_and_losses(pm, orc, torch, name):
    hs, acts, F, O, B, X, y = case_inputs(name)
    net = bf16_net(pm, F, O, hs, acts, seed=23)
    W1, W2 = net.get_params()
    dW1, dW2 = net.gradients(dev(torch, X), dev(torch, y))
    loss = net.losses()
    r1, r2, rl, allow = orc.gradients(hs, acts, W1, W2, X, y, rounding="bf16")
    assert err_rows(dW1.cpu().numpy(), r1, hs, allow).max() <= TOL_STEP
    assert err_cols(dW2.cpu().numpy(), r2, hs).max() <= TOL_STEP
    assert err_losses(loss, rl).max() <= TOL_STEP
    net.close()


@pytest.mark.parametrize("name", ["ragged", "f100_b250", "f1000_b300", "f64_b64_o10"])
def test_bf16_train_step_is_sgd_on_the_same_gradients(pm, orc, torch, name):
    hs, acts, F, O, B, X, y = case_inputs(name)
    lr = 0.05
    net = bf16_net(pm, F, O, hs, acts, seed=24)
    W1, W2 = net.get_params()
    Xd, yd = dev(torch, X), dev(torch, y)
    dW1, dW2 = [t.cpu().numpy() for t in net.gradients(Xd, yd)]
    net.train_step(Xd, yd, lr)
    loss = net.losses()
    T1, T2 = net.get_params()
    ulp1 = np.spacing(np.maximum(np.abs(W1), np.abs(T1))) * 2
    ulp2 = np.spacing(np.maximum(np.abs(W2), np.abs(T2))) * 2
    assert np.all(np.abs(T1 - (W1 - lr * dW1)) <= ulp1)
    assert np.all(np.abs(T2 - (W2 - lr * dW2)) <= ulp2)
    O1, O2, ol = orc.train(hs, acts, W1, W2, X, y, [(0, B)], lr, rounding="bf16")
    allow = orc.gradients(hs, acts, W1, W2, X, y, rounding="bf16")[3]
    assert err_losses(loss, ol).max() <= TOL_STEP
    assert err_rows(T1, O1, hs, lr * allow).max() <= TOL_STEP
    assert err_cols(T2, O2, hs).max() <= TOL_STEP
    net.close()


def test_precision_switch_leaves_no_state(pm, orc, torch):
    """fp32 results after a bf16 call are bitwise those of a fresh fp32
    handle, and the two modes really differ."""
    hs, acts, F, O, B, X, y = case_inputs("f100_b250")
    Xd, yd = dev(torch, X), dev(torch, y)
    ref = pm.PackedMLP(F, O, hs, acts, seed=25)
    want = ref.forward(Xd).cpu().numpy()
    g_want = [t.cpu().numpy() for t in ref.gradients(Xd, yd)]
    net = pm.PackedMLP(F, O, hs, acts, seed=25)
    net.set_precision(pm.PMLP_BF16_GEMM)
    b16 = net.forward(Xd).cpu().numpy()
    net.gradients(Xd, yd)
    net.set_precision(pm.PMLP_FP32)
    assert np.array_equal(net.forward(Xd).cpu().numpy(), want)
    g = [t.cpu().numpy() for t in net.gradients(Xd, yd)]
    assert np.array_equal(g[0], g_want[0]) and np.array_equal(g[1], g_want[1])
    assert not np.array_equal(b16, want)
    with pytest.raises(pm.PmlpError) as e:
        net.set_precision(7)
    assert e.value.code == pm.PMLP_EINVAL
    net.close()
    ref.close()


@pytest.mark.parametrize("wname", ["w60_f10", "w1k_f50"])
def test_bf16_one_epoch(pm, orc, torch, wname):
    w = wl.WORKLOADS[wname]
    hs, acts = w.model_grid()
    X, y = wl.workload_dataset(w)
    net = bf16_net(pm, w.F, w.O, hs, acts, seed=w.init_seed)
    W1, W2 = net.get_params()
    Xd, yd = dev(torch, X), dev(torch, y)
    batches = w.batches()
    for s, n in batches:
        net.train_step(Xd[s:s + n], yd[s:s + n], w.lr)
    last = net.losses()
    R1, R2, rl = orc.train(hs, acts, W1, W2, X, y, batches, w.lr, rounding="bf16")
    assert err_losses(last, rl).max() <= TOL_EPOCH
    logits = np.concatenate([net.forward(Xd[s:s + 1024]).cpu().numpy()
                             for s in range(0, w.S, 1024)])
    got = cross_entropy(logits, y)
    assert err_losses(got, orc.dataset_loss(hs, acts, R1, R2, X, y, rounding="bf16")).max() \
        <= TOL_EPOCH
    # against the exact fp64 oracle
    E1, E2, el = orc.train(hs, acts, W1, W2, X, y, batches, w.lr)
    assert err_losses(last, el).max() <= TOL_EPOCH_VS_EXACT
    assert err_losses(got, orc.dataset_loss(hs, acts, E1, E2, X, y)).max() <= TOL_EPOCH_VS_EXACT
    net.close()


def test_bf16_full_size_w10k_f1000_on_sampled_models(pm, orc, torch):
    """The 10,000-model F = 1000 workload at its full batch of 1024, in the
    launch configuration the benchmark times, on a strided sample of models."""
    w = wl.WORKLOADS["w10k_f1000"]
    hs, acts = w.model_grid()
    X, y = wl.make_dataset(w.F, w.O, w.B, w.data_seed)
    net = bf16_net(pm, w.F, w.O, hs, acts, seed=w.init_seed)
    models = np.unique(np.concatenate([np.arange(7, w.M, w.M // 12), [0, 999, w.M - 1]]))
    sW1, sW2 = net.get_models(models)
    shs, sacts = hs[models], acts[models]
    rows = np.concatenate([np.arange(o, o + h) for o, h in zip(offsets(hs)[models], shs)])
    Xd, yd = dev(torch, X), dev(torch, y)
    dW1, dW2 = net.gradients(Xd, yd)
    loss = net.losses()
    rows_t = torch.from_numpy(rows).cuda()
    g1 = dW1.index_select(0, rows_t).cpu().numpy()
    g2 = dW2.index_select(1, rows_t).cpu().numpy()
    del dW1, dW2
    r1, r2, rl, allow = orc.gradients(shs, sacts, sW1, sW2, X, y, rounding="bf16")
    assert err_rows(g1, r1, shs, allow).max() <= TOL_STEP
    assert err_cols(g2, r2, shs).max() <= TOL_STEP
    assert err_losses(loss[models], rl).max() <= TOL_STEP
    net.train_step(Xd, yd, w.lr)
    T1, T2 = net.get_models(models)
    O1, O2, _ = orc.train(shs, sacts, sW1, sW2, X, y, [(0, w.B)], w.lr, rounding="bf16")
    assert err_rows(T1, O1, shs, w.lr * allow).max() <= TOL_STEP
    assert err_cols(T2, O2, shs).max() <= TOL_STEP
    net.close()


def test_bf16_weight_copy_follows_every_update(pm, torch):
    """The bf16 operand copy of W1 tracks W1 through fp32-mode steps, bf16-mode
    steps and set_params: forward results equal, bit for bit, those of a fresh
    bf16 handle given the same weights."""
    hs, acts, F, O, B, X, y = case_inputs("f100_b250")
    Xd, yd = dev(torch, X), dev(torch, y)
    net = pm.PackedMLP(F, O, hs, acts, seed=26)
    ref = bf16_net(pm, F, O, hs, acts, seed=27)

    def same_as_fresh():
        W1, W2 = net.get_params()
        ref.set_params(W1, W2)
        return np.array_equal(net.forward(Xd).cpu().numpy(), ref.forward(Xd).cpu().numpy())

    net.set_precision(pm.PMLP_BF16_GEMM)
    assert same_as_fresh()
    net.set_precision(pm.PMLP_FP32)
    net.train_step(Xd, yd, 0.1)                 # fp32 update
    net.set_precision(pm.PMLP_BF16_GEMM)
    assert same_as_fresh()
    net.train_step(Xd, yd, 0.1)                 # bf16 update (copy kept by the update)
    assert same_as_fresh()
    W1, W2 = net.get_params()
    net.set_params(W1 * 0.5, W2)                # host update
    assert same_as_fresh()
    net.close()
    ref.close()
