"""GPU parity of the regression head (PMLP_MSE): per-model mean squared error
against real targets, G = 2 (logit - Y) / (B O) from the loss kernel, and
the same forward, backward and update kernels as classification.  Both
kernel paths; the bars of the other parity tests (1e-5 per step, 1e-3 per
epoch) against the oracle's head="mse"."""
import zlib

import numpy as np
import pytest

import pmlp_workloads as wl
from parity import err_cols, err_logits, err_losses, err_rows, offsets

pytestmark = pytest.mark.gpu

TOL_STEP = 1e-5
TOL_EPOCH = 1e-3


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


@pytest.fixture(params=["default", "generic"])
def path(request, monkeypatch):
    if request.param == "generic":
        monkeypatch.setenv("PMLP_GENERIC_KERNELS", "1")
    else:
        monkeypatch.delenv("PMLP_GENERIC_KERNELS", raising=False)
    return request.param


def dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


# the scalar M3 kernels (O <= 4), the matrix-core ones (O > 4), the
# four-column tail of the fused backward (F = 100), split segments, a
# batch wider than 256
CASES = {
    "f13_b7_o3": dict(M=37, hmax=40, F=13, O=3, B=7),
    "f100_b250": dict(M=30, hmax=300, F=100, O=2, B=250),
    "f32_b29_o10": dict(M=25, hmax=200, F=32, O=10, B=29),
    "f20_b70_o16": dict(M=20, hmax=120, F=20, O=16, B=70),
    "split": dict(hs=[1300, 513, 512, 1, 700, 3, 1024], F=10, O=2, B=33),
    "b300_f100": dict(M=12, hmax=50, F=100, O=2, B=300),
}


def case_inputs(name):
    c = CASES[name]
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    if "hs" in c:
        hs = np.asarray(c["hs"], np.int32)
        acts = rng.integers(0, 10, len(hs)).astype(np.int32)
    else:
        hs, acts = wl.random_models(rng, c["M"], c["hmax"])
    X, Y = wl.make_regression_dataset(c["F"], c["O"], c["B"], seed=int(rng.integers(1 << 30)))
    return hs, acts, c["F"], c["O"], c["B"], X, Y


@pytest.mark.parametrize("name", sorted(CASES))
def test_mse_gradients_and_losses(pm, orc, torch, name, path):
    hs, acts, F, O, B, X, Y = case_inputs(name)
    net = pm.PackedMLP(F, O, hs, acts, seed=61, head="mse")
    W1, W2 = net.get_params()
    Xd, Yd = dev(torch, X), dev(torch, Y)
    got = net.forward(Xd).cpu().numpy()
    assert err_logits(got, orc.forward(hs, acts, W1, W2, X)).max() <= TOL_STEP
    dW1, dW2 = [t.cpu().numpy() for t in net.gradients(Xd, Yd)]
    r1, r2, rl, allow = orc.gradients(hs, acts, W1, W2, X, Y, head="mse")
    assert err_rows(dW1, r1, hs, allow).max() <= TOL_STEP
    assert err_cols(dW2, r2, hs).max() <= TOL_STEP
    assert err_losses(net.losses(), rl).max() <= TOL_STEP
    net.close()


@pytest.mark.parametrize("name", ["f13_b7_o3", "f100_b250", "f32_b29_o10"])
def test_mse_train_step_is_sgd_on_the_same_gradients(pm, orc, torch, name, path):
    hs, acts, F, O, B, X, Y = case_inputs(name)
    lr = 0.05
    net = pm.PackedMLP(F, O, hs, acts, seed=62, head="mse")
    W1, W2 = net.get_params()
    net.train_step(dev(torch, X), dev(torch, Y), lr)
    G1, G2 = net.get_params()
    R1, R2, rl = orc.train(hs, acts, W1, W2, X, Y, [(0, B)], lr, head="mse")
    _, _, _, allow = orc.gradients(hs, acts, W1, W2, X, Y, head="mse")
    assert err_rows(G1, R1, hs, lr * allow).max() <= TOL_STEP
    assert err_cols(G2, R2, hs).max() <= TOL_STEP
    assert err_losses(net.losses(), rl).max() <= TOL_STEP
    net.close()


def test_mse_one_epoch(pm, orc, torch, path):
    rng = np.random.default_rng(63)
    hs, acts = wl.random_models(rng, 60, 40)
    F, O, S, B, lr = 12, 3, 600, 32, 0.05
    X, Y = wl.make_regression_dataset(F, O, S, seed=64)
    net = pm.PackedMLP(F, O, hs, acts, seed=65, head="mse")
    W1, W2 = net.get_params()
    Xd, Yd = dev(torch, X), dev(torch, Y)
    batches = wl.batch_bounds(S, B)
    for s, n in batches:
        net.train_step(Xd[s:s + n], Yd[s:s + n], lr)
    got = net.losses()
    R1, R2, rl = orc.train(hs, acts, W1, W2, X, Y, batches, lr, head="mse")
    assert err_losses(got, rl).max() <= TOL_EPOCH
    G1, G2 = net.get_params()
    full = orc.dataset_loss(hs, acts, G1, G2, X, Y, head="mse")
    want = orc.dataset_loss(hs, acts, R1, R2, X, Y, head="mse")
    assert err_losses(full, want).max() <= TOL_EPOCH
    # the regression trained: the oracle's dataset loss fell for most models
    # (a width-1 model whose unit is dead cannot move)
    start = orc.dataset_loss(hs, acts, W1, W2, X, Y, head="mse")
    assert np.mean(want < start) >= 0.8
    net.close()


def test_mse_independence_bitwise(pm, torch):
    hs, acts, F, O, B, X, Y = case_inputs("f32_b29_o10")
    net = pm.PackedMLP(F, O, hs, acts, seed=66, head="mse")
    W1, W2 = net.get_params()
    Xd, Yd = dev(torch, X), dev(torch, Y)
    ga = [t.cpu().numpy() for t in net.gradients(Xd, Yd)]
    la = net.losses()
    off = offsets(hs)
    j = 9
    P2 = W2.copy()
    P2[:, off[j]:off[j + 1]] *= -1.5
    net.set_params(W1, P2)
    gb = [t.cpu().numpy() for t in net.gradients(Xd, Yd)]
    lb = net.losses()
    keep = np.ones(len(hs), bool)
    keep[j] = False
    rows = np.repeat(keep, hs)
    assert np.array_equal(la[keep], lb[keep])
    assert np.array_equal(ga[0][rows], gb[0][rows])
    assert np.array_equal(ga[1][:, rows], gb[1][:, rows])
    net.close()


def test_heads_reject_each_others_calls(pm, torch):
    F, O, B = 4, 2, 8
    X, y = wl.make_dataset(F, O, B, seed=1)
    _, Y = wl.make_regression_dataset(F, O, B, seed=1)
    Xd, yd, Yd = dev(torch, X), dev(torch, y), dev(torch, Y)
    reg = pm.pmlp_create(F, O, [3, 2], [1, 2], 0, pm.PMLP_MSE)
    cls = pm.pmlp_create(F, O, [3, 2], [1, 2], 0, 0)
    with pytest.raises(pm.PmlpError) as e:
        pm.pmlp_train_step(reg, Xd, yd, B, 0.1)
    assert e.value.code == pm.PMLP_ESTATE
    with pytest.raises(pm.PmlpError) as e:
        pm.pmlp_train_step_mse(cls, Xd, Yd, B, 0.1)
    assert e.value.code == pm.PMLP_ESTATE
    with pytest.raises(pm.PmlpError) as e:
        pm.pmlp_train_step_mse(reg, Xd, None, B, 0.1)
    assert e.value.code == pm.PMLP_EINVAL
    pm.pmlp_train_step_mse(reg, Xd, Yd, B, 0.1)
    assert np.all(np.isfinite(pm.pmlp_losses(reg)))
    pm.pmlp_destroy(reg)
    pm.pmlp_destroy(cls)
