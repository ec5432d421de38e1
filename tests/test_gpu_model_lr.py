"""Per-model learning rates (pmlp_train_step_lr; per-model hyper-parameters
of Section 7) on the GPU, on both kernel paths and in both precision modes."""
import zlib

import numpy as np
import pytest

import pmlp_workloads as wl
from parity import err_cols, err_losses, err_rows, offsets

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


CASES = {
    "f100_b250": dict(M=30, hmax=300, F=100, O=2, B=250),   # fused backward
    "f32_b29_o10": dict(M=25, hmax=200, F=32, O=10, B=29),
    "f150_b300": dict(M=20, hmax=120, F=150, O=2, B=300),   # generic kernels
}


def case_inputs(name):
    c = CASES[name]
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    hs, acts = wl.random_models(rng, c["M"], c["hmax"])
    X, y = wl.make_dataset(c["F"], c["O"], c["B"], seed=int(rng.integers(1 << 30)))
    rates = rng.uniform(0.0, 0.2, c["M"]).astype(np.float32)
    rates[0] = 0.0
    return hs, acts, c["F"], c["O"], c["B"], X, y, rates


def _mode(pm, precision):
    return pm.PMLP_BF16_GEMM if precision == "bf16" else pm.PMLP_FP32


@pytest.mark.parametrize("precision", ["fp32", "bf16"])
@pytest.mark.parametrize("name", sorted(CASES))
def test_per_model_step_matches_oracle(pm, orc, torch, name, precision, path):
    rnd = "bf16" if precision == "bf16" else "exact"
    hs, acts, F, O, B, X, y, rates = case_inputs(name)
    net = pm.PackedMLP(F, O, hs, acts, seed=41, precision=_mode(pm, precision))
    W1, W2 = net.get_params()
    net.train_step(dev(torch, X), dev(torch, y), dev(torch, rates))
    T1, T2 = net.get_params()
    O1, O2, ol = orc.train(hs, acts, W1, W2, X, y, [(0, B)], rates.astype(np.float64),
                           rounding=rnd)
    allow = orc.gradients(hs, acts, W1, W2, X, y, rounding=rnd)[3]
    lr_rows = np.repeat(rates.astype(np.float64), hs)[:, None]
    assert err_losses(net.losses(), ol).max() <= TOL_STEP
    assert err_rows(T1, O1, hs, lr_rows * allow).max() <= TOL_STEP
    assert err_cols(T2, O2, hs).max() <= TOL_STEP
    off = offsets(hs)          # rate 0: model 0 is left exactly as it was
    assert np.array_equal(T1[off[0]:off[1]], W1[off[0]:off[1]])
    assert np.array_equal(T2[:, off[0]:off[1]], W2[:, off[0]:off[1]])
    net.close()


@pytest.mark.parametrize("precision", ["fp32", "bf16"])
@pytest.mark.parametrize("name", ["f100_b250", "f150_b300"])
def test_equal_rates_are_the_scalar_step_bitwise(pm, torch, name, precision, path):
    hs, acts, F, O, B, X, y, _ = case_inputs(name)
    Xd, yd = dev(torch, X), dev(torch, y)
    a = pm.PackedMLP(F, O, hs, acts, seed=42, precision=_mode(pm, precision))
    b = pm.PackedMLP(F, O, hs, acts, seed=42, precision=_mode(pm, precision))
    for _ in range(2):
        a.train_step(Xd, yd, 0.07)
        b.train_step(Xd, yd, dev(torch, np.full(len(hs), 0.07, np.float32)))
    A1, A2 = a.get_params()
    B1, B2 = b.get_params()
    assert np.array_equal(A1, B1) and np.array_equal(A2, B2)
    assert np.array_equal(a.losses(), b.losses())
    a.close()
    b.close()


def test_one_epoch_with_per_model_rates(pm, orc, torch, path):
    w = wl.WORKLOADS["w1k_f50"]
    hs, acts = w.model_grid()
    X, y = wl.workload_dataset(w)
    rates = np.random.default_rng(7).uniform(0.0, 0.05, w.M).astype(np.float32)
    net = pm.PackedMLP(w.F, w.O, hs, acts, seed=w.init_seed)
    W1, W2 = net.get_params()
    Xd, yd, rd = dev(torch, X), dev(torch, y), dev(torch, rates)
    batches = w.batches()
    for s, n in batches:
        net.train_step(Xd[s:s + n], yd[s:s + n], rd)
    R1, R2, rl = orc.train(hs, acts, W1, W2, X, y, batches, rates.astype(np.float64))
    assert err_losses(net.losses(), rl).max() <= TOL_EPOCH
    T1, _ = net.get_params()
    assert err_rows(T1, R1, hs).max() <= TOL_EPOCH
    net.close()


def test_non_finite_rate_is_reported(pm, torch):
    net = pm.PackedMLP(3, 2, [2, 3], [0, 1])
    X = dev(torch, np.ones((4, 3), np.float32))
    y = dev(torch, np.array([0, 1, 1, 0], np.int32))
    net.train_step(X, y, dev(torch, np.array([0.1, np.inf], np.float32)))
    with pytest.raises(pm.PmlpError) as e:
        net.losses()
    assert e.value.code == pm.PMLP_EINVAL and "learning rate" in str(e.value)
    with pytest.raises(pm.PmlpError):
        pm.pmlp_train_step_lr(net.handle, X, y, 4, None)
    with pytest.raises(ValueError):
        net.train_step(X, y, dev(torch, np.array([0.1], np.float32)))
    net.close()
