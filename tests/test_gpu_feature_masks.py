"""GPU parity of per-model input feature masks (feature selection,
Section 7) with the oracle, which trains each model on its own columns of X.

Cases span the kernels whose dW1 epilogue drops the masked gradient: the
three-piece fused backward (F = 100 at 256 samples, F = 50 at 128), the fp32
LDS-resident backward, the matrix-core backward for O > 4, the generic
products, the bf16 operand mode and a handle with biases (never masked).
Bars: 1e-5 per step, 1e-3 after an epoch; masked weights and masked
gradients exactly zero.
"""
import zlib

import numpy as np
import pytest

import pmlp_workloads as wl
from parity import err_cols, err_logits, err_losses, err_rows

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
    "x3_f100_b256": dict(M=24, hmax=200, F=100, O=2, B=256),
    "x3_f50_b128": dict(M=24, hmax=150, F=50, O=2, B=128),
    "lds_f13_b40_o3": dict(M=30, hmax=60, F=13, O=3, B=40),
    "mf_f32_b32_o10": dict(M=20, hmax=300, F=32, O=10, B=32),
    "gemm_f70_b300": dict(M=12, hmax=90, F=70, O=2, B=300),
}


def case_inputs(name):
    c = CASES[name]
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    hs, acts = wl.random_models(rng, c["M"], c["hmax"])
    X, y = wl.make_dataset(c["F"], c["O"], c["B"], seed=int(rng.integers(1 << 30)))
    mask = rng.random((c["M"], c["F"])) < 0.55
    mask[0] = True
    mask[1] = False
    return hs, acts, c["F"], c["O"], c["B"], X, y, mask


def masked_rows(hs, mask):
    return ~mask[np.repeat(np.arange(len(hs)), hs)]


@pytest.mark.parametrize("precision", ["fp32", "bf16"])
@pytest.mark.parametrize("name", sorted(CASES))
def test_forward_and_gradients_with_masks(pm, orc, torch, name, precision, path):
    rnd = "bf16" if precision == "bf16" else "exact"
    hs, acts, F, O, B, X, y, mask = case_inputs(name)
    mode = pm.PMLP_BF16_GEMM if precision == "bf16" else pm.PMLP_FP32
    net = pm.PackedMLP(F, O, hs, acts, seed=61, precision=mode)
    net.set_feature_mask(mask)
    W1, W2 = net.get_params()
    off = masked_rows(hs, mask)
    assert np.all(W1[off] == 0.0)            # zeroed when the masks were set
    Xd, yd = dev(torch, X), dev(torch, y)
    Z, H = net.hidden(Xd)
    RZ, RH = orc.hidden(hs, acts, W1, X, rounding=rnd, mask=mask)
    assert err_cols(Z.cpu().numpy(), RZ, hs).max() <= TOL_STEP
    got = net.forward(Xd).cpu().numpy()
    assert err_logits(got, orc.forward(hs, acts, W1, W2, X, rounding=rnd, mask=mask)).max() <= TOL_STEP
    dW1, dW2 = [t.cpu().numpy() for t in net.gradients(Xd, yd)]
    r1, r2, rl, allow = orc.gradients(hs, acts, W1, W2, X, y, rounding=rnd, mask=mask)
    assert np.all(dW1[off] == 0.0)
    assert err_rows(dW1, r1, hs, allow).max() <= TOL_STEP
    assert err_cols(dW2, r2, hs).max() <= TOL_STEP
    assert err_losses(net.losses(), rl).max() <= TOL_STEP
    net.close()


@pytest.mark.parametrize("name", sorted(CASES))
def test_train_step_with_masks(pm, orc, torch, name, path):
    hs, acts, F, O, B, X, y, mask = case_inputs(name)
    net = pm.PackedMLP(F, O, hs, acts, seed=62)
    net.set_feature_mask(mask)
    W1, W2 = net.get_params()
    net.train_step(dev(torch, X), dev(torch, y), 0.05)
    T1, T2 = net.get_params()
    assert np.all(T1[masked_rows(hs, mask)] == 0.0)
    O1, O2, ol = orc.train(hs, acts, W1, W2, X, y, [(0, B)], 0.05, mask=mask)
    allow = orc.gradients(hs, acts, W1, W2, X, y, mask=mask)[3]
    assert err_losses(net.losses(), ol).max() <= TOL_STEP
    assert err_rows(T1, O1, hs, 0.05 * allow).max() <= TOL_STEP
    assert err_cols(T2, O2, hs).max() <= TOL_STEP
    net.close()


def test_masks_with_biases_leave_the_bias_trained(pm, orc, torch, path):
    hs, acts, F, O, B, X, y, mask = case_inputs("x3_f50_b128")
    F, B = 48, 128                            # rows of 52 with the bias column
    X, y = wl.make_dataset(F, O, B, seed=5)
    mask = mask[:, :F]
    net = pm.PackedMLP(F, O, hs, acts, seed=63, biases=True)
    net.set_feature_mask(mask)
    W1, W2 = net.get_params()
    b1, b2 = net.get_biases()
    Xd, yd = dev(torch, X), dev(torch, y)
    dW1, dW2, db1, db2 = [t.cpu().numpy() for t in net.gradients(Xd, yd)]
    r1, r2, rl, allow, s1, s2, allow_b = orc.gradients(hs, acts, W1, W2, X, y, b1=b1, b2=b2,
                                                       mask=mask)
    assert np.all(dW1[masked_rows(hs, mask)] == 0.0)
    assert err_rows(dW1, r1, hs, allow).max() <= TOL_STEP
    assert err_rows(db1[:, None], s1[:, None], hs, allow_b[:, None]).max() <= TOL_STEP
    net.train_step(Xd, yd, 0.05)
    c1, _ = net.get_biases()
    q1 = orc.train(hs, acts, W1, W2, X, y, [(0, B)], 0.05, b1=b1, b2=b2, mask=mask)[3]
    assert err_rows(c1[:, None], q1[:, None], hs, 0.05 * allow_b[:, None]).max() <= TOL_STEP
    net.close()


def test_set_params_rezeroes_and_none_removes_the_masks(pm, torch):
    hs, acts, F, O, B, X, y, mask = case_inputs("lds_f13_b40_o3")
    net = pm.PackedMLP(F, O, hs, acts, seed=64)
    net.set_feature_mask(mask)
    W1, W2 = net.get_params()
    net.set_params(np.ones_like(W1), W2)
    T1, _ = net.get_params()
    off = masked_rows(hs, mask)
    assert np.all(T1[off] == 0.0) and np.all(T1[~off] == 1.0)
    net.set_feature_mask(None)
    net.train_step(dev(torch, X), dev(torch, y), 0.5)
    U1, _ = net.get_params()
    assert np.any(U1[off] != 0.0)             # no mask any more: those weights train
    net.close()


def test_one_epoch_with_masks(pm, orc, torch, path):
    """1,000 models (h = 1..100 x 10 activations), F = 50, B = 128, one epoch
    of 10,000 samples; each model sees a random half of the features."""
    w = wl.WORKLOADS["w1k_f50"]
    hs, acts = w.model_grid()
    X, y = wl.workload_dataset(w)
    mask = np.random.default_rng(71).random((w.M, w.F)) < 0.5
    net = pm.PackedMLP(w.F, w.O, hs, acts, seed=w.init_seed)
    net.set_feature_mask(mask)
    W1, W2 = net.get_params()
    Xd, yd = dev(torch, X), dev(torch, y)
    batches = w.batches()
    for s, n in batches:
        net.train_step(Xd[s:s + n], yd[s:s + n], w.lr)
    R1, R2, rl = orc.train(hs, acts, W1, W2, X, y, batches, w.lr, mask=mask)
    assert err_losses(net.losses(), rl).max() <= TOL_EPOCH
    T1, T2 = net.get_params()
    assert np.all(T1[masked_rows(hs, mask)] == 0.0)
    assert err_rows(T1, R1, hs).max() <= TOL_EPOCH
    assert err_cols(T2, R2, hs).max() <= TOL_EPOCH
    net.close()
