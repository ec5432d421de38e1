"""GPU parity with biases (PMLP_BIAS): hidden biases stored as the weight of
a constant input 1 (a column of W1), output biases added by the M3 forward,
db1 from the dW1 product's bias column, db2 = sum_b G in the loss kernel.
Both kernel paths, both precision modes; same bars as the other parity
tests (1e-5 per step, 1e-3 per epoch)."""
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


CASES = {
    "f100_b250": dict(M=30, hmax=300, F=100, O=2, B=250),      # fused backward, spare column
    "f128_b100_o4": dict(M=15, hmax=90, F=128, O=4, B=100),    # extended width 132: generic bwd
    "f13_b7_o3": dict(M=37, hmax=40, F=13, O=3, B=7),
    "f32_b29_o10": dict(M=25, hmax=200, F=32, O=10, B=29),
    "split": dict(hs=[1300, 513, 512, 1, 700, 3, 1024], F=10, O=2, B=33),   # two-halves segments
    "f1000_b300": dict(M=6, hmax=80, F=1000, O=2, B=300),
    # the three-piece fused backward with the bias in its four-column tail:
    # F = 96 (rows of 100 with the bias column) at 256 samples and F = 48
    # (rows of 52) at 128 samples
    "x3_f96_b256": dict(M=20, hmax=150, F=96, O=2, B=256),
    "x3_f48_b128": dict(M=20, hmax=150, F=48, O=2, B=128),
}


def case_inputs(name):
    c = CASES[name]
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    if "hs" in c:
        hs = np.asarray(c["hs"], np.int32)
        acts = rng.integers(0, 10, len(hs)).astype(np.int32)
    else:
        hs, acts = wl.random_models(rng, c["M"], c["hmax"])
    X, y = wl.make_dataset(c["F"], c["O"], c["B"], seed=int(rng.integers(1 << 30)))
    return hs, acts, c["F"], c["O"], c["B"], X, y


def g_scale(logits, y):
    """[M, 1]: the largest sum over samples of |G| bounds, (p + [o = y]) / B."""
    L = np.asarray(logits, np.float64)
    P = np.exp(L - L.max(axis=2, keepdims=True))
    P /= P.sum(axis=2, keepdims=True)
    P[np.arange(L.shape[0]), :, y] += 1.0
    return (P.sum(axis=0) / L.shape[0]).max(axis=1, keepdims=True)


def _net(pm, F, O, hs, acts, seed, precision="fp32"):
    mode = pm.PMLP_BF16_GEMM if precision == "bf16" else pm.PMLP_FP32
    return pm.PackedMLP(F, O, hs, acts, seed=seed, precision=mode, biases=True)


def test_bias_init_is_bit_exact(pm, orc):
    hs, acts, F, O, B, X, y = case_inputs("f13_b7_o3")
    net = _net(pm, F, O, hs, acts, 51)
    b1, b2 = net.get_biases()
    r1, r2 = orc.init_biases(F, O, hs, 51)
    assert np.array_equal(b1, r1) and np.array_equal(b2, r2)
    W1, W2 = net.get_params()                      # weights unchanged by the bias column
    R1, R2 = orc.init_params(F, O, hs, 51)
    assert np.array_equal(W1, R1) and np.array_equal(W2, R2)
    net.close()


@pytest.mark.parametrize("precision", ["fp32", "bf16"])
@pytest.mark.parametrize("name", sorted(CASES))
def test_hidden_forward_gradients_with_biases(pm, orc, torch, name, precision, path):
    rnd = "bf16" if precision == "bf16" else "exact"
    hs, acts, F, O, B, X, y = case_inputs(name)
    net = _net(pm, F, O, hs, acts, 52, precision)
    W1, W2 = net.get_params()
    b1, b2 = net.get_biases()
    Xd, yd = dev(torch, X), dev(torch, y)
    Z, H = net.hidden(Xd)
    RZ, RH = orc.hidden(hs, acts, W1, X, rounding=rnd, b1=b1)
    assert err_cols(Z.cpu().numpy(), RZ, hs).max() <= TOL_STEP
    assert err_cols(H.cpu().numpy(), RH, hs).max() <= TOL_STEP
    got = net.forward(Xd).cpu().numpy()
    want = orc.forward(hs, acts, W1, W2, X, rounding=rnd, b1=b1, b2=b2)
    assert err_logits(got, want).max() <= TOL_STEP
    dW1, dW2, db1, db2 = [t.cpu().numpy() for t in net.gradients(Xd, yd)]
    r1, r2, rl, allow, s1, s2, allow_b = orc.gradients(hs, acts, W1, W2, X, y, rounding=rnd,
                                                       b1=b1, b2=b2)
    assert err_rows(dW1, r1, hs, allow).max() <= TOL_STEP
    assert err_cols(dW2, r2, hs).max() <= TOL_STEP
    # db1: the bias column of the dW1 product (allowance of an input fixed at 1)
    assert err_rows(db1[:, None], s1[:, None], hs, allow_b[:, None]).max() <= TOL_STEP
    # db2 = sum_b G cancels across samples: bound by the size of its terms
    assert np.all(np.abs(db2 - s2) <= TOL_STEP * g_scale(want, y)), np.abs(db2 - s2).max()
    assert err_losses(net.losses(), rl).max() <= TOL_STEP
    net.close()


@pytest.mark.parametrize("name", ["f100_b250", "f128_b100_o4", "split", "x3_f96_b256",
                                  "x3_f48_b128"])
def test_train_step_updates_biases(pm, orc, torch, name, path):
    hs, acts, F, O, B, X, y = case_inputs(name)
    rates = np.random.default_rng(3).uniform(0.0, 0.2, len(hs)).astype(np.float32)
    net = _net(pm, F, O, hs, acts, 53)
    W1, W2 = net.get_params()
    b1, b2 = net.get_biases()
    net.train_step(dev(torch, X), dev(torch, y), dev(torch, rates))
    T1, T2 = net.get_params()
    c1, c2 = net.get_biases()
    O1, O2, ol, q1, q2 = orc.train(hs, acts, W1, W2, X, y, [(0, B)], rates.astype(np.float64),
                                   b1=b1, b2=b2)
    g = orc.gradients(hs, acts, W1, W2, X, y, b1=b1, b2=b2)
    allow, allow_b = g[3], g[6]
    lr_rows = np.repeat(rates.astype(np.float64), hs)[:, None]
    assert err_losses(net.losses(), ol).max() <= TOL_STEP
    assert err_rows(T1, O1, hs, lr_rows * allow).max() <= TOL_STEP
    assert err_cols(T2, O2, hs).max() <= TOL_STEP
    assert err_rows(c1[:, None], q1[:, None], hs, lr_rows * allow_b[:, None]).max() <= TOL_STEP
    logits = orc.forward(hs, acts, W1, W2, X, b1=b1, b2=b2)
    assert np.all(np.abs(c2 - q2) <= TOL_STEP * (np.abs(q2) + rates[:, None] * g_scale(logits, y)))
    net.close()


def test_one_epoch_with_biases(pm, orc, torch, path):
    w = wl.WORKLOADS["w1k_f50"]
    hs, acts = w.model_grid()
    X, y = wl.workload_dataset(w)
    net = _net(pm, w.F, w.O, hs, acts, w.init_seed)
    W1, W2 = net.get_params()
    b1, b2 = net.get_biases()
    Xd, yd = dev(torch, X), dev(torch, y)
    batches = w.batches()
    for s, n in batches:
        net.train_step(Xd[s:s + n], yd[s:s + n], w.lr)
    R1, R2, rl, q1, q2 = orc.train(hs, acts, W1, W2, X, y, batches, w.lr, b1=b1, b2=b2)
    assert err_losses(net.losses(), rl).max() <= TOL_EPOCH
    T1, _ = net.get_params()
    assert err_rows(T1, R1, hs).max() <= TOL_EPOCH
    c1, c2 = net.get_biases()
    assert err_rows(c1[:, None], q1[:, None], hs).max() <= TOL_EPOCH
    net.close()


def test_bias_calls_on_a_handle_without_biases(pm, torch):
    net = pm.PackedMLP(3, 2, [2, 3], [0, 1])
    with pytest.raises(pm.PmlpError) as e:
        pm.pmlp_get_biases(net.handle, 5, 2, 2)
    assert e.value.code == pm.PMLP_ESTATE
    X = dev(torch, np.ones((4, 3), np.float32))
    y = dev(torch, np.zeros(4, np.int32))
    t = torch.empty(64, device="cuda")
    with pytest.raises(pm.PmlpError) as e:
        pm.pmlp_gradients_ex(net.handle, X, y, 4, t, t, t, t)
    assert e.value.code == pm.PMLP_ESTATE
    net.close()


def test_set_biases_round_trip_and_zero_biases_match_no_biases(pm, torch):
    hs, acts, F, O, B, X, y = case_inputs("f100_b250")
    Xd = dev(torch, X)
    a = _net(pm, F, O, hs, acts, 54)
    c = pm.PackedMLP(F, O, hs, acts, seed=54)
    a.set_biases(np.zeros(a.N, np.float32), np.zeros((a.M, O), np.float32))
    b1, b2 = a.get_biases()
    assert not b1.any() and not b2.any()
    assert np.array_equal(a.forward(Xd).cpu().numpy(), c.forward(Xd).cpu().numpy())
    a.close()
    c.close()
