"""Parity of the HIP path (through the C ABI) with the fp64 CPU oracle.

Every test is marked `gpu`.  Tolerances (per-model normwise, see
tests/parity.py): 1e-5 for one forward/backward step in fp32, 1e-3 for
per-model losses after one epoch.  Inputs are seeded and synthetic
(pmlp_workloads); nothing here is produced by the HIP path and then
reused as an expected value.
"""
import zlib

import numpy as np
import pytest

import pmlp_workloads as wl
from conftest import load_golden
from parity import (cross_entropy, dw2_terms, err_cols, err_dw2, err_logits, err_losses,
                    err_rows, offsets, submodel)

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


def dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def make_net(pm, F, O, hs, acts, seed=0, W1=None, W2=None):
    net = pm.PackedMLP(F, O, hs, acts, seed=seed)
    if W1 is not None or W2 is not None:
        net.set_params(W1, W2)
    return net


# Shapes spanning the kernels' tiling: B = 1 and ragged batches, a batch
# wider than 256 (two passes in the backward kernel) and wider than 1024,
# F not a multiple of 4 or 16, O up to 16, widths 1 and segments wider than
# the M3 tile (split into two halves).
CASES = {
    "tiny_b1": dict(hs=[1, 2, 3, 1], F=3, O=2, B=1),
    "ragged": dict(M=37, hmax=40, F=13, O=3, B=7),
    "tile_spanning": dict(hs=[1300, 513, 512, 1, 700, 3, 1024], F=10, O=2, B=33),
    "o10_b32": dict(M=20, hmax=30, F=32, O=10, B=32),
    "o16": dict(M=10, hmax=20, F=5, O=16, B=48),
    "b300_f100": dict(M=12, hmax=50, F=100, O=2, B=300),
    "f1": dict(M=8, hmax=9, F=1, O=2, B=17),
    "b1100": dict(M=6, hmax=20, F=20, O=2, B=1100),
    "all_width_one": dict(hs=[1] * 70, F=7, O=4, B=20),
    # a pack of one model: wide (wider than the tile limit at this size, so
    # two halves) and of width one
    "one_model_wide": dict(hs=[1000], F=20, O=2, B=40),
    "one_model_narrow": dict(hs=[1], F=5, O=3, B=9),
    # shapes of the LDS-resident kernels: batch padded to 16..256, F giving
    # 1, 2, 4, 7 and 8 sixteen-wide column tiles, K tails of 0, 4 and 12
    "f100_b250": dict(M=30, hmax=300, F=100, O=2, B=250),
    "f52_b128": dict(M=25, hmax=120, F=52, O=2, B=128),
    "f128_b100_o4": dict(M=15, hmax=90, F=128, O=4, B=100),
    "f32_b32_o10": dict(M=25, hmax=200, F=32, O=10, B=29),
    "f140_b64": dict(M=12, hmax=64, F=140, O=2, B=64),
    "f12_b16": dict(M=40, hmax=30, F=12, O=2, B=16),
    # the forward with the M3 epilogue: several segments inside one 16-unit
    # tile, segments ending exactly on and just off tile edges, split
    # segments, and the two-pass 256-sample tile
    "fwd_mixed_b256": dict(hs=[3, 1, 1, 17, 16, 15, 600, 2, 1, 33, 1000, 5, 48, 1, 16, 513],
                           F=20, O=2, B=256),
    "fwd_mixed_o4": dict(hs=[3, 1, 1, 17, 16, 15, 600, 2, 1, 33, 1000, 5, 48, 1, 16, 513],
                         F=36, O=4, B=120),
    # the three-piece bf16 kernels: forward with no fp32 remainder (K = 64),
    # with a run-time remainder (K = 40, 52), one or three 32-wide chunks;
    # fused backward at F4 = 100 and 52 with zero-padded columns, for both
    # 128- and 256-sample batches
    "x3_f64_b256": dict(M=14, hmax=80, F=64, O=2, B=256),
    "x3_f40_b200": dict(M=14, hmax=80, F=40, O=3, B=200),
    "x3_f97_b100": dict(M=20, hmax=120, F=97, O=2, B=100),
    "x3_f50_b256": dict(M=20, hmax=120, F=50, O=2, B=256),
    "x3_tiny": dict(hs=[1, 2], F=97, O=2, B=129),
    # widest forward shape of the three-piece kernel: four chunks, one unit
    # tile per wave, three run-time remainder steps
    "x3_f140_b128": dict(M=12, hmax=64, F=140, O=2, B=128),
    # the forward with the activation and M3 in its epilogue: several
    # segments in one 16-unit block, segments ending on and off block edges,
    # halves of wide segments, ragged batches of 256- and 128-sample tiles
    "fm3_mixed_b256": dict(hs=[3, 1, 1, 17, 16, 15, 600, 2, 1, 33, 1000, 5, 48, 1, 16, 513],
                           F=64, O=2, B=250),
    "fm3_mixed_b128": dict(hs=[1] * 40 + [7, 9, 16, 32, 17, 1300, 2, 3, 64, 513],
                           F=100, O=2, B=100),
    "fm3_f128_b128": dict(M=40, hmax=90, F=128, O=2, B=128),
    # the three-piece fused backward at other column counts and four
    # outputs: five blocks, two and seven blocks with the four-column tail,
    # four blocks at O = 4; 116 columns at 256 samples exceed LDS and take
    # the fp32 kernels
    "bx3_f80_b256": dict(M=20, hmax=150, F=80, O=2, B=256),
    "bx3_f36_b128_o4": dict(M=25, hmax=100, F=36, O=4, B=128),
    "bx3_f116_b120": dict(M=15, hmax=120, F=116, O=2, B=120),
    "f116_b200": dict(M=15, hmax=120, F=116, O=2, B=200),
    "bx3_f64_b256_o4": dict(M=20, hmax=100, F=64, O=4, B=256),
    # the three-piece GEMMs (shapes the LDS-resident kernels do not take):
    # 64-, 128- and 256-wide q tiles, K tails of 8 and 0, a ragged last q tile
    "gx3_f1000_b64": dict(M=8, hmax=60, F=1000, O=2, B=64),
    "gx3_f1000_b120_o4": dict(M=8, hmax=60, F=1000, O=4, B=120),
    "gx3_f300_b520": dict(M=10, hmax=90, F=300, O=2, B=520),
    # K = 4 (one stage, twelve of its sixteen k zero) in both products, the
    # dW1 product with four q columns; widths 1 and a two-halves segment
    "gx3_f3_b600_o3": dict(hs=[1, 700, 2, 1300, 5], F=3, O=3, B=600),
    "gx3_f1_b300": dict(M=9, hmax=40, F=1, O=2, B=300),
}

# Kernel paths: the persistent LDS-resident kernels (default where a shape
# allows them), the same with the forward in one kernel (product with the
# activation and M3 in its epilogue, opt-in) where that kernel applies, and
# the generic kernels; selected when the handle is made.
PATHS = ["default", "fused_forward", "generic"]


@pytest.fixture(params=PATHS)
def path(request, monkeypatch):
    monkeypatch.delenv("PMLP_GENERIC_KERNELS", raising=False)
    monkeypatch.delenv("PMLP_FUSED_FORWARD", raising=False)
    if request.param == "generic":
        monkeypatch.setenv("PMLP_GENERIC_KERNELS", "1")
    elif request.param == "fused_forward":
        monkeypatch.setenv("PMLP_FUSED_FORWARD", "1")
    return request.param


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


# --------------------------------------------------------------------------
# Initialisation and the paper's worked examples
# --------------------------------------------------------------------------

@pytest.mark.parametrize("F,O,hs,seed", [
    (10, 2, None, 3000),           # the 60-model grid (h = 1..10 x 6 activations)
    (13, 3, [5, 1, 700, 2], 99),
    (1, 16, [1, 1, 1], 7),
])
def test_init_is_bit_exact(pm, orc, F, O, hs, seed):
    if hs is None:
        hs, acts = wl.WORKLOADS["w60_f10"].model_grid()
    else:
        hs = np.asarray(hs, np.int32)
        acts = np.zeros(len(hs), np.int32)
    net = make_net(pm, F, O, hs, acts, seed=seed)
    W1, W2 = net.get_params()
    R1, R2 = orc.init_params(F, O, hs, seed)
    assert np.array_equal(W1, R1) and np.array_equal(W2, R2)
    net.close()


@pytest.mark.parametrize("O", [2, 3])
def test_scatter_add_worked_example(pm, torch, O):
    """Section 3 Scatter Add example: [1..6] keyed by [0,1,1,2,2,2] gives
    [1, 5, 15]; reproduced with W1 = I, identity activation and W2 = 1."""
    g = load_golden("scatter_example.json")
    S = np.asarray(g["S"], np.float32)
    hs = np.bincount(np.asarray(g["I"][0])).astype(np.int32)
    F = S.shape[1]
    net = make_net(pm, F, O, hs, np.zeros(len(hs), np.int32),
                   W1=np.eye(F, dtype=np.float32), W2=np.ones((O, F), np.float32))
    out = net.forward(dev(torch, S)).cpu().numpy()
    for o in range(O):
        assert np.array_equal(out[0, :, o], np.asarray(g["R"][0], np.float32))
    net.close()


def test_packing_example_4_3_4(pm, orc, torch):
    """Section 3 / Figure 2: a 4-1-2 and a 4-2-2 MLP packed as 4-3-4."""
    g = load_golden("packing_example.json")
    hs = np.asarray(g["hidden_sizes"], np.int32)
    rng = np.random.default_rng(7)
    X = rng.standard_normal((5, g["F"])).astype(np.float32)
    W1 = rng.uniform(-1, 1, (3, g["F"])).astype(np.float32)
    W2 = rng.uniform(-1, 1, (g["O"], 3)).astype(np.float32)
    for act in range(10):
        acts = np.full(2, act, np.int32)
        net = make_net(pm, g["F"], g["O"], hs, acts, W1=W1, W2=W2)
        got = net.forward(dev(torch, X)).cpu().numpy()
        want = orc.forward(hs, acts, W1, W2, X)
        assert err_logits(got, want).max() <= TOL_STEP, act
        net.close()


# --------------------------------------------------------------------------
# One step, element by element, on shapes spanning the tiling
# --------------------------------------------------------------------------

@pytest.mark.parametrize("name", sorted(CASES))
def test_hidden_layer(pm, orc, torch, name):
    hs, acts, F, O, B, X, y = case_inputs(name)
    net = make_net(pm, F, O, hs, acts, seed=11)
    W1, W2 = net.get_params()
    Z, H = net.hidden(dev(torch, X))
    RZ, RH = orc.hidden(hs, acts, W1, X)
    assert err_cols(Z.cpu().numpy(), RZ, hs).max() <= TOL_STEP
    assert err_cols(H.cpu().numpy(), RH, hs).max() <= TOL_STEP
    net.close()


@pytest.mark.parametrize("name", sorted(CASES))
def test_forward_logits(pm, orc, torch, name, path):
    hs, acts, F, O, B, X, y = case_inputs(name)
    net = make_net(pm, F, O, hs, acts, seed=12)
    W1, W2 = net.get_params()
    got = net.forward(dev(torch, X)).cpu().numpy()
    want = orc.forward(hs, acts, W1, W2, X)
    assert got.shape == (B, len(hs), O)
    assert err_logits(got, want).max() <= TOL_STEP
    net.close()


@pytest.mark.parametrize("name", sorted(CASES))
def test_gradients_and_losses(pm, orc, torch, name, path):
    hs, acts, F, O, B, X, y = case_inputs(name)
    net = make_net(pm, F, O, hs, acts, seed=13)
    W1, W2 = net.get_params()
    dW1, dW2 = net.gradients(dev(torch, X), dev(torch, y))
    loss = net.losses()
    r1, r2, rl, allow = orc.gradients(hs, acts, W1, W2, X, y)
    assert err_rows(dW1.cpu().numpy(), r1, hs, allow).max() <= TOL_STEP
    terms = dw2_terms(orc, hs, acts, W1, W2, X, y)
    assert err_dw2(dW2.cpu().numpy(), r2, hs, terms).max() <= TOL_STEP
    assert err_losses(loss, rl).max() <= TOL_STEP
    net.close()


@pytest.mark.parametrize("name", ["ragged", "tile_spanning", "o10_b32", "b300_f100",
                                  "f100_b250", "f128_b100_o4", "f32_b32_o10", "fm3_mixed_b256",
                                  "bx3_f36_b128_o4", "bx3_f116_b120",
                                  "gx3_f1000_b120_o4", "gx3_f300_b520"])
def test_train_step_is_sgd_on_the_same_gradients(pm, orc, torch, name, path):
    """The fused update equals W - lr * dW with dW from the gradient mode
    (to fp32 rounding of W), and the step's losses match the oracle."""
    hs, acts, F, O, B, X, y = case_inputs(name)
    lr = 0.05
    net = make_net(pm, F, O, hs, acts, seed=14)
    W1, W2 = net.get_params()
    Xd, yd = dev(torch, X), dev(torch, y)
    dW1, dW2 = net.gradients(Xd, yd)
    dW1, dW2 = dW1.cpu().numpy(), dW2.cpu().numpy()
    net.train_step(Xd, yd, lr)
    loss = net.losses()
    T1, T2 = net.get_params()
    ulp1 = np.spacing(np.maximum(np.abs(W1), np.abs(T1))) * 2
    ulp2 = np.spacing(np.maximum(np.abs(W2), np.abs(T2))) * 2
    assert np.all(np.abs(T1 - (W1 - lr * dW1)) <= ulp1)
    assert np.all(np.abs(T2 - (W2 - lr * dW2)) <= ulp2)
    O1, O2, ol = orc.train(hs, acts, W1, W2, X, y, [(0, B)], lr)
    allow = orc.gradients(hs, acts, W1, W2, X, y)[3]   # kink ties move dW1, hence W1'
    assert err_losses(loss, ol).max() <= TOL_STEP
    assert err_rows(T1, O1, hs, lr * allow).max() <= TOL_STEP
    assert err_cols(T2, O2, hs).max() <= TOL_STEP
    net.close()


# --------------------------------------------------------------------------
# Gradient isolation (Section 3) on the GPU
# --------------------------------------------------------------------------

# (F, O, B): the scalar M3 kernels (O <= 4) and the matrix-core ones (O > 4)
# with narrow and wide batches, and the three-piece bf16 kernels (F4 = 100
# and 52 with 256- and 128-sample batches); "nan" makes model j diverge (its
# output weights NaN), which must not reach the models sharing its tiles
# either.
@pytest.mark.parametrize("F,O,B", [(9, 3, 40), (32, 10, 32), (20, 12, 70), (100, 2, 200),
                                   (50, 2, 100)])
@pytest.mark.parametrize("kind", ["finite", "nan"])
def test_perturbing_one_model_leaves_the_others_bitwise(pm, torch, F, O, B, kind):
    rng = np.random.default_rng(5)
    hs, acts = wl.random_models(rng, 40, 900)
    X, y = wl.make_dataset(F, O, B, seed=8)
    net = make_net(pm, F, O, hs, acts, seed=15)
    W1, W2 = net.get_params()
    Xd, yd = dev(torch, X), dev(torch, y)
    la = net.forward(Xd).cpu().numpy()
    ga = [t.cpu().numpy() for t in net.gradients(Xd, yd)]
    lossa = net.losses()
    off = offsets(hs)
    j = 17
    P1, P2 = W1.copy(), W2.copy()
    if kind == "finite":
        P1[off[j]:off[j + 1]] += 0.25
        P2[:, off[j]:off[j + 1]] -= 0.5
    else:
        P2[:, off[j]:off[j + 1]] = np.nan
    net.set_params(P1, P2)
    lb = net.forward(Xd).cpu().numpy()
    gb = [t.cpu().numpy() for t in net.gradients(Xd, yd)]
    lossb = net.losses()
    keep = np.ones(len(hs), bool)
    keep[j] = False
    rows = np.repeat(keep, hs)
    assert np.array_equal(la[:, keep], lb[:, keep])
    assert np.array_equal(lossa[keep], lossb[keep])
    assert np.array_equal(ga[0][rows], gb[0][rows])
    assert np.array_equal(ga[1][:, rows], gb[1][:, rows])
    if kind == "finite":
        assert not np.array_equal(la[:, j], lb[:, j])
    else:
        assert np.isnan(lb[:, j]).all()
    net.close()


def test_packed_model_equals_model_alone(pm, torch):
    rng = np.random.default_rng(6)
    hs, acts = wl.random_models(rng, 30, 1000)
    F, O, B = 20, 2, 64
    X, y = wl.make_dataset(F, O, B, seed=9)
    net = make_net(pm, F, O, hs, acts, seed=16)
    W1, W2 = net.get_params()
    Xd, yd = dev(torch, X), dev(torch, y)
    logits = net.forward(Xd).cpu().numpy()
    g1, g2 = [t.cpu().numpy() for t in net.gradients(Xd, yd)]
    off = offsets(hs)
    for m in (0, 7, 29):
        s = slice(off[m], off[m + 1])
        one = make_net(pm, F, O, hs[m:m + 1], acts[m:m + 1], W1=W1[s], W2=W2[:, s])
        lo = one.forward(Xd).cpu().numpy()
        a1, a2 = [t.cpu().numpy() for t in one.gradients(Xd, yd)]
        assert err_logits(lo, logits[:, m:m + 1]).max() <= 1e-6
        assert err_rows(a1, g1[s], hs[m:m + 1]).max() <= 1e-6
        assert err_cols(a2, g2[:, s], hs[m:m + 1]).max() <= 1e-6
        one.close()
    net.close()


# --------------------------------------------------------------------------
# Whole epochs (per-model losses within 1e-3 after one epoch)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("wname", ["w60_f10", "w1k_f50"])
def test_one_epoch(pm, orc, torch, wname, path):
    w = wl.WORKLOADS[wname]
    hs, acts = w.model_grid()
    X, y = wl.workload_dataset(w)
    net = make_net(pm, w.F, w.O, hs, acts, seed=w.init_seed)
    W1, W2 = net.get_params()
    Xd, yd = dev(torch, X), dev(torch, y)
    batches = w.batches()
    for s, n in batches:
        net.train_step(Xd[s:s + n], yd[s:s + n], w.lr)
    last = net.losses()
    T1, T2 = net.get_params()
    R1, R2, rl = orc.train(hs, acts, W1, W2, X, y, batches, w.lr)
    assert err_losses(last, rl).max() <= TOL_EPOCH
    # full-train-set loss with the post-epoch weights: GPU forward + fp64 CE
    logits = np.concatenate([net.forward(Xd[s:s + 1024]).cpu().numpy()
                             for s in range(0, w.S, 1024)])
    got = cross_entropy(logits, y)
    want = orc.dataset_loss(hs, acts, R1, R2, X, y)
    assert err_losses(got, want).max() <= TOL_EPOCH
    assert err_rows(T1, R1, hs).max() <= TOL_EPOCH
    net.close()


# --------------------------------------------------------------------------
# Full-size 10,000-model workloads: one step in the launch configuration the
# benchmark times, checked on a strided sample of models (exact, since the
# models are independent).
# --------------------------------------------------------------------------

@pytest.mark.parametrize("wname", ["w10k_f100", "w10k_f32_o10", "w10k_f1000", "paper_10k"])
def test_full_size_step_on_sampled_models(pm, orc, torch, wname):
    w = wl.WORKLOADS[wname]
    hs, acts = w.model_grid()
    X, y = wl.make_dataset(w.F, w.O, w.B, w.data_seed)
    net = make_net(pm, w.F, w.O, hs, acts, seed=w.init_seed)
    models = np.arange(7, w.M, w.M // 12)
    models = np.unique(np.concatenate([models, [0, 999, w.M - 1]]))
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
    r1, r2, rl, allow = orc.gradients(shs, sacts, sW1, sW2, X, y)
    assert err_rows(g1, r1, shs, allow).max() <= TOL_STEP
    assert err_dw2(g2, r2, shs, dw2_terms(orc, shs, sacts, sW1, sW2, X, y)).max() <= TOL_STEP
    assert err_losses(loss[models], rl).max() <= TOL_STEP
    # the fused update path on the same batch
    net.train_step(Xd, yd, w.lr)
    assert err_losses(net.losses()[models], rl).max() <= TOL_STEP
    T1, T2 = net.get_models(models)
    O1, O2, _ = orc.train(shs, sacts, sW1, sW2, X, y, [(0, w.B)], w.lr)
    assert err_rows(T1, O1, shs, w.lr * allow).max() <= TOL_STEP
    assert err_cols(T2, O2, shs).max() <= TOL_STEP
    net.close()


# --------------------------------------------------------------------------
# Error paths
# --------------------------------------------------------------------------

def test_losses_before_any_step_is_a_state_error(pm):
    net = make_net(pm, 3, 2, [2, 3], [0, 1])
    with pytest.raises(pm.PmlpError) as e:
        net.losses()
    assert e.value.code == pm.PMLP_ESTATE
    net.close()


def test_label_out_of_range_is_reported(pm, torch):
    net = make_net(pm, 3, 2, [2, 3], [0, 1])
    X = dev(torch, np.ones((4, 3), np.float32))
    net.train_step(X, dev(torch, np.array([0, 1, 2, 0], np.int32)), 0.1)
    with pytest.raises(pm.PmlpError) as e:
        net.losses()
    assert e.value.code == pm.PMLP_EINVAL
    net.train_step(X, dev(torch, np.array([0, 1, 1, 0], np.int32)), 0.1)
    assert np.all(np.isfinite(net.losses()))
    net.close()


def test_get_models_equals_slices_of_get_params(pm):
    rng = np.random.default_rng(12)
    hs, acts = wl.random_models(rng, 30, 70)
    net = make_net(pm, 11, 3, hs, acts, seed=17)
    W1, W2 = net.get_params()
    off = offsets(hs)
    models = np.array([29, 0, 7, 7, 15], np.int32)     # any order, repeats allowed
    rows = np.concatenate([np.arange(off[m], off[m + 1]) for m in models])
    a1, a2 = net.get_models(models)
    assert np.array_equal(a1, W1[rows]) and np.array_equal(a2, W2[:, rows])
    with pytest.raises(pm.PmlpError) as e:
        net.get_models([0, 30])
    assert e.value.code == pm.PMLP_EINVAL
    net.close()


# (F, O, B, path, precision) -> the kernels the library reports for the
# forward product and the fused backward, and their arithmetic
VARIANTS = [
    ((100, 2, 256, "default", "fp32"), ("k_fwd_x3", 2), ("k_bwd_x3", 2)),
    ((100, 2, 256, "fused_forward", "fp32"), ("k_fwd_x3m", 2), ("k_bwd_x3", 2)),
    ((50, 2, 128, "fused_forward", "fp32"), ("k_fwd_x3m", 2), ("k_bwd_x3", 2)),
    ((100, 4, 256, "fused_forward", "fp32"), ("k_fwd_x3", 2), ("k_bwd_x3", 2)),
    ((40, 2, 256, "default", "fp32"), ("k_fwd_x3", 2), ("k_bwd_lds", 1)),
    ((116, 2, 120, "default", "fp32"), ("k_fwd_x3", 2), ("k_bwd_x3", 2)),
    ((116, 2, 200, "default", "fp32"), ("k_fwd_lds", 1), ("k_bwd_lds", 1)),
    ((20, 3, 300, "default", "fp32"), ("k_gemm_x3", 2), None),
    ((1000, 2, 64, "default", "fp32"), ("k_gemm_x3", 2), None),
    ((32, 10, 32, "default", "fp32"), ("k_fwd_lds_ring", 1), ("k_bwd_mf", 1)),
    ((20, 2, 100, "default", "fp32"), ("k_fwd_lds", 1), ("k_bwd_lds", 1)),
    ((100, 2, 256, "generic", "fp32"), ("k_gemm_nt", 1), None),
    ((100, 2, 256, "default", "bf16"), ("k_gemm_bf", 3), None),
]


@pytest.mark.parametrize("shape,fwd,bwd", VARIANTS)
def test_kernel_variants_are_reported(pm, torch, monkeypatch, shape, fwd, bwd):
    F, O, B, path, precision = shape
    monkeypatch.delenv("PMLP_GENERIC_KERNELS", raising=False)
    monkeypatch.delenv("PMLP_FUSED_FORWARD", raising=False)
    if path == "generic":
        monkeypatch.setenv("PMLP_GENERIC_KERNELS", "1")
    elif path == "fused_forward":
        monkeypatch.setenv("PMLP_FUSED_FORWARD", "1")
    rng = np.random.default_rng(1)
    hs, acts = wl.random_models(rng, 20, 60)
    net = make_net(pm, F, O, hs, acts, seed=3)
    if precision == "bf16":
        net.set_precision(pm.PMLP_BF16_GEMM)
    X, y = wl.make_dataset(F, O, B, seed=2)
    net.train_step(dev(torch, X), dev(torch, y), 0.01)
    v = net.kernel_variants()
    assert v["fwd_m3" if fwd[0] == "k_fwd_x3m" else "gemm_fwd"] == fwd
    if bwd is not None:
        assert v["bwd_fused"] == bwd
    else:
        assert v["gemm_bwd"] == fwd and v["m3_bwd"] == ("k_m3_bwd", 0)
    assert v["ce"] == ("k_ce", 0)
    net.close()


def test_nonfinite_losses_are_counted(pm, torch):
    """A diverged model (NaN output weights) gives a NaN loss; the library
    counts it per step while the other models train on unaffected."""
    hs = np.array([2, 3, 4], np.int32)
    net = make_net(pm, 3, 2, hs, [0, 1, 2])
    W1, W2 = net.get_params()
    W2[:, 2:5] = np.nan                                   # model 1
    net.set_params(W1, W2)
    X = dev(torch, np.linspace(-1, 1, 12, dtype=np.float32).reshape(4, 3))
    y = dev(torch, np.array([0, 1, 1, 0], np.int32))
    assert net.nonfinite_count() == 0
    net.train_step(X, y, 0.1)
    net.train_step(X, y, 0.1)
    loss = net.losses()
    assert np.isnan(loss[1]) and np.all(np.isfinite(loss[[0, 2]]))
    assert net.nonfinite_count() == 2
    assert net.nonfinite_count() == 0
    net.close()


def test_largest_batch(pm, orc, torch):
    """The largest batch the library takes (2^20 samples, the three-piece
    GEMMs with 4096 q tiles and a 2^20-deep k loop): logits, per-model losses
    and the weights after one step against the oracle.  The weights are
    compared relative to their own size, where the fp32 accumulation over
    2^20 samples in the gradients (an update of about 1% of each weight)
    stays far inside the bar."""
    hs = np.array([1, 3, 2, 5, 16, 1], np.int32)
    acts = np.array([0, 1, 2, 3, 6, 9], np.int32)
    F, O, B, lr = 3, 2, 1 << 20, 0.05
    X, y = wl.make_dataset(F, O, B, seed=77)
    net = make_net(pm, F, O, hs, acts, seed=15)
    W1, W2 = net.get_params()
    Xd, yd = dev(torch, X), dev(torch, y)
    got = net.forward(Xd).cpu().numpy()
    assert err_logits(got, orc.forward(hs, acts, W1, W2, X)).max() <= TOL_STEP
    net.train_step(Xd, yd, lr)
    loss = net.losses()
    T1, T2 = net.get_params()
    O1, O2, ol = orc.train(hs, acts, W1, W2, X, y, [(0, B)], lr)
    allow = orc.gradients(hs, acts, W1, W2, X, y)[3]
    assert err_losses(loss, ol).max() <= TOL_STEP
    assert err_rows(T1, O1, hs, lr * allow).max() <= TOL_STEP
    assert err_cols(T2, O2, hs).max() <= TOL_STEP
    v = net.kernel_variants()
    assert v["gemm_fwd"] == ("k_gemm_x3", 2)
    net.close()


def test_bad_batch_arguments(pm, torch):
    net = make_net(pm, 3, 2, [2, 3], [0, 1])
    X = dev(torch, np.ones((4, 3), np.float32))
    y = dev(torch, np.zeros(4, np.int32))
    for B in (0, -1, (1 << 20) + 1):
        with pytest.raises(pm.PmlpError) as e:
            pm.pmlp_train_step(net.handle, X, y, B, 0.1)
        assert e.value.code == pm.PMLP_EINVAL
    with pytest.raises(pm.PmlpError):
        pm.pmlp_train_step(net.handle, X, y, 4, float("nan"))
    net.close()
