"""Whole-epoch parity at the full-size workloads.

The models of a pack train independently (Section 3: the scatter-add keeps
each model's gradient path separate), so a sample of the models can be
trained alone by the oracle and compared exactly with the same models inside
the full pack, after the full pack has trained for an epoch on the GPU in the
launch configuration the benchmark times.  Per-model normwise bars: 1e-3 for
the losses of the last step, the loss over the whole training set with the
post-epoch weights, and the post-epoch W1 and W2; in the bf16 operand mode the losses are held to the
same bar against the oracle's bf16 mode and to 2e-2 against the exact
oracle, the weights to 2e-2.  Every epoch ends with its partial batch.

Model samples: two models per activation, one narrow and one wide; at the
F = 1000 workload the oracle pays 0.3 s of one core per hidden unit for the
epoch, so its sample keeps to widths up to 40.
"""
import numpy as np
import pytest

import pmlp_workloads as wl
from parity import cross_entropy, err_cols, err_losses, err_rows

pytestmark = pytest.mark.gpu

TOL_EPOCH = 1e-3
TOL_BF16_VS_EXACT = 2e-2


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


def sample_models(w, narrow, wide):
    """Model indices of (activation a, width narrow(a)) and (a, wide(a)) for
    every activation of the act-major, width-ascending grid."""
    per = w.sizes[1] - w.sizes[0] + 1
    out = []
    for a in range(len(w.acts)):
        for h in (narrow(a), wide(a)):
            out.append(a * per + (h - w.sizes[0]))
    return np.unique(np.asarray(out, np.int64))


# widths 1 .. 478 and 1000 .. 451 (1000 and 573 are split into two M3 pieces)
WIDE = (lambda a: 1 + 53 * a, lambda a: 1000 - 61 * a)
# widths 1 .. 28 and 40 .. 22
NARROW = (lambda a: 1 + 3 * a, lambda a: 40 - 2 * a)


def run_epochs(pm, torch, w, models, precision="fp32", epochs=1):
    """Train the full pack on the GPU; return the sampled models' initial
    weights, last-step losses, post-epoch weights and whole-set losses."""
    hs, acts = w.model_grid()
    X, y = wl.workload_dataset(w)
    mode = {"fp32": pm.PMLP_FP32, "bf16": pm.PMLP_BF16_GEMM,
            "bf16_store": pm.PMLP_BF16_STORE}[precision]
    net = pm.PackedMLP(w.F, w.O, hs, acts, seed=w.init_seed, precision=mode)
    sW1, sW2 = net.get_models(models)
    Xd = torch.from_numpy(X).cuda()
    yd = torch.from_numpy(y).cuda()
    batches = w.batches()
    for _ in range(epochs):
        for s, n in batches:
            net.train_step(Xd[s:s + n], yd[s:s + n], w.lr)
    last = net.losses()[models]
    gW1, gW2 = net.get_models(models)
    midx = torch.from_numpy(models).cuda()
    logits = []
    for s in range(0, w.S, 1024):
        out = net.forward(Xd[s:s + 1024])
        logits.append(out.index_select(1, midx).cpu().numpy())
        del out
    full = cross_entropy(np.concatenate(logits), y)
    net.close()
    return dict(hs=hs[models], acts=acts[models], W1=sW1, W2=sW2, X=X, y=y, batches=batches * epochs,
                last=last, gW1=gW1, gW2=gW2, full=full)


def check_against_oracle(orc, w, r, rounding="exact", tol=TOL_EPOCH, wtol=TOL_EPOCH):
    """Losses within tol; post-epoch weights within wtol (None: not compared)."""
    R1, R2, rl = orc.train(r["hs"], r["acts"], r["W1"], r["W2"], r["X"], r["y"], r["batches"],
                           w.lr, rounding=rounding)
    assert err_losses(r["last"], rl).max() <= tol
    want = orc.dataset_loss(r["hs"], r["acts"], R1, R2, r["X"], r["y"], rounding=rounding)
    assert err_losses(r["full"], want).max() <= tol
    if wtol is not None:
        assert err_rows(r["gW1"], R1, r["hs"]).max() <= wtol
        assert err_cols(r["gW2"], R2, r["hs"]).max() <= wtol


@pytest.mark.parametrize("wname", ["w10k_f100", "w10k_f32_o10"])
def test_one_epoch_at_full_size(pm, orc, torch, wname):
    """10,000 models (N = 5,005,000): F = 100, B = 256 (39 batches + 16
    samples) and F = 32, O = 10, B = 32 (1,562 batches + 16 samples)."""
    w = wl.WORKLOADS[wname]
    models = sample_models(w, *WIDE)
    r = run_epochs(pm, torch, w, models)
    check_against_oracle(orc, w, r)


def test_one_epoch_f1000_fp32(pm, orc, torch):
    """F = 1000, B = 1024, 100,000 samples (97 batches + 672 samples)."""
    w = wl.WORKLOADS["w10k_f1000"]
    r = run_epochs(pm, torch, w, sample_models(w, *NARROW))
    check_against_oracle(orc, w, r)


def test_one_epoch_f1000_bf16(pm, orc, torch):
    """The bf16 operand mode at F = 1000, B = 1024: losses within 1e-3 of the
    oracle's bf16 mode and within 2e-2 of the exact oracle; weights within
    2e-2 of the bf16 mode.  The weights get the bf16 bar because the operand
    rounding of W1 is discontinuous: two trajectories that differ only by
    fp32 rounding round some W1 entries to neighbouring bf16 values (a jump
    of 2^-8 relative) at later steps, which ReLU-type kinks then amplify
    (measured 1.1e-3 on ReLU and LeakyReLU models, 1e-5 on the others)."""
    w = wl.WORKLOADS["w10k_f1000"]
    r = run_epochs(pm, torch, w, sample_models(w, *NARROW), precision="bf16")
    check_against_oracle(orc, w, r, rounding="bf16", wtol=TOL_BF16_VS_EXACT)
    check_against_oracle(orc, w, r, rounding="exact", tol=TOL_BF16_VS_EXACT, wtol=None)


def test_one_epoch_f1000_bf16_store(pm, orc, torch):
    """The bf16 storage mode (Z kept in bfloat16) at F = 1000, B = 1024:
    the bars of the bf16 operand mode, against the oracle's storage mode
    and the exact oracle.  The two sides take different sides of some
    bfloat16 rounding ties of Z at every step (both correct), which the
    per-step tests resolve by handing the GPU's choice to the oracle; over
    an epoch they stay within these bars."""
    w = wl.WORKLOADS["w10k_f1000"]
    r = run_epochs(pm, torch, w, sample_models(w, *NARROW), precision="bf16_store")
    check_against_oracle(orc, w, r, rounding="bf16_store", wtol=TOL_BF16_VS_EXACT)
    check_against_oracle(orc, w, r, rounding="exact", tol=TOL_BF16_VS_EXACT, wtol=None)


def test_ten_epochs_w1k(pm, orc, torch):
    """1,000 models (N = 50,500), F = 50, B = 128, 10 epochs of 10,000
    samples (78 batches + 16 samples each), every tenth model checked."""
    w = wl.WORKLOADS["w1k_f50"]
    models = np.arange(3, w.M, 10)
    r = run_epochs(pm, torch, w, models, epochs=w.epochs)
    check_against_oracle(orc, w, r)
