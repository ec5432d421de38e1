"""Pins of the oracle's SELU, Hardshrink(0.5) and Mish (activation ids 10-12,
the rest of the paper's activation list, Section 4.2).

Values and derivatives are checked against PyTorch's CPU float64 functions
and autograd (library routines, not the oracle), including the conventions
at the kinks; the loss gradient against central finite differences; the
kink allowance and the value-tie counter against constructed ties.
"""
import numpy as np
import pytest
import torch

SELU, HARDSHRINK, MISH = 10, 11, 12
TORCH_FN = {SELU: torch.nn.functional.selu,
            HARDSHRINK: lambda t: torch.nn.functional.hardshrink(t, 0.5),
            MISH: torch.nn.functional.mish}


def _torch_value_and_grad(act_id, zs):
    t = torch.tensor(np.asarray(zs, np.float64), requires_grad=True)
    v = TORCH_FN[act_id](t)
    v.sum().backward()
    return v.detach().numpy(), t.grad.numpy()


@pytest.mark.parametrize("act_id", [SELU, HARDSHRINK, MISH])
def test_values_and_derivatives_match_torch(orc, act_id):
    zs = np.concatenate([np.linspace(-30, 30, 241), [-0.5, 0.5, -0.5000001, 0.5000001,
                                                       -1e-3, 1e-3, 0.0, 19.99, 20.01, 45.0]])
    want_v, want_d = _torch_value_and_grad(act_id, zs)
    got_v = np.array([orc.act(act_id, float(z)) for z in zs])
    got_d = np.array([orc.act_deriv(act_id, float(z)) for z in zs])
    np.testing.assert_allclose(got_v, want_v, rtol=1e-12, atol=1e-300)
    np.testing.assert_allclose(got_d, want_d, rtol=1e-12, atol=1e-15)


def test_kink_conventions(orc):
    lam, alpha = 1.0507009873554805, 1.6732632423543772
    assert orc.act_deriv(SELU, 0.0) == pytest.approx(lam * alpha, rel=1e-15)
    assert orc.act(HARDSHRINK, 0.5) == 0.0 and orc.act(HARDSHRINK, -0.5) == 0.0
    assert orc.act_deriv(HARDSHRINK, 0.5) == 0.0 and orc.act_deriv(HARDSHRINK, -0.5) == 0.0
    assert orc.act(HARDSHRINK, 0.51) == 0.51 and orc.act_deriv(HARDSHRINK, -0.51) == 1.0


def test_gradients_match_finite_differences(orc):
    rng = np.random.default_rng(17)
    F, O, B = 3, 3, 5
    hs = np.tile(np.array([1, 2, 3], np.int32), 3)
    acts = np.repeat(np.array([SELU, HARDSHRINK, MISH], np.int32), 3)
    N = int(hs.sum())
    X = rng.standard_normal((B, F)).astype(np.float32)
    y = rng.integers(0, O, B).astype(np.int32)
    W1 = rng.uniform(-1, 1, (N, F))
    W2 = rng.uniform(-1, 1, (O, N))
    dW1, dW2, _, _ = orc.gradients(hs, acts, W1, W2, X, y)
    Z, _ = orc.hidden(hs, acts, W1, X)
    unit_act = np.repeat(acts, hs)
    dist = np.where(unit_act == HARDSHRINK, np.abs(np.abs(Z) - 0.5), np.abs(Z))
    assert dist.min() > 1e-3          # no sample near a kink: finite differences apply

    def total_loss(a1, a2):
        return orc.gradients(hs, acts, a1, a2, X, y, with_allowance=False)[2].sum()

    h = 1e-6
    fd1 = np.zeros_like(W1)
    for i in np.ndindex(W1.shape):
        P, M_ = W1.copy(), W1.copy()
        P[i] += h
        M_[i] -= h
        fd1[i] = (total_loss(P, W2) - total_loss(M_, W2)) / (2 * h)
    fd2 = np.zeros_like(W2)
    for i in np.ndindex(W2.shape):
        P, M_ = W2.copy(), W2.copy()
        P[i] += h
        M_[i] -= h
        fd2[i] = (total_loss(W1, P) - total_loss(W1, M_)) / (2 * h)
    assert np.abs(fd1 - dW1).max() <= 1e-6 * np.abs(dW1).max()
    assert np.abs(fd2 - dW2).max() <= 1e-6 * np.abs(dW2).max()


@pytest.mark.parametrize("act_id,z0", [(SELU, 0.0), (HARDSHRINK, 0.5), (HARDSHRINK, -0.5)])
def test_kink_allowance_covers_the_other_branch(orc, act_id, z0):
    """A unit whose Z sits exactly on a kink: the gradient with the other
    one-sided derivative stays within the oracle's allowance."""
    X = np.array([[1.0, 1.0], [0.5, -2.0], [2.0, 0.25]], np.float32)
    y = np.array([0, 1, 0], np.int32)
    W1 = np.array([[z0 / 2, z0 / 2]])                  # Z[0] = z0 exactly
    W2 = np.array([[0.3], [-0.6]])
    d0, _, _, allow = orc.gradients([1], [act_id], W1, W2, X, y, kink_rel=1e-6)
    # the other branch at sample 0: dW1 changes by dH * jump * X[0]
    L = orc.forward([1], [act_id], W1, W2, X)[:, 0, :]
    P = np.exp(L - L.max(axis=1, keepdims=True))
    P /= P.sum(axis=1, keepdims=True)
    G = P.copy()
    G[np.arange(3), y] -= 1
    G /= 3
    dH0 = G[0] @ W2[:, 0]
    lam, alpha = 1.0507009873554805, 1.6732632423543772
    jump = lam * (alpha - 1) if act_id == SELU else 1.0
    other = d0 + dH0 * jump * X[0].astype(np.float64)
    assert np.all(allow[0] >= np.abs(other[0] - d0[0]) * (1 - 1e-12))
    assert np.all(allow[0] > 0)


def test_value_ties_count_hardshrink_jumps_only(orc):
    X = np.array([[1.0, 1.0], [0.3, 0.1]], np.float32)
    W1 = np.array([[0.25, 0.25], [0.25, 0.25], [0.25, 0.25], [0.1, 0.4]])   # Z[0] = 0.5 for units 0-2
    hs, acts = [1, 1, 1, 1], [HARDSHRINK, SELU, 1, HARDSHRINK]
    counts = orc.value_ties(hs, acts, W1, X)
    assert list(counts) == [1, 0, 0, 1]           # unit 3: Z[0] = 0.5 as well
    far = orc.value_ties([1], [HARDSHRINK], np.array([[0.05, 0.05]]), X)
    assert list(far) == [0]


def test_training_counts_ties_at_each_step(orc):
    """The tie count of training equals value_ties evaluated at the weights
    each step actually uses."""
    rng = np.random.default_rng(3)
    hs = np.array([3, 4, 2], np.int32)
    acts = np.array([HARDSHRINK, MISH, HARDSHRINK], np.int32)
    X = rng.standard_normal((12, 2)).astype(np.float32)
    y = rng.integers(0, 2, 12).astype(np.int32)
    W1 = np.array([[0.25, 0.25], [0.1, -0.3], [0.6, 0.2], [0.1, 0.1], [0.2, 0.2], [0.3, 0.3],
                   [0.4, 0.4], [0.3, -0.2], [0.5, 0.0]])
    X[0] = [1.0, 1.0]                                  # unit 0 meets the jump at step 1
    W2 = rng.uniform(-0.5, 0.5, (2, 9))
    batches = [(0, 6), (6, 6)]
    _, _, _, ties = orc.train(hs, acts, W1, W2, X, y, batches, 0.1, return_ties=True)
    want = orc.value_ties(hs, acts, W1, X[:6])
    W1a, W2a, _ = orc.train(hs, acts, W1, W2, X, y, batches[:1], 0.1)
    want = want + orc.value_ties(hs, acts, W1a, X[6:])
    assert list(ties) == list(want) and ties[0] >= 1 and ties[1] == 0


# --------------------------------------------------------------------------
# Branch choices at Hardshrink's jumps.  At a value tie several results are
# correct; a checked result names the side it took and the oracle follows it
# inside the tie band only.  Pinned against other activations and against
# PyTorch autograd, not against the oracle's own formulas.
# --------------------------------------------------------------------------

def _tied_single_unit():
    """One unit, w = 0.5, inputs 1, 2, 3, -1: Z = 0.5 (a tie), 1, 1.5, -0.5 (a tie)."""
    X = np.array([[1.0], [2.0], [3.0], [-1.0]], np.float32)
    W1 = np.array([[0.5]])
    W2 = np.array([[0.8], [-0.3]])
    y = np.array([0, 1, 1, 0], np.int32)
    return np.array([1], np.int32), X, W1, W2, y


def test_forced_pass_at_every_tie_equals_the_identity_activation(orc):
    hs, X, W1, W2, y = _tied_single_unit()
    br = np.ones((4, 1), np.uint8)                       # every sample passes
    g = orc.gradients(hs, [HARDSHRINK], W1, W2, X, y, branch=br)
    assert orc.branch_conflicts() == 0
    ident = orc.gradients(hs, [0], W1, W2, X, y)         # identity everywhere
    for a, b in zip(g[:3], ident[:3]):
        np.testing.assert_array_equal(a, b)
    _, H = orc.hidden(hs, [HARDSHRINK], W1, X, branch=br)
    np.testing.assert_array_equal(H[:, 0], [0.5, 1.0, 1.5, -0.5])


def test_forced_zero_at_the_ties_equals_the_unforced_oracle(orc):
    hs, X, W1, W2, y = _tied_single_unit()
    br = np.array([[0], [1], [1], [0]], np.uint8)        # the oracle's own sides
    a = orc.gradients(hs, [HARDSHRINK], W1, W2, X, y, branch=br)
    assert orc.branch_conflicts() == 0
    b = orc.gradients(hs, [HARDSHRINK], W1, W2, X, y)
    for u, v in zip(a[:3], b[:3]):
        np.testing.assert_array_equal(u, v)


def test_forced_branches_match_torch_autograd(orc):
    """Sample 0 passes, sample 3 is zeroed: the same as PyTorch's Hardshrink
    with threshold 0.499 on sample 0 and 0.501 on sample 3 (a threshold
    moved across the tie, everything else unchanged)."""
    hs, X, W1, W2, y = _tied_single_unit()
    br = np.array([[1], [1], [1], [0]], np.uint8)
    dW1, dW2, loss, _ = orc.gradients(hs, [HARDSHRINK], W1, W2, X, y, branch=br)
    w1 = torch.tensor(W1, requires_grad=True)
    w2 = torch.tensor(W2, requires_grad=True)
    z = torch.tensor(X, dtype=torch.float64) @ w1.T                       # [4, 1]
    lam = torch.tensor([[0.499], [0.5], [0.5], [0.501]], dtype=torch.float64)
    h = torch.where(z.abs() > lam, z, torch.zeros_like(z))
    logits = h @ w2.T
    ce = torch.nn.functional.cross_entropy(logits, torch.tensor(y, dtype=torch.long))
    ce.backward()
    np.testing.assert_allclose(dW1, w1.grad.numpy(), rtol=1e-14)
    np.testing.assert_allclose(dW2, w2.grad.numpy(), rtol=1e-14)
    assert loss[0] == pytest.approx(ce.item(), rel=1e-14)


def test_a_choice_outside_the_band_is_counted_and_ignored(orc):
    hs, X, W1, W2, y = _tied_single_unit()
    br = np.array([[0], [0], [1], [0]], np.uint8)        # sample 1 (Z = 1) is no tie
    a = orc.gradients(hs, [HARDSHRINK], W1, W2, X, y, branch=br)
    assert orc.branch_conflicts() == 1
    b = orc.gradients(hs, [HARDSHRINK], W1, W2, X, y)
    np.testing.assert_array_equal(a[0], b[0])
    # in training, rows are offsets into the sample arrays: batch (2, 2)
    # reads rows 2 and 3 only
    orc.train(hs, [HARDSHRINK], W1, W2, X, y, [(2, 2)], 0.1, branch=br)
    assert orc.branch_conflicts() == 0
