"""Pins of the CPU oracle to facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: values the
paper prints (Section 3 examples), closed forms, textbook matrix products,
library special functions, finite differences and the independence
invariants the method is built on.  None of them needs a GPU.
"""
import math

import numpy as np
import pytest
from scipy import special

from conftest import load_golden
import pmlp_workloads as wl


def _reference_act(act_id, z):
    """Activation values from library special functions (not the oracle)."""
    z = np.asarray(z, np.float64)
    if act_id == 0:
        return z.copy()
    if act_id == 1:
        return np.maximum(z, 0.0)
    if act_id == 2:
        return np.tanh(z)
    if act_id == 3:
        return special.expit(z)
    if act_id == 4:
        return np.where(z > 0, z, np.expm1(np.minimum(z, 0)))
    if act_id == 5:
        return np.where(z > 0, z, 0.01 * z)
    if act_id == 6:
        return z * special.ndtr(z)            # x * Phi(x), Phi = normal CDF
    if act_id == 7:
        return z * special.expit(z)
    if act_id == 8:
        return np.where(z > 20, z, np.logaddexp(0.0, z))
    if act_id == 9:
        return z * special.expit(2 * z)
    raise ValueError(act_id)


# --------------------------------------------------------------------------
# Values printed in the paper
# --------------------------------------------------------------------------

def test_scatter_add_worked_example(orc):
    """Section 3 Scatter Add example: [1..6] keyed by [0,1,1,2,2,2] -> [1,5,15].

    With W1 = I (F = 6), identity activation and W2 = 1, the hidden layer
    equals the source row and each model's logit is the scatter-add of its
    hidden segment; hidden sizes 1, 2, 3 reproduce the index row."""
    g = load_golden("scatter_example.json")
    S = np.asarray(g["S"], np.float32)
    I = np.asarray(g["I"][0])
    R = np.asarray(g["R"][0], np.float64)
    hs = np.bincount(I).astype(np.int32)
    assert list(hs) == [1, 2, 3]
    F = S.shape[1]
    for O in (2, 3):
        logits = orc.forward(hs, np.zeros(3, np.int32), np.eye(F), np.ones((O, F)), S)
        assert logits.shape == (1, 3, O)
        for o in range(O):
            assert np.array_equal(logits[0, :, o], R)


def test_packing_example_4_3_4(orc):
    """Section 3 / Figure 2: 4-1-2 and 4-2-2 packed as 4-3-4 with I row [0,1,1].

    The packed network's logits equal each MLP evaluated alone with plain
    matrix products (textbook forward of Section 3)."""
    g = load_golden("packing_example.json")
    hs = np.asarray(g["hidden_sizes"], np.int32)
    F, O = g["F"], g["O"]
    assert int(hs.sum()) == g["packed_hidden"] and len(hs) * O == g["packed_outputs"]
    mid = np.repeat(np.arange(len(hs)), hs)
    assert all(list(mid) == row for row in g["I"])
    rng = np.random.default_rng(7)
    X = rng.standard_normal((5, F)).astype(np.float32)
    W1 = rng.uniform(-1, 1, (3, F))
    W2 = rng.uniform(-1, 1, (O, 3))
    for act in range(10):
        acts = np.full(2, act, np.int32)
        got = orc.forward(hs, acts, W1, W2, X)
        for m in range(2):
            cols = mid == m
            Z = X.astype(np.float64) @ W1[cols].T
            want = _reference_act(act, Z) @ W2[:, cols].T
            np.testing.assert_allclose(got[:, m, :], want, rtol=1e-13, atol=1e-13)


# --------------------------------------------------------------------------
# Special cases that reduce to textbook routines / closed forms
# --------------------------------------------------------------------------

def test_single_identity_model_is_two_matmuls(orc):
    rng = np.random.default_rng(1)
    F, O, h, B = 7, 4, 9, 6
    X = rng.standard_normal((B, F)).astype(np.float32)
    W1 = rng.standard_normal((h, F))
    W2 = rng.standard_normal((O, h))
    got = orc.forward([h], [0], W1, W2, X)[:, 0, :]
    want = (X.astype(np.float64) @ W1.T) @ W2.T
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_all_width_one_is_elementwise(orc):
    """All h_m = 1: the M3 product degenerates to logits[b,m,o] = act(Z[b,m]) W2[o,m]."""
    rng = np.random.default_rng(2)
    F, O, B = 5, 3, 8
    acts = np.arange(10, dtype=np.int32)
    hs = np.ones(10, np.int32)
    X = rng.standard_normal((B, F)).astype(np.float32)
    W1 = rng.standard_normal((10, F))
    W2 = rng.standard_normal((O, 10))
    got = orc.forward(hs, acts, W1, W2, X)
    Z = X.astype(np.float64) @ W1.T
    for m in range(10):
        want = _reference_act(m, Z[:, m])[:, None] * W2[:, m][None, :]
        np.testing.assert_allclose(got[:, m, :], want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("O", [2, 3, 10])
def test_zero_output_weights_closed_form(orc, O):
    """W2 = 0: every loss is ln O, dH = 0 so dW1 = 0, and dW2 = G^T H with
    G = (1/O - onehot(y)) / B."""
    rng = np.random.default_rng(3)
    hs, acts = wl.random_models(rng, 12, 6)
    N, F, B = int(hs.sum()), 4, 9
    X = rng.standard_normal((B, F)).astype(np.float32)
    y = rng.integers(0, O, B).astype(np.int32)
    W1 = rng.standard_normal((N, F))
    dW1, dW2, loss, _ = orc.gradients(hs, acts, W1, np.zeros((O, N)), X, y)
    np.testing.assert_allclose(loss, math.log(O), rtol=1e-15, atol=0)
    assert np.all(dW1 == 0.0)
    G = (np.full((B, O), 1.0 / O) - np.eye(O)[y]) / B
    Z = X.astype(np.float64) @ W1.T
    mid = np.repeat(np.arange(len(hs)), hs)
    H = np.stack([_reference_act(acts[mid[n]], Z[:, n]) for n in range(N)], axis=1)
    np.testing.assert_allclose(dW2, G.T @ H, rtol=1e-12, atol=1e-14)


def test_cross_entropy_two_class_closed_form(orc):
    """O = 2: per-sample CE = log(1 + exp(l_other - l_y)) (softplus of the margin)."""
    rng = np.random.default_rng(4)
    F, B = 3, 11
    X = rng.standard_normal((B, F)).astype(np.float32)
    y = rng.integers(0, 2, B).astype(np.int32)
    W1 = rng.standard_normal((2, F))
    W2 = rng.standard_normal((2, 2))
    _, _, loss, _ = orc.gradients([2], [0], W1, W2, X, y)
    logits = (X.astype(np.float64) @ W1.T) @ W2.T
    margin = logits[np.arange(B), 1 - y] - logits[np.arange(B), y]
    np.testing.assert_allclose(loss[0], np.mean(np.logaddexp(0.0, margin)), rtol=1e-14)


# --------------------------------------------------------------------------
# Activations
# --------------------------------------------------------------------------

@pytest.mark.parametrize("act_id", range(10))
def test_activation_values_match_special_functions(orc, act_id):
    zs = np.concatenate([np.linspace(-30, 30, 241), [-1e-3, 1e-3, 0.0, 19.99, 20.01, 45.0]])
    got = np.array([orc.act(act_id, float(z)) for z in zs])
    want = _reference_act(act_id, zs)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-300)


@pytest.mark.parametrize("act_id", range(10))
def test_activation_derivatives_match_finite_differences(orc, act_id):
    zs = np.concatenate([np.linspace(-8, 8, 97), [-19.5, 25.0]])
    zs = zs[np.abs(zs) > 1e-3]                     # away from the ReLU/LeakyReLU kink
    zs = zs[np.abs(zs - 20.0) > 1e-3]               # and from the softplus switch
    eps = 1e-6
    for z in zs:
        fd = (orc.act(act_id, z + eps) - orc.act(act_id, z - eps)) / (2 * eps)
        assert abs(orc.act_deriv(act_id, z) - fd) <= 1e-8 * max(1.0, abs(fd)), (act_id, z)


def test_activation_kink_conventions(orc):
    assert orc.act_deriv(1, 0.0) == 0.0                 # ReLU'(0) = 0
    assert orc.act_deriv(5, 0.0) == 0.01                # LeakyReLU'(0) = slope
    assert orc.act_deriv(4, 0.0) == 1.0                 # ELU'(0) = 1 (alpha = 1)
    assert orc.act_deriv(8, 21.0) == 1.0                # softplus linear region


# --------------------------------------------------------------------------
# Gradients: central finite differences of the summed loss
# --------------------------------------------------------------------------

def test_gradients_match_finite_differences(orc):
    rng = np.random.default_rng(5)
    F, O, B = 3, 3, 5
    hs = np.tile(np.array([1, 2, 3], np.int32), 10)
    acts = np.repeat(np.arange(10, dtype=np.int32), 3)
    N = int(hs.sum())
    X = rng.standard_normal((B, F)).astype(np.float32)
    y = rng.integers(0, O, B).astype(np.int32)
    W1 = rng.uniform(-1, 1, (N, F))
    W2 = rng.uniform(-1, 1, (O, N))
    dW1, dW2, loss, _ = orc.gradients(hs, acts, W1, W2, X, y)

    def total(a, b):
        return orc.gradients(hs, acts, a, b, X, y, with_allowance=False)[2].sum()

    eps = 1e-6
    Z = X.astype(np.float64) @ W1.T
    mid = np.repeat(np.arange(len(hs)), hs)
    kinky = np.isin(acts[mid], [1, 5]) & (np.abs(Z).min(axis=0) < 1e-4)
    fd1 = np.zeros_like(W1)
    for n in range(N):
        for f in range(F):
            a, b = W1.copy(), W1.copy()
            a[n, f] += eps
            b[n, f] -= eps
            fd1[n, f] = (total(a, W2) - total(b, W2)) / (2 * eps)
    fd2 = np.zeros_like(W2)
    for o in range(O):
        for n in range(N):
            a, b = W2.copy(), W2.copy()
            a[o, n] += eps
            b[o, n] -= eps
            fd2[o, n] = (total(W1, a) - total(W1, b)) / (2 * eps)
    ok = ~kinky
    err1 = np.abs(fd1 - dW1)[ok].max() / np.abs(dW1[ok]).max()
    err2 = np.abs(fd2 - dW2).max() / np.abs(dW2).max()
    assert err1 < 1e-6 and err2 < 1e-6, (err1, err2)


def test_kink_allowance_covers_branch_choice(orc):
    """A ReLU unit with Z exactly 0: the derivative is ambiguous and the
    allowance must cover the gap between the two one-sided gradients."""
    F, O = 2, 2
    X = np.array([[1.0, -1.0], [0.5, 2.0]], np.float32)
    y = np.array([0, 1], np.int32)
    W1 = np.array([[0.75, 0.75]])           # Z[0] = 0 exactly, Z[1] > 0
    W2 = np.array([[0.3], [-0.6]])
    d0, _, _, allow = orc.gradients([1], [1], W1, W2, X, y, kink_rel=1e-6)
    # Right-hand derivative: a ReLU with its kink nudged below zero.
    _, _, _, _ = orc.gradients([1], [1], W1, W2, X, y)
    dright = orc.gradients([1], [0], W1, W2, X, y, with_allowance=False)[0]  # slope 1 everywhere
    assert np.all(allow > 0)
    assert np.all(np.abs(dright - d0) <= allow + 1e-15)


# --------------------------------------------------------------------------
# Independence invariants (Section 3: gradient paths never mix)
# --------------------------------------------------------------------------

def _problem(seed, M=24, hmax=9, F=5, O=3, B=7):
    rng = np.random.default_rng(seed)
    hs, acts = wl.random_models(rng, M, hmax)
    N = int(hs.sum())
    X = rng.standard_normal((2 * B, F)).astype(np.float32)
    y = rng.integers(0, O, 2 * B).astype(np.int32)
    W1 = rng.uniform(-0.5, 0.5, (N, F))
    W2 = rng.uniform(-0.5, 0.5, (O, N))
    return hs, acts, X, y, W1, W2


def test_perturbing_one_model_leaves_others_bitwise_unchanged(orc):
    hs, acts, X, y, W1, W2 = _problem(11)
    off = np.concatenate([[0], np.cumsum(hs)])
    j = 5
    W1p, W2p = W1.copy(), W2.copy()
    W1p[off[j]:off[j + 1]] += 0.25
    W2p[:, off[j]:off[j + 1]] -= 0.5
    a = orc.gradients(hs, acts, W1, W2, X, y)
    b = orc.gradients(hs, acts, W1p, W2p, X, y)
    la, lb = orc.forward(hs, acts, W1, W2, X), orc.forward(hs, acts, W1p, W2p, X)
    keep = np.ones(len(hs), bool)
    keep[j] = False
    rows = np.repeat(keep, hs)
    assert np.array_equal(la[:, keep], lb[:, keep])
    assert np.array_equal(a[2][keep], b[2][keep])
    assert np.array_equal(a[0][rows], b[0][rows])
    assert np.array_equal(a[1][:, rows], b[1][:, rows])
    assert not np.array_equal(a[2][j], b[2][j])


def test_packed_model_equals_model_alone(orc):
    hs, acts, X, y, W1, W2 = _problem(12)
    off = np.concatenate([[0], np.cumsum(hs)])
    batches = [(0, 7), (7, 7)]
    P1, P2, pl = orc.train(hs, acts, W1, W2, X, y, batches, lr=0.1)
    for m in (0, 3, len(hs) - 1):
        s = slice(off[m], off[m + 1])
        A1, A2, al = orc.train(hs[m:m + 1], acts[m:m + 1], W1[s], W2[:, s], X, y, batches, lr=0.1)
        assert np.array_equal(P1[s], A1) and np.array_equal(P2[:, s], A2)
        assert pl[m] == al[0]


def test_model_order_is_irrelevant(orc):
    hs, acts, X, y, W1, W2 = _problem(13)
    off = np.concatenate([[0], np.cumsum(hs)])
    perm = np.random.default_rng(0).permutation(len(hs))
    rows = np.concatenate([np.arange(off[m], off[m + 1]) for m in perm])
    a = orc.gradients(hs, acts, W1, W2, X, y)
    b = orc.gradients(hs[perm], acts[perm], W1[rows], W2[:, rows], X, y)
    assert np.array_equal(a[2][perm], b[2])
    assert np.array_equal(a[0][rows], b[0])
    assert np.array_equal(a[1][:, rows], b[1])


def test_train_step_is_sgd_on_gradients(orc):
    hs, acts, X, y, W1, W2 = _problem(14)
    dW1, dW2, loss, _ = orc.gradients(hs, acts, W1, W2, X[:7], y[:7])
    T1, T2, tl = orc.train(hs, acts, W1, W2, X, y, [(0, 7)], lr=0.05)
    np.testing.assert_array_equal(T1, W1 - 0.05 * dW1)
    np.testing.assert_array_equal(T2, W2 - 0.05 * dW2)
    np.testing.assert_array_equal(tl, loss)


def test_small_learning_rate_decreases_loss(orc):
    hs, acts, X, y, W1, W2 = _problem(15)
    before = orc.dataset_loss(hs, acts, W1, W2, X[:7], y[:7])
    T1, T2, _ = orc.train(hs, acts, W1, W2, X, y, [(0, 7)], lr=1e-3)
    after = orc.dataset_loss(hs, acts, T1, T2, X[:7], y[:7])
    assert np.all(after < before)


def test_subset_training_matches_full(orc):
    hs, acts, X, y, W1, W2 = _problem(16)
    full = orc.train(hs, acts, W1, W2, X, y, [(0, 7), (7, 7)], lr=0.1)
    sub = [1, 4, 9]
    part = orc.train(hs, acts, W1, W2, X, y, [(0, 7), (7, 7)], lr=0.1, models=sub)
    off = np.concatenate([[0], np.cumsum(hs)])
    for m in sub:
        s = slice(off[m], off[m + 1])
        assert np.array_equal(full[0][s], part[0][s]) and full[2][m] == part[2][m]


def test_invalid_labels_and_sizes_rejected(orc):
    hs, acts, X, y, W1, W2 = _problem(17)
    bad = y.copy()
    bad[0] = 99
    _, _, loss, _ = orc.gradients(hs, acts, W1, W2, X, bad)
    assert np.all(np.isnan(loss))
    with pytest.raises(RuntimeError):
        orc.forward(np.array([0], np.int32), [0], W1[:1], W2[:, :1], X)
    with pytest.raises(RuntimeError):
        orc.forward([1], [13], W1[:1], W2[:, :1], X)


# --------------------------------------------------------------------------
# Initialisation (counter-based splitmix64)
# --------------------------------------------------------------------------

def test_splitmix64_published_outputs(orc):
    g = load_golden("splitmix64.json")
    gamma = 0x9E3779B97F4A7C15
    got = [orc.splitmix64((g["state"] + k * gamma) % 2**64) for k in range(5)]
    assert got == [int(v) for v in g["outputs"]]


def test_init_follows_counter_definition(orc):
    hs = np.array([3, 1, 4], np.int32)
    F, O, seed = 6, 2, 99
    W1, W2 = orc.init_params(F, O, hs, seed)
    key = orc.splitmix64(seed)
    N = int(hs.sum())

    def draw(tag, idx, fan_in):
        r = orc.splitmix64(key ^ (tag << 60) ^ idx)
        u = (r >> 40) / float(1 << 24)
        return np.float32(2.0 * u - 1.0) * np.float32(1.0 / math.sqrt(fan_in))

    for n in range(N):
        for f in range(F):
            assert W1[n, f] == draw(1, n * F + f, F)
    mid = np.repeat(np.arange(3), hs)
    for o in range(O):
        for n in range(N):
            assert W2[o, n] == draw(2, o * N + n, hs[mid[n]])


def test_init_distribution(orc):
    hs = np.array([400, 900], np.int32)
    F = 256
    W1, W2 = orc.init_params(F, 3, hs, 5)
    b1 = 1.0 / math.sqrt(F)
    assert np.abs(W1).max() <= b1
    assert abs(W1.mean()) < 3 * b1 / math.sqrt(3 * W1.size) * 3
    assert abs(W1.var() / (b1 * b1 / 3) - 1) < 0.01
    b2 = 1.0 / math.sqrt(900)
    assert np.abs(W2[:, 400:]).max() <= b2 and np.abs(W2[:, 400:]).max() > 0.95 * b2


# --------------------------------------------------------------------------
# Workload generator (inputs only)
# --------------------------------------------------------------------------

def test_workload_shapes():
    w = wl.WORKLOADS["w10k_f100"]
    hs, acts = w.model_grid()
    assert w.M == len(hs) == 10000 and w.N == int(hs.sum()) == 5005000
    assert list(hs[:3]) == [1, 2, 3] and acts[999] == 0 and acts[1000] == 1
    assert wl.batch_bounds(10000, 256)[-1] == (9984, 16)
    assert len(wl.batch_bounds(10000, 256)) == 40
    assert wl.WORKLOADS["w60_f10"].N == 330
    assert wl.WORKLOADS["w1k_f50"].N == 50500
    X, y = wl.make_dataset(5, 3, 100, 1)
    X2, y2 = wl.make_dataset(5, 3, 100, 1)
    assert X.dtype == np.float32 and y.dtype == np.int32
    assert np.array_equal(X, X2) and np.array_equal(y, y2)
    assert set(np.unique(y)) <= {0, 1, 2}


def test_hidden_layer_is_matmul_then_activation(orc):
    """Steps 1-2 of the packed procedure: Z is one plain matrix product over
    all concatenated hidden units; H applies each portion's activation."""
    rng = np.random.default_rng(21)
    hs, acts = wl.random_models(rng, 15, 7)
    N, F, B = int(hs.sum()), 6, 5
    X = rng.standard_normal((B, F)).astype(np.float32)
    W1 = rng.standard_normal((N, F))
    Z, H = orc.hidden(hs, acts, W1, X)
    np.testing.assert_allclose(Z, X.astype(np.float64) @ W1.T, rtol=1e-13, atol=1e-13)
    mid = np.repeat(np.arange(len(hs)), hs)
    for n in range(N):
        np.testing.assert_allclose(H[:, n], _reference_act(acts[mid[n]], Z[:, n]),
                                   rtol=1e-12, atol=1e-300)


def test_cancellation_allowance_covers_fp32_error_of_dH(orc):
    """One width-1 unit with nearly equal output weights (dH = G W2 cancels
    ~500-fold): a CPU fp32 evaluation with G carrying a few ulp of error
    stays within the allowance; with output weights of opposite sign (no
    cancellation across outputs) it is negligible."""
    rng = np.random.default_rng(12)
    F, O, B = 6, 2, 40
    X = rng.standard_normal((B, F)).astype(np.float32)
    y = rng.integers(0, O, B).astype(np.int32)
    W1 = rng.uniform(-0.5, 0.5, (1, F))
    for W2, cancels in ((np.array([[0.5392], [0.5415]]), True),
                        (np.array([[0.5392], [-0.5415]]), False)):
        d0, _, _, allow = orc.gradients([1], [2], W1, W2, X, y)
        if not cancels:
            assert allow.max() <= 1e-7 * np.abs(d0).max()
            continue
        L = orc.forward([1], [2], W1, W2, X)[:, 0, :]
        P = np.exp(L - L.max(axis=1, keepdims=True))
        P /= P.sum(axis=1, keepdims=True)
        G = P.copy()
        G[np.arange(B), y] -= 1
        G /= B
        Z = (X.astype(np.float64) @ W1[0])
        worst = 0.0
        for trial in range(10):
            Gp = (G * (1 + rng.uniform(-3, 3, G.shape) * 2.0 ** -24)).astype(np.float32)
            dH = (Gp[:, 0] * np.float32(W2[0, 0]) + Gp[:, 1] * np.float32(W2[1, 0]))
            dZ = dH.astype(np.float64) * (1 - np.tanh(Z) ** 2)
            dW1 = dZ @ X.astype(np.float64)
            assert np.all(np.abs(dW1 - d0[0]) <= allow[0]), trial
            worst = max(worst, np.abs(dW1 - d0[0]).max())
        # the fp32 error really exceeds the per-model budget of 1e-5 here
        assert worst > 1e-5 * np.abs(d0[0]).max()


def test_per_model_learning_rates_train_each_model_at_its_rate(orc):
    """Per-model rates (Section 7's per-model hyper-parameters): each model
    ends exactly where training it alone at its own rate ends."""
    hs, acts, X, y, W1, W2 = _problem(29)
    M = len(hs)
    rates = np.linspace(0.0, 0.4, M)
    batches = [(0, 7), (7, 7)]
    P1, P2, pl = orc.train(hs, acts, W1, W2, X, y, batches, rates)
    off = np.concatenate([[0], np.cumsum(hs)])
    for m in (0, 5, M - 1):
        s = slice(off[m], off[m + 1])
        A1, A2, al = orc.train(hs[m:m + 1], acts[m:m + 1], W1[s], W2[:, s], X, y, batches, rates[m])
        assert np.array_equal(P1[s], A1) and np.array_equal(P2[:, s], A2) and pl[m] == al[0]
    assert np.array_equal(P1[off[0]:off[1]], W1[off[0]:off[1]])      # rate 0: unchanged
    with pytest.raises(ValueError):
        orc.train(hs, acts, W1, W2, X, y, batches, rates[:-1])
