"""Pins of the oracle's biases (b1 [N] on the hidden units, b2 [M, O] on the
outputs; Section 3 drops them only to keep the explanation short).

Against textbook affine maps (numpy), closed forms, central finite
differences, the no-bias results, training each model alone, and the
published counter-based initialisation."""
import math

import numpy as np
import pytest


def _problem(seed, M=12, hmax=7, F=5, O=3, B=9):
    rng = np.random.default_rng(seed)
    hs = rng.integers(1, hmax + 1, M).astype(np.int32)
    acts = rng.integers(0, 13, M).astype(np.int32)
    N = int(hs.sum())
    X = rng.standard_normal((B, F)).astype(np.float32)
    y = rng.integers(0, O, B).astype(np.int32)
    W1 = rng.uniform(-0.5, 0.5, (N, F))
    W2 = rng.uniform(-0.5, 0.5, (O, N))
    b1 = rng.uniform(-0.5, 0.5, N)
    b2 = rng.uniform(-0.5, 0.5, (M, O))
    return hs, acts, X, y, W1, W2, b1, b2


def test_identity_model_is_two_affine_maps(orc):
    rng = np.random.default_rng(1)
    F, h, O, B = 4, 6, 3, 8
    X = rng.standard_normal((B, F)).astype(np.float32)
    W1, W2 = rng.standard_normal((h, F)), rng.standard_normal((O, h))
    b1, b2 = rng.standard_normal(h), rng.standard_normal((1, O))
    got = orc.forward([h], [0], W1, W2, X, b1=b1, b2=b2)[:, 0, :]
    want = (X.astype(np.float64) @ W1.T + b1) @ W2.T + b2[0]
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-13)
    Z, _ = orc.hidden([h], [0], W1, X, b1=b1)
    np.testing.assert_allclose(Z, X.astype(np.float64) @ W1.T + b1, rtol=1e-13, atol=1e-13)


def test_zero_biases_equal_no_biases_bitwise(orc):
    hs, acts, X, y, W1, W2, b1, b2 = _problem(2)
    z1, z2 = np.zeros_like(b1), np.zeros_like(b2)
    assert np.array_equal(orc.forward(hs, acts, W1, W2, X),
                          orc.forward(hs, acts, W1, W2, X, b1=z1, b2=z2))
    g = orc.gradients(hs, acts, W1, W2, X, y)
    gb = orc.gradients(hs, acts, W1, W2, X, y, b1=z1, b2=z2)
    for a, b in zip(g[:3], gb[:3]):
        assert np.array_equal(a, b)
    t = orc.train(hs, acts, W1, W2, X, y, [(0, 9)], 0.1)
    tb = orc.train(hs, acts, W1, W2, X, y, [(0, 9)], 0.1, b1=z1, b2=z2)
    for a, b in zip(t, tb[:3]):
        assert np.array_equal(a, b)


def test_db2_closed_form_with_zero_output_weights(orc):
    """W2 = 0, b2 = 0: every model predicts uniformly, G = (1/O - onehot)/B,
    so db2[m, o] = (B/O - #{b: y_b = o}) / B and db1 = 0."""
    hs, acts, X, y, W1, W2, b1, b2 = _problem(3)
    O, B = W2.shape[0], X.shape[0]
    _, _, loss, _, db1, db2, _ = orc.gradients(hs, acts, W1, np.zeros_like(W2), X, y,
                                            b1=b1, b2=np.zeros_like(b2))
    want = (B / O - np.bincount(y, minlength=O)) / B
    np.testing.assert_allclose(db2, np.tile(want, (len(hs), 1)), rtol=0, atol=1e-15)
    assert np.all(db1 == 0.0)
    np.testing.assert_allclose(loss, math.log(O), rtol=1e-14)


def test_bias_gradients_match_finite_differences(orc):
    hs, acts, X, y, W1, W2, b1, b2 = _problem(4, M=13, hmax=3, F=3, O=3, B=5)
    acts = np.arange(13, dtype=np.int32)
    Z, _ = orc.hidden(hs, acts, W1, X, b1=b1)
    unit_act = np.repeat(acts, hs)
    dist = np.where(unit_act == 11, np.abs(np.abs(Z) - 0.5), np.abs(Z))
    assert dist[:, np.isin(unit_act, (1, 5, 10, 11))].min() > 1e-3   # away from kinks
    _, _, _, _, db1, db2, _ = orc.gradients(hs, acts, W1, W2, X, y, b1=b1, b2=b2)

    def total(c1, c2):
        return orc.gradients(hs, acts, W1, W2, X, y, b1=c1, b2=c2, with_allowance=False)[2].sum()

    h = 1e-6
    fd1 = np.array([(total(b1 + h * e, b2) - total(b1 - h * e, b2)) / (2 * h)
                    for e in np.eye(len(b1))])
    fd2 = np.array([(total(b1, b2 + h * e.reshape(b2.shape)) - total(b1, b2 - h * e.reshape(b2.shape)))
                    / (2 * h) for e in np.eye(b2.size)]).reshape(b2.shape)
    assert np.abs(fd1 - db1).max() <= 1e-6 * np.abs(db1).max()
    assert np.abs(fd2 - db2).max() <= 1e-6 * np.abs(db2).max()


def test_training_with_biases_is_each_model_alone(orc):
    hs, acts, X, y, W1, W2, b1, b2 = _problem(5, B=12)
    batches = [(0, 6), (6, 6)]
    rates = np.linspace(0.05, 0.3, len(hs))
    P1, P2, pl, q1, q2 = orc.train(hs, acts, W1, W2, X, y, batches, rates, b1=b1, b2=b2)
    off = np.concatenate([[0], np.cumsum(hs)])
    for m in range(len(hs)):
        s = slice(off[m], off[m + 1])
        A1, A2, al, a1, a2 = orc.train(hs[m:m + 1], acts[m:m + 1], W1[s], W2[:, s], X, y, batches,
                                       rates[m], b1=b1[s], b2=b2[m:m + 1])
        assert np.array_equal(P1[s], A1) and np.array_equal(P2[:, s], A2)
        assert np.array_equal(q1[s], a1) and np.array_equal(q2[m], a2[0]) and pl[m] == al[0]
    # one step is SGD on the bias gradients
    g = orc.gradients(hs, acts, W1, W2, X[:6], y[:6], b1=b1, b2=b2)
    t = orc.train(hs, acts, W1, W2, X, y, batches[:1], 0.2, b1=b1, b2=b2)
    assert np.array_equal(t[3], b1 - 0.2 * g[4]) and np.array_equal(t[4], b2 - 0.2 * g[5])


def test_bias_init_follows_counter_definition(orc):
    hs = np.array([3, 1, 4], np.int32)
    F, O, seed = 6, 2, 99
    b1, b2 = orc.init_biases(F, O, hs, seed)
    key = orc.splitmix64(seed)

    def draw(tag, idx, fan_in):
        r = orc.splitmix64(key ^ (tag << 60) ^ idx)
        u = (r >> 40) / float(1 << 24)
        return np.float32(2.0 * u - 1.0) * np.float32(1.0 / math.sqrt(fan_in))

    for n in range(int(hs.sum())):
        assert b1[n] == draw(3, n, F)
    for m in range(3):
        for o in range(O):
            assert b2[m, o] == draw(4, m * O + o, hs[m])


def test_bf16_mode_treats_b1_as_a_weight_of_a_constant_input(orc):
    """In the bf16 operand mode, b1 is the weight of an input fixed at 1: the
    results equal those of the no-bias network with X extended by a column
    of ones and W1 by the column b1."""
    hs, acts, X, y, W1, W2, b1, b2 = _problem(6)
    Xe = np.concatenate([X, np.ones((X.shape[0], 1), np.float32)], axis=1)
    W1e = np.concatenate([W1, b1[:, None]], axis=1)
    for rnd in ("exact", "bf16"):
        got = orc.forward(hs, acts, W1, W2, X, b1=b1, b2=b2, rounding=rnd)
        want = orc.forward(hs, acts, W1e, W2, Xe, rounding=rnd) + b2[None]
        np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-13)
        g = orc.gradients(hs, acts, W1, W2, X, y, b1=b1, b2=b2, rounding=rnd)
        # the extended net's W1 gradient holds db1 in its last column (b2 adds
        # the same shift to every logit of a model in both nets only when b2 = 0)
        ge = orc.gradients(hs, acts, W1e, W2, Xe, y, rounding=rnd)
        gz = orc.gradients(hs, acts, W1, W2, X, y, b1=b1, b2=np.zeros_like(b2), rounding=rnd)
        np.testing.assert_allclose(gz[0], ge[0][:, :-1], rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(gz[4], ge[0][:, -1], rtol=1e-12, atol=1e-15)
        assert g[4].shape == b1.shape


def test_db1_allowance_is_that_of_a_constant_input(orc):
    """The allowance of db1 equals the dW1 allowance of the extra column of
    an equivalent network whose input carries a column of ones (b2 = 0)."""
    rng = np.random.default_rng(8)
    hs, acts, X, y, W1, W2, b1, b2 = _problem(8, M=6, hmax=5, F=3, O=2, B=6)
    acts = np.array([1, 5, 10, 11, 1, 5], np.int32)
    X[0] = [1.0, 1.0, 1.0]
    W1[:, :] = 0.1
    b1[:] = -0.3                      # Z[0] = 0 on every unit: kinks at 0 are hit
    Xe = np.concatenate([X, np.ones((6, 1), np.float32)], axis=1)
    W1e = np.concatenate([W1, b1[:, None]], axis=1)
    g = orc.gradients(hs, acts, W1, W2, X, y, b1=b1, b2=np.zeros_like(b2))
    ge = orc.gradients(hs, acts, W1e, W2, Xe, y)
    np.testing.assert_allclose(g[6], ge[3][:, -1], rtol=1e-12, atol=1e-18)
    assert g[6].max() > 0
