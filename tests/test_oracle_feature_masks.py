"""Pins of the oracle's per-model input feature masks (feature selection,
Section 7: each model may see its own subset of the input features).

A model with mask sel is, by definition, the same model with X[:, sel] as
its whole input.  Pinned against textbook numpy products of the sliced
arrays, against central finite differences, against the unmasked oracle
(an all-ones mask changes nothing) and by the invariants that follow from
the definition: masked inputs are never read, masked weights stay zero,
and a model's result does not depend on the masks of the others.
"""
import numpy as np
import pytest



def _case(seed=3, M=6, F=9, O=3, B=11, hmax=5):
    rng = np.random.default_rng(seed)
    hs = rng.integers(1, hmax + 1, M).astype(np.int32)
    acts = rng.integers(0, 13, M).astype(np.int32)
    N = int(hs.sum())
    X = rng.standard_normal((B, F)).astype(np.float32)
    y = rng.integers(0, O, B).astype(np.int32)
    W1 = rng.uniform(-0.6, 0.6, (N, F))
    W2 = rng.uniform(-0.8, 0.8, (O, N))
    mask = rng.random((M, F)) < 0.6
    mask[0] = True                       # one model sees everything
    mask[1] = False                      # one model sees nothing (Z = 0)
    mask[2, :] = False
    mask[2, 4] = True                    # one model sees a single feature
    return hs, acts, X, y, W1, W2, mask


def test_all_ones_mask_is_no_mask(orc):
    hs, acts, X, y, W1, W2, _ = _case()
    ones = np.ones((len(hs), X.shape[1]), bool)
    for a, b in zip(orc.gradients(hs, acts, W1, W2, X, y, mask=ones),
                    orc.gradients(hs, acts, W1, W2, X, y)):
        np.testing.assert_array_equal(a, b)
    a = orc.train(hs, acts, W1, W2, X, y, [(0, 6), (6, 5)], 0.1, mask=ones)
    b = orc.train(hs, acts, W1, W2, X, y, [(0, 6), (6, 5)], 0.1)
    for u, v in zip(a, b):
        np.testing.assert_array_equal(u, v)


def test_identity_model_on_the_selected_columns(orc):
    """M = 1, identity activation: logits = X_s W1_s^T W2^T and the textbook
    gradients of softmax cross-entropy through two matrix products."""
    rng = np.random.default_rng(8)
    F, O, B, h = 7, 4, 13, 5
    X = rng.standard_normal((B, F)).astype(np.float32)
    y = rng.integers(0, O, B).astype(np.int32)
    W1 = rng.uniform(-1, 1, (h, F))
    W2 = rng.uniform(-1, 1, (O, h))
    sel = np.array([0, 2, 3, 6])
    mask = np.zeros((1, F), bool)
    mask[0, sel] = True
    Xs = X.astype(np.float64)[:, sel]
    H = Xs @ W1[:, sel].T
    L = H @ W2.T
    got = orc.forward([h], [0], W1, W2, X, mask=mask)[:, 0, :]
    np.testing.assert_allclose(got, L, rtol=1e-13)
    P = np.exp(L - L.max(1, keepdims=True))
    P /= P.sum(1, keepdims=True)
    G = (P - np.eye(O)[y]) / B
    want2 = G.T @ H
    want1 = np.zeros((h, F))
    want1[:, sel] = (G @ W2).T @ Xs
    dW1, dW2, loss, _ = orc.gradients([h], [0], W1, W2, X, y, mask=mask)
    np.testing.assert_allclose(dW2, want2, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(dW1, want1, rtol=1e-12, atol=1e-15)
    assert np.all(dW1[:, [1, 4, 5]] == 0.0)
    want_loss = np.mean(np.log(np.exp(L).sum(1)) - L[np.arange(B), y])
    assert loss[0] == pytest.approx(want_loss, rel=1e-13)


def test_gradients_match_finite_differences_with_masks(orc):
    hs, _, X, y, W1, W2, mask = _case(seed=21, M=4, F=6, O=3, B=7, hmax=3)
    acts = np.array([2, 3, 7, 12], np.int32)      # smooth activations
    dW1, dW2, _, _ = orc.gradients(hs, acts, W1, W2, X, y, mask=mask)

    def total(a1, a2):
        return orc.gradients(hs, acts, a1, a2, X, y, mask=mask)[2].sum()

    eps = 1e-6
    rows = np.repeat(np.arange(len(hs)), hs)
    for n in range(W1.shape[0]):
        for f in range(W1.shape[1]):
            if not mask[rows[n], f]:
                assert dW1[n, f] == 0.0
                continue
            p, q = W1.copy(), W1.copy()
            p[n, f] += eps
            q[n, f] -= eps
            fd = (total(p, W2) - total(q, W2)) / (2 * eps)
            assert abs(fd - dW1[n, f]) <= 1e-7 * max(1.0, abs(fd))
    for o in range(W2.shape[0]):
        for n in range(W2.shape[1]):
            p, q = W2.copy(), W2.copy()
            p[o, n] += eps
            q[o, n] -= eps
            fd = (total(W1, p) - total(W1, q)) / (2 * eps)
            assert abs(fd - dW2[o, n]) <= 1e-7 * max(1.0, abs(fd))


def test_masked_inputs_and_weights_are_never_read(orc):
    hs, acts, X, y, W1, W2, mask = _case(seed=5)
    mask[:, 5] = False              # a feature no model reads
    rows = np.repeat(np.arange(len(hs)), hs)
    batches = [(0, 4), (4, 7)]
    a = orc.train(hs, acts, W1, W2, X, y, batches, 0.2, mask=mask)
    X2, W12 = X.copy(), W1.copy()
    X2[:, 5] = 1e6                  # X is shared: change only what no model reads
    W12[~mask[rows]] = 7.5          # masked weights of every model
    b = orc.train(hs, acts, W12, W2, X2, y, batches, 0.2, mask=mask)
    for u, v in zip(a, b):
        np.testing.assert_array_equal(u, v)
    assert np.all(a[0][~mask[rows]] == 0.0)     # masked weights come out zero


def test_each_model_equals_itself_alone_with_its_own_mask(orc):
    hs, acts, X, y, W1, W2, mask = _case(seed=9)
    off = np.concatenate([[0], np.cumsum(hs)])
    g = orc.gradients(hs, acts, W1, W2, X, y, mask=mask)
    for m in range(len(hs)):
        s = slice(off[m], off[m + 1])
        one = orc.gradients(hs[m:m + 1], acts[m:m + 1], W1[s], W2[:, s], X, y,
                            mask=mask[m:m + 1])
        np.testing.assert_array_equal(one[0], g[0][s])
        np.testing.assert_array_equal(one[1], g[1][:, s])
        assert one[2][0] == g[2][m]
    # and on the sliced input, with no mask at all
    m = 4
    sel = np.flatnonzero(mask[m])
    s = slice(off[m], off[m + 1])
    alone = orc.gradients(hs[m:m + 1], acts[m:m + 1], W1[s][:, sel], W2[:, s],
                          X[:, sel], y)
    np.testing.assert_array_equal(alone[0], g[0][s][:, sel])
    np.testing.assert_array_equal(alone[1], g[1][:, s])


def test_model_that_sees_nothing_has_zero_hidden_input(orc):
    hs, acts, X, y, W1, W2, mask = _case(seed=3)
    Z, _ = orc.hidden(hs, acts, W1, X, mask=mask)
    off = np.concatenate([[0], np.cumsum(hs)])
    assert np.all(Z[:, off[1]:off[2]] == 0.0)
    Zfull, _ = orc.hidden(hs, acts, W1, X)
    np.testing.assert_array_equal(Z[:, off[0]:off[1]], Zfull[:, off[0]:off[1]])


def test_dataset_loss_with_masks_is_the_mean_of_batch_losses(orc):
    hs, acts, X, y, W1, W2, mask = _case(seed=12, B=40)
    full = orc.dataset_loss(hs, acts, W1, W2, X, y, chunk=7, mask=mask)
    parts = [orc.gradients(hs, acts, W1, W2, X[s:s + 8], y[s:s + 8], mask=mask)[2] * 8
             for s in range(0, 40, 8)]
    np.testing.assert_allclose(full, np.sum(parts, axis=0) / 40, rtol=1e-12)
