"""Pins of the oracle's regression head (mean squared error against real
targets), CPU only.

The paper states that the packed method serves regression as well as
classification (Section 5); the head used here is the per-model mean
squared error over the batch and the O outputs,
    L_m = 1/(B O) sum_b sum_o (logit[b,m,o] - t[b,o])^2.
Each test checks the oracle against something other than itself: a closed
form, a textbook computation with numpy matrix products, central finite
differences, and the invariants of independent training.
"""
import numpy as np

import pmlp_workloads as wl


def _problem(seed, M=12, hmax=7, F=5, O=3, B=9):
    rng = np.random.default_rng(seed)
    hs, acts = wl.random_models(rng, M, hmax)
    N = int(hs.sum())
    X = rng.standard_normal((B, F)).astype(np.float32)
    T = rng.standard_normal((B, O)).astype(np.float32)
    W1 = rng.uniform(-0.8, 0.8, (N, F))
    W2 = rng.uniform(-0.8, 0.8, (O, N))
    return hs, acts, X, T, W1, W2


def test_zero_output_weights_closed_form(orc):
    hs, acts, X, T, W1, _ = _problem(1)
    B, O = T.shape
    W2 = np.zeros((O, W1.shape[0]))
    dW1, dW2, loss, _ = orc.gradients(hs, acts, W1, W2, X, T, head="mse")
    t = T.astype(np.float64)
    # logits are all zero: every loss is the mean square of the targets
    assert np.allclose(loss, np.mean(t * t), rtol=1e-14, atol=0)
    # no gradient reaches W1 through zero output weights
    assert np.array_equal(dW1, np.zeros_like(dW1))
    # dW2 = G^T H with G = -2 t / (B O), H from the hidden layer
    _, H = orc.hidden(hs, acts, W1, X)
    ref = (-2.0 / (B * O)) * t.T @ H
    assert np.abs(dW2 - ref).max() <= 1e-13 * max(1.0, np.abs(ref).max())


def test_identity_model_loss_is_textbook_mse(orc):
    rng = np.random.default_rng(2)
    F, O, B, h = 6, 4, 11, 5
    X = rng.standard_normal((B, F)).astype(np.float32)
    T = rng.standard_normal((B, O)).astype(np.float32)
    W1 = rng.uniform(-1, 1, (h, F))
    W2 = rng.uniform(-1, 1, (O, h))
    _, _, loss, _ = orc.gradients([h], [0], W1, W2, X, T, head="mse")
    logits = (X.astype(np.float64) @ W1.T) @ W2.T
    ref = np.mean((logits - T.astype(np.float64)) ** 2)
    assert abs(loss[0] - ref) <= 1e-14 * ref


def test_mse_gradients_match_finite_differences(orc):
    rng = np.random.default_rng(7)
    F, O, B = 3, 3, 5
    hs = np.tile(np.array([1, 2, 3], np.int32), 13)
    acts = np.repeat(np.arange(13, dtype=np.int32), 3)
    N = int(hs.sum())
    X = rng.standard_normal((B, F)).astype(np.float32)
    T = rng.standard_normal((B, O)).astype(np.float32)
    W1 = rng.uniform(-1, 1, (N, F))
    W2 = rng.uniform(-1, 1, (O, N))
    dW1, dW2, _, _ = orc.gradients(hs, acts, W1, W2, X, T, head="mse")

    def total(a, b):
        return orc.gradients(hs, acts, a, b, X, T, with_allowance=False, head="mse")[2].sum()

    eps = 1e-6
    Z = X.astype(np.float64) @ W1.T
    mid = np.repeat(np.arange(len(hs)), hs)
    # away from the ReLU / LeakyReLU / SELU kink at 0 and Hardshrink's jumps at +-0.5
    kinky = ((np.isin(acts[mid], [1, 5, 10]) & (np.abs(Z).min(axis=0) < 1e-4)) |
             ((acts[mid] == 11) & (np.abs(np.abs(Z) - 0.5).min(axis=0) < 1e-4)))
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


def test_mse_perturbing_one_model_leaves_the_others_bitwise(orc):
    hs, acts, X, T, W1, W2 = _problem(3)
    off = np.concatenate([[0], np.cumsum(hs)])
    a = orc.gradients(hs, acts, W1, W2, X, T, head="mse")
    j = 4
    P1, P2 = W1.copy(), W2.copy()
    P1[off[j]:off[j + 1]] *= 1.7
    P2[:, off[j]:off[j + 1]] += 0.3
    b = orc.gradients(hs, acts, P1, P2, X, T, head="mse")
    keep = np.ones(len(hs), bool)
    keep[j] = False
    rows = np.repeat(keep, hs)
    assert np.array_equal(a[2][keep], b[2][keep])
    assert np.array_equal(a[0][rows], b[0][rows])
    assert np.array_equal(a[1][:, rows], b[1][:, rows])
    assert a[2][j] != b[2][j]


def test_mse_training_is_each_model_alone_and_sgd_on_its_gradients(orc):
    hs, acts, X, T, W1, W2 = _problem(4, B=12)
    off = np.concatenate([[0], np.cumsum(hs)])
    lr = 0.05
    batches = [(0, 7), (7, 5)]
    P1, P2, loss = orc.train(hs, acts, W1, W2, X, T, batches, lr, head="mse")
    for m in (0, 5, 11):
        s = slice(off[m], off[m + 1])
        q1, q2, l1 = orc.train(hs[m:m + 1], acts[m:m + 1], W1[s], W2[:, s], X, T, batches, lr,
                               head="mse")
        assert np.array_equal(q1, P1[s]) and np.array_equal(q2, P2[:, s])
        assert l1[0] == loss[m]
    # one step is SGD on the gradients of that batch
    g1, g2, l0, _ = orc.gradients(hs, acts, W1, W2, X[:7], T[:7], with_allowance=False,
                                  head="mse")
    S1, S2, ls = orc.train(hs, acts, W1, W2, X, T, [(0, 7)], lr, head="mse")
    assert np.array_equal(S1, W1 - lr * g1) and np.array_equal(S2, W2 - lr * g2)
    assert np.array_equal(ls, l0)


def test_mse_dataset_loss_is_the_batch_mean(orc):
    hs, acts, X, T, W1, W2 = _problem(5, B=20)
    full = orc.dataset_loss(hs, acts, W1, W2, X, T, chunk=6, head="mse")
    _, _, one, _ = orc.gradients(hs, acts, W1, W2, X, T, with_allowance=False, head="mse")
    assert np.allclose(full, one, rtol=1e-13, atol=0)
