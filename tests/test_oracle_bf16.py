"""Pins of the oracle's bf16 operand-rounding mode (the bf16-in / fp32-
accumulate variant of the two input-layer products).

The rounding itself is checked against PyTorch's CPU float32 -> bfloat16
conversion and against hand-worked ties; the mode is checked against
textbook products (numpy matmuls) of operands rounded by PyTorch, so that
rounding the wrong operand, rounding the product, or dropping the rounding
of dZ each fail a test.  No GPU needed.
"""
import numpy as np
import pytest
import torch

import pmlp_workloads as wl


def _torch_bf16(x):
    """Nearest-even bfloat16 of fp32 values, by PyTorch (not the oracle)."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def test_bf16_rounding_matches_torch(orc):
    rng = np.random.default_rng(11)
    parts = [
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(5000) * 1e-30).astype(np.float32),
        (rng.standard_normal(5000) * 1e30).astype(np.float32),
        # every fp32 whose low 16 bits sit at or next to the rounding midpoint
        (np.arange(4096, dtype=np.uint32) << 16 | 0x8000).view(np.float32),
        (np.arange(4096, dtype=np.uint32) << 16 | 0x7FFF).view(np.float32),
        (np.arange(4096, dtype=np.uint32) << 16 | 0x8001).view(np.float32),
        np.array([0.0, -0.0, 1e-45, -1e-45, 1.1754942e-38, 3.3895314e38, 3.39e38,
                  3.4028235e38, np.inf, -np.inf], np.float32),
    ]
    x = np.concatenate(parts)
    mine = orc.bf16_round(x)
    ref = _torch_bf16(x)
    assert np.array_equal(mine.view(np.uint32), ref.view(np.uint32))
    nan = orc.bf16_round(np.array([np.nan, -np.nan], np.float32))
    assert np.isnan(nan).all()


def test_bf16_ties_go_to_even(orc):
    # bfloat16 keeps 8 significant bits: the ulp of [1, 2) is 2^-7
    x = np.array([1 + 2.0 ** -8,            # tie, kept part even -> down
                  1 + 3 * 2.0 ** -8,        # tie, kept part odd -> up to 1 + 2^-6
                  1 + 2.0 ** -8 + 2.0 ** -20,  # above the tie -> up
                  -(1 + 2.0 ** -8),
                  255.5, 256.5, 257.0], np.float32)
    want = np.array([1.0, 1 + 2.0 ** -6, 1 + 2.0 ** -7, -1.0, 256.0, 256.0, 256.0],
                    np.float32)
    assert np.array_equal(orc.bf16_round(x), want)


def _problem(seed, hs, acts, F=13, O=3, B=9):
    rng = np.random.default_rng(seed)
    N = int(sum(hs))
    W1 = rng.uniform(-0.5, 0.5, (N, F)).astype(np.float32)
    W2 = rng.uniform(-0.5, 0.5, (O, N)).astype(np.float32)
    X = rng.standard_normal((B, F)).astype(np.float32)
    y = rng.integers(0, O, B).astype(np.int32)
    return np.asarray(hs, np.int32), np.asarray(acts, np.int32), W1, W2, X, y


def test_bf16_forward_is_exact_forward_of_rounded_inputs(orc):
    hs, acts, W1, W2, X, y = _problem(3, [1, 4, 7, 2, 9, 3, 5, 6, 8, 2], list(range(10)))
    got = orc.forward(hs, acts, W1, W2, X, rounding="bf16")
    want = orc.forward(hs, acts, _torch_bf16(W1), W2, _torch_bf16(X))
    assert np.array_equal(got, want)
    # W2 and the hidden activations are not rounded: rounding W2 changes the result
    other = orc.forward(hs, acts, _torch_bf16(W1), _torch_bf16(W2), _torch_bf16(X))
    assert not np.array_equal(got, other)
    Z, H = orc.hidden(hs, acts, W1, X, rounding="bf16")
    Z0, H0 = orc.hidden(hs, acts, _torch_bf16(W1), _torch_bf16(X))
    assert np.array_equal(Z, Z0) and np.array_equal(H, H0)


def _softmax_grad(L, y):
    B = L.shape[0]
    P = np.exp(L - L.max(axis=1, keepdims=True))
    P /= P.sum(axis=1, keepdims=True)
    loss = np.mean(-np.log(P[np.arange(B), y]))
    G = P.copy()
    G[np.arange(B), y] -= 1.0
    return loss, G / B


@pytest.mark.parametrize("act_id", [0, 2])
def test_bf16_gradients_textbook_single_model(orc, act_id):
    """M = 1 with identity or tanh: the whole step is three matmuls, one
    softmax and a closed-form derivative, with X, W1 and dZ rounded by
    PyTorch to bfloat16 before the two input-layer products."""
    hs, acts, W1, W2, X, y = _problem(5 + act_id, [11], [act_id], F=17, O=4, B=23)
    Xr = _torch_bf16(X).astype(np.float64)
    W1r = _torch_bf16(W1).astype(np.float64)
    Z = Xr @ W1r.T
    H = Z if act_id == 0 else np.tanh(Z)
    dact = np.ones_like(Z) if act_id == 0 else 1.0 - np.tanh(Z) ** 2
    L = H @ W2.astype(np.float64).T
    loss, G = _softmax_grad(L, y)
    dZ = (G @ W2.astype(np.float64)) * dact
    dZr = _torch_bf16(dZ.astype(np.float32)).astype(np.float64)
    dW1 = dZr.T @ Xr
    dW2 = G.T @ H
    g1, g2, gl, _ = orc.gradients(hs, acts, W1, W2, X, y, rounding="bf16")
    assert abs(gl[0] - loss) <= 1e-12 * abs(loss)
    assert np.max(np.abs(g1 - dW1)) <= 1e-12 * np.max(np.abs(dW1))
    assert np.max(np.abs(g2 - dW2)) <= 1e-12 * np.max(np.abs(dW2))
    # without rounding dZ the product differs (the rounding of dZ is live)
    dW1_unrounded = dZ.T @ Xr
    assert np.max(np.abs(dW1_unrounded - dW1)) > 1e-6 * np.max(np.abs(dW1))


def test_bf16_train_is_sgd_on_bf16_gradients(orc):
    hs, acts, W1, W2, X, y = _problem(9, [3, 5, 2, 8], [1, 3, 6, 9], F=21, O=2, B=12)
    lr = 0.3
    W1a, W2a, la = orc.train(hs, acts, W1, W2, np.concatenate([X, X]), np.concatenate([y, y]),
                             [(0, 12), (12, 12)], lr, rounding="bf16")
    g1, g2, _, _ = orc.gradients(hs, acts, W1, W2, X, y, rounding="bf16")
    W1b = W1.astype(np.float64) - lr * g1
    W2b = W2.astype(np.float64) - lr * g2
    h1, h2, lb, _ = orc.gradients(hs, acts, W1b, W2b, X, y, rounding="bf16")
    assert np.array_equal(la, lb)
    assert np.array_equal(W1a, W1b - lr * h1)
    assert np.array_equal(W2a, W2b - lr * h2)


def test_rounding_mode_does_not_leak(orc):
    hs, acts, W1, W2, X, y = _problem(13, [4, 6], [2, 7])
    exact = orc.forward(hs, acts, W1, W2, X)
    orc.forward(hs, acts, W1, W2, X, rounding="bf16")
    assert np.array_equal(orc.forward(hs, acts, W1, W2, X), exact)
    with pytest.raises(ValueError):
        orc.forward(hs, acts, W1, W2, X, rounding="fp8")


def test_bf16_loss_close_to_exact_loss(orc):
    """The variant changes a one-epoch loss by far less than the 2e-2
    relative tolerance used for it (F = 50, 8 models)."""
    hs = np.asarray([3, 10, 3, 10, 3, 10, 3, 10], np.int32)
    acts = np.asarray([0, 0, 1, 1, 2, 2, 3, 3], np.int32)
    X, y = wl.make_dataset(50, 2, 800, 1234)
    W1, W2 = orc.init_params(50, 2, hs, 7)
    batches = wl.batch_bounds(800, 64)
    W1e, W2e, _ = orc.train(hs, acts, W1, W2, X, y, batches, 0.05)
    W1b, W2b, _ = orc.train(hs, acts, W1, W2, X, y, batches, 0.05, rounding="bf16")
    le = orc.dataset_loss(hs, acts, W1e, W2e, X, y)
    lb = orc.dataset_loss(hs, acts, W1b, W2b, X, y, rounding="bf16")
    rel = np.abs(lb - le) / np.abs(le)
    assert rel.max() < 2e-2
    assert rel.max() > 0  # the variant is really different


def test_bf16_tie_allowance_covers_the_neighbouring_rounding(orc):
    """M = 1 identity: perturb the exact dZ by up to tie_rel/2 of its term
    magnitude before the bfloat16 rounding (what a correct fp32 evaluation
    may do); the textbook dW1 of the perturbed dZ stays within the
    allowance, and the allowance is zero for all but a few entries."""
    hs, acts, W1, W2, X, y = _problem(21, [40], [0], F=9, O=2, B=64)
    tie_rel = 1e-5
    Xr = _torch_bf16(X).astype(np.float64)
    Z = Xr @ _torch_bf16(W1).astype(np.float64).T
    _, G = _softmax_grad(Z @ W2.astype(np.float64).T, y)
    dZ = G @ W2.astype(np.float64)
    mag = np.abs(G) @ np.abs(W2.astype(np.float64))
    g1, _, _, allow = orc.gradients(hs, acts, W1, W2, X, y, rounding="bf16", tie_rel=tie_rel,
                                    cond_rel=0.0)
    rng = np.random.default_rng(4)
    flipped = 0
    for trial in range(20):
        pert = dZ + rng.uniform(-0.5, 0.5, dZ.shape) * tie_rel * mag
        dZr = _torch_bf16(pert.astype(np.float32)).astype(np.float64)
        flipped += int(np.sum(dZr != _torch_bf16(dZ.astype(np.float32))))
        dW1 = dZr.T @ Xr
        assert np.all(np.abs(dW1 - g1) <= allow + 1e-12 * np.abs(g1).max())
    assert flipped > 0                       # the perturbation does reach ties
    assert 0 < np.count_nonzero(allow.sum(axis=1)) < 0.5 * allow.shape[0]
