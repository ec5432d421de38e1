"""Pins of the oracle's bf16 storage mode (`rounding="bf16_store"`): the
bf16 operand variant with the hidden pre-activation Z also kept in
bfloat16, as the bf16 end-to-end storage variant of the packed network keeps
it between the forward product and the kernels that read it (the memory
remark of Section 5).

Z is stored as the nearest-even bfloat16 of its fp32 value, and the
activation, its slope and everything after them use the stored value.  The
mode is checked against textbook numpy products of values rounded by
PyTorch (not by the oracle), so that rounding Z in the wrong place (before
fp32, after the activation, only in the forward) or not at all fails a test;
the stored-Z choices are checked on constructed ties whose midpoints are
known exactly.  No GPU needed.
"""
import numpy as np
import pytest
import torch


def _torch_bf16(x):
    """Nearest-even bfloat16 of fp32 values, by PyTorch (not the oracle)."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def _problem(seed, hs, acts, F=13, O=3, B=9):
    rng = np.random.default_rng(seed)
    N = int(sum(hs))
    W1 = rng.uniform(-0.5, 0.5, (N, F)).astype(np.float32)
    W2 = rng.uniform(-0.5, 0.5, (O, N)).astype(np.float32)
    X = rng.standard_normal((B, F)).astype(np.float32)
    y = rng.integers(0, O, B).astype(np.int32)
    return np.asarray(hs, np.int32), np.asarray(acts, np.int32), W1, W2, X, y


def _softmax_grad(L, y):
    B = L.shape[0]
    P = np.exp(L - L.max(axis=1, keepdims=True))
    P /= P.sum(axis=1, keepdims=True)
    loss = np.mean(-np.log(P[np.arange(B), y]))
    G = P.copy()
    G[np.arange(B), y] -= 1.0
    return loss, G / B


def _stored(Z):
    """Z as the storage variant keeps it: fp64 -> fp32 -> bfloat16."""
    return _torch_bf16(Z.astype(np.float32)).astype(np.float64)


def test_hidden_is_the_bf16_of_the_fp32_pre_activation(orc):
    hs, acts, W1, W2, X, y = _problem(31, [3, 6, 2, 9], [1, 2, 3, 6], F=29, B=17)
    Z, H = orc.hidden(hs, acts, W1, X, rounding="bf16_store")
    Zb, _ = orc.hidden(hs, acts, W1, X, rounding="bf16")
    assert np.array_equal(Z, _stored(Zb))
    # the activation sees the stored value: relu and tanh columns by hand
    off = np.concatenate([[0], np.cumsum(hs)])
    relu = slice(off[0], off[1])
    tanh = slice(off[1], off[2])
    assert np.array_equal(H[:, relu], np.maximum(Z[:, relu], 0.0))
    assert np.allclose(H[:, tanh], np.tanh(Z[:, tanh]), rtol=1e-15, atol=0)
    # and storing changes Z (the rounding is live)
    assert not np.array_equal(Z, Zb)


@pytest.mark.parametrize("act_id", [0, 2])
def test_gradients_textbook_single_model(orc, act_id):
    """M = 1 with identity or tanh: X and W1 rounded, Z stored in bf16, the
    slope taken at the stored Z, dZ rounded before the dW1 product."""
    hs, acts, W1, W2, X, y = _problem(41 + act_id, [11], [act_id], F=17, O=4, B=23)
    Xr = _torch_bf16(X).astype(np.float64)
    W1r = _torch_bf16(W1).astype(np.float64)
    Zs = _stored(Xr @ W1r.T)
    H = Zs if act_id == 0 else np.tanh(Zs)
    dact = np.ones_like(Zs) if act_id == 0 else 1.0 - np.tanh(Zs) ** 2
    L = H @ W2.astype(np.float64).T
    loss, G = _softmax_grad(L, y)
    dZ = (G @ W2.astype(np.float64)) * dact
    dW1 = _torch_bf16(dZ.astype(np.float32)).astype(np.float64).T @ Xr
    dW2 = G.T @ H
    got = orc.forward(hs, acts, W1, W2, X, rounding="bf16_store")
    assert np.max(np.abs(got[:, 0, :] - L)) <= 1e-12 * np.max(np.abs(L))
    g1, g2, gl, _ = orc.gradients(hs, acts, W1, W2, X, y, rounding="bf16_store")
    assert abs(gl[0] - loss) <= 1e-12 * abs(loss)
    assert np.max(np.abs(g1 - dW1)) <= 1e-12 * np.max(np.abs(dW1))
    assert np.max(np.abs(g2 - dW2)) <= 1e-12 * np.max(np.abs(dW2))
    if act_id == 2:
        # the slope at the unstored Z differs: the backward must use the stored one
        Zb = Xr @ W1r.T
        dZ_other = (G @ W2.astype(np.float64)) * (1.0 - np.tanh(Zb) ** 2)
        other = _torch_bf16(dZ_other.astype(np.float32)).astype(np.float64).T @ Xr
        assert np.max(np.abs(other - dW1)) > 1e-6 * np.max(np.abs(dW1))


def test_exactly_representable_z_reduces_to_the_operand_mode(orc):
    """Small-integer inputs and weights give Z that bfloat16 holds exactly:
    the storage mode then equals the operand mode bit for bit."""
    rng = np.random.default_rng(5)
    hs = np.asarray([4, 2, 7], np.int32)
    acts = np.asarray([1, 4, 2], np.int32)
    X = rng.integers(-2, 3, (10, 6)).astype(np.float32)
    W1 = rng.integers(-1, 2, (13, 6)).astype(np.float64)
    W2 = rng.uniform(-0.5, 0.5, (2, 13))
    y = rng.integers(0, 2, 10).astype(np.int32)
    for fn in (lambda r: orc.forward(hs, acts, W1, W2, X, rounding=r),
               lambda r: orc.gradients(hs, acts, W1, W2, X, y, rounding=r)[:3]):
        a, b = fn("bf16"), fn("bf16_store")
        for u, v in zip(a if isinstance(a, tuple) else [a], b if isinstance(b, tuple) else [b]):
            assert np.array_equal(u, v)


def test_train_is_sgd_on_stored_z_gradients(orc):
    hs, acts, W1, W2, X, y = _problem(9, [3, 5, 2, 8], [1, 3, 6, 9], F=21, O=2, B=12)
    lr = 0.3
    W1a, W2a, la = orc.train(hs, acts, W1, W2, np.concatenate([X, X]), np.concatenate([y, y]),
                             [(0, 12), (12, 12)], lr, rounding="bf16_store")
    g1, g2, _, _ = orc.gradients(hs, acts, W1, W2, X, y, rounding="bf16_store")
    W1b = W1.astype(np.float64) - lr * g1
    W2b = W2.astype(np.float64) - lr * g2
    h1, h2, lb, _ = orc.gradients(hs, acts, W1b, W2b, X, y, rounding="bf16_store")
    assert np.array_equal(la, lb)
    assert np.array_equal(W1a, W1b - lr * h1)
    assert np.array_equal(W2a, W2b - lr * h2)


def test_stored_z_choice_is_taken_only_inside_the_band(orc):
    # the operand rounding applies to W1 itself, so the tie is put into Z
    # as a sum of weights that are bfloat16 already
    hs = np.asarray([1], np.int32)
    acts = np.asarray([0], np.int32)
    for delta, inside in ((2.0 ** -23, True), (2.0 ** -12, False)):
        # Z = 1 + 2^-8 + delta from three features whose weights bfloat16
        # holds exactly (2^-8 + delta itself does not fit in 8 bits)
        X3 = np.ones((1, 3), np.float32)
        W1 = np.asarray([[1.0, 2.0 ** -8, delta]], np.float64)
        assert np.array_equal(_torch_bf16(W1.astype(np.float32)), W1.astype(np.float32))
        Z, _ = orc.hidden(hs, acts, W1, X3, rounding="bf16_store")
        own = Z[0, 0]
        assert own == 1.0 + 2.0 ** -7                     # above the midpoint: rounds up
        lower = np.asarray([[1.0]], np.float32)            # the other neighbour
        Zc, _ = orc.hidden(hs, acts, W1, X3, rounding="bf16_store", stored_z=lower)
        if inside:
            assert Zc[0, 0] == 1.0 and orc.stored_z_conflicts() == 0
        else:
            assert Zc[0, 0] == own and orc.stored_z_conflicts() == 1
        # a value two units away is never taken
        far = np.asarray([[1.0 + 2.0 ** -6]], np.float32)
        Zf, _ = orc.hidden(hs, acts, W1, X3, rounding="bf16_store", stored_z=far)
        assert Zf[0, 0] == own and orc.stored_z_conflicts() == 1
        # the own value as the choice: no conflict, same result
        Zo, _ = orc.hidden(hs, acts, W1, X3, rounding="bf16_store",
                           stored_z=np.asarray([[own]], np.float32))
        assert Zo[0, 0] == own and orc.stored_z_conflicts() == 0


def test_stored_z_choice_propagates_through_the_step(orc):
    """A taken choice changes the activation, the logits, the slope and
    both gradients exactly as the textbook step on the chosen value."""
    hs = np.asarray([1], np.int32)
    acts = np.asarray([2], np.int32)   # tanh
    X = np.ones((1, 3), np.float32)
    W1 = np.asarray([[1.0, 2.0 ** -8, 2.0 ** -23]], np.float64)
    W2 = np.asarray([[0.7], [-0.4]], np.float64)
    y = np.asarray([1], np.int32)
    choice = np.asarray([[1.0]], np.float32)
    g1, g2, gl, _ = orc.gradients(hs, acts, W1, W2, X, y, rounding="bf16_store",
                                  stored_z=choice)
    assert orc.stored_z_conflicts() == 0
    zs = 1.0
    L = (np.tanh(zs) * W2[:, 0])[None, :]
    loss, G = _softmax_grad(L, y)
    dZ = (G @ W2) * (1.0 - np.tanh(zs) ** 2)
    dW1 = _torch_bf16(dZ.astype(np.float32)).astype(np.float64).T @ np.ones((1, 3))
    assert abs(gl[0] - loss) <= 1e-15
    assert np.allclose(g1, dW1, rtol=1e-14, atol=0)
    assert np.allclose(g2, G.T * np.tanh(zs), rtol=1e-14, atol=0)


def test_stored_z_mode_does_not_leak(orc):
    hs, acts, W1, W2, X, y = _problem(13, [4, 6], [2, 7])
    exact = orc.forward(hs, acts, W1, W2, X)
    Z, _ = orc.hidden(hs, acts, W1, X, rounding="bf16_store")
    orc.forward(hs, acts, W1, W2, X, rounding="bf16_store", stored_z=Z.astype(np.float32))
    assert np.array_equal(orc.forward(hs, acts, W1, W2, X), exact)
    with pytest.raises(ValueError):
        orc.hidden(hs, acts, W1, X, rounding="bf16_store", stored_z=np.zeros((9, 3), np.float32))


def test_stored_z_choice_under_cancellation(orc):
    """Z = 2 - 2 + 2^-20 (terms of size 4): every bfloat16 whose rounding
    interval comes within band * 4 of Z is a correct stored value, here
    also one two units of 2^-27 away, as long as the band reaches it."""
    hs = np.asarray([1], np.int32)
    acts = np.asarray([0], np.int32)
    X = np.ones((1, 3), np.float32)
    W1 = np.asarray([[2.0, -2.0, 2.0 ** -20]], np.float64)
    Z, _ = orc.hidden(hs, acts, W1, X, rounding="bf16_store")
    assert Z[0, 0] == 2.0 ** -20
    two_away = np.asarray([[2.0 ** -20 + 2.0 ** -26]], np.float32)   # two bfloat16 units up
    # its rounding interval starts 2^-26 - 2^-28 = 1.1e-8 above Z
    Zc, _ = orc.hidden(hs, acts, W1, X, rounding="bf16_store", stored_z=two_away, zband=1e-6)
    assert Zc[0, 0] == two_away[0, 0] and orc.stored_z_conflicts() == 0
    Zn, _ = orc.hidden(hs, acts, W1, X, rounding="bf16_store", stored_z=two_away, zband=1e-9)
    assert Zn[0, 0] == 2.0 ** -20 and orc.stored_z_conflicts() == 1
    # a value that is not a bfloat16 is never taken
    odd = np.asarray([[2.0 ** -20 * (1 + 2.0 ** -12)]], np.float32)
    Zo, _ = orc.hidden(hs, acts, W1, X, rounding="bf16_store", stored_z=odd, zband=1e-6)
    assert Zo[0, 0] == 2.0 ** -20 and orc.stored_z_conflicts() == 1
