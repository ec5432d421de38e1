"""Error metrics shared by the GPU parity tests.

Per-model normwise error of a tensor T (the bar the parity tests use):
    err_m(T) = max_i |g_i - r_i| / max_i |r_i|   over model m's slice of T,
with g the GPU value and r the oracle's fp64 value.  Elementwise relative
error is not used: cancellation makes it meaningless for small entries.
For dW1 an allowance per element (the oracle's bound on what a different
branch choice at a ReLU/LeakyReLU kink can change) is subtracted first.
"""
import numpy as np


def offsets(hs):
    return np.concatenate([[0], np.cumsum(np.asarray(hs, np.int64))])


def _seg_max(v, hs):
    off = offsets(hs)
    return np.maximum.reduceat(v, off[:-1])


def err_rows(g, r, hs, allow=None):
    """Per-model error for arrays whose axis 0 is the hidden unit (W1, dW1)."""
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    N = r.shape[0]
    d = np.abs(g - r)
    if allow is not None:
        d = np.maximum(d - allow, 0.0)
    dn = d.reshape(N, -1).max(axis=1)
    rn = np.abs(r).reshape(N, -1).max(axis=1)
    return _seg_max(dn, hs) / np.maximum(_seg_max(rn, hs), 1e-300)


def err_cols(g, r, hs):
    """Per-model error for [O, N] arrays (W2, dW2)."""
    return err_rows(np.asarray(g).T, np.asarray(r).T, hs)


def err_logits(g, r):
    """Per-model error for [B, M, O] logits."""
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    d = np.abs(g - r).max(axis=(0, 2))
    return d / np.maximum(np.abs(r).max(axis=(0, 2)), 1e-300)


def err_losses(g, r):
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    return np.abs(g - r) / np.maximum(np.abs(r), 1e-300)


def cross_entropy(logits, y):
    """Per-model mean softmax cross-entropy of [B, M, O] logits, fp64."""
    l = np.asarray(logits, np.float64)
    mx = l.max(axis=2, keepdims=True)
    lse = mx[..., 0] + np.log(np.exp(l - mx).sum(axis=2))
    ly = np.take_along_axis(l, np.asarray(y)[:, None, None].repeat(l.shape[1], 1), 2)[..., 0]
    return (lse - ly).mean(axis=0)


def submodel(hs, acts, W1, W2, models):
    """Hidden sizes, activations and weights of a subset of the models, packed
    in the given order (exact stand-in for those models: they are trained
    independently of the rest)."""
    off = offsets(hs)
    rows = np.concatenate([np.arange(off[m], off[m + 1]) for m in models])
    return (np.asarray(hs)[models], np.asarray(acts)[models], W1[rows], W2[:, rows], rows)


def dw2_terms(orc, hs, acts, W1, W2, X, y, **kw):
    """[O, N]: sum_b |G[b,o]| |H[b,n]|, the size of the terms dW2 = G^T H
    sums (oracle values).  dW2 can cancel across samples (a width-1 model
    with two outputs has dW2[1] = -dW2[0], often small), so, as for db2,
    its per-model error is taken relative to this size rather than to
    |dW2|; where nothing cancels the two agree."""
    _, H = orc.hidden(hs, acts, W1, X, **{k: v for k, v in kw.items()
                                          if k in ("rounding", "b1", "mask", "stored_z", "zband")})
    L = orc.forward(hs, acts, W1, W2, X, **kw)
    P = np.exp(L - L.max(axis=2, keepdims=True))
    P /= P.sum(axis=2, keepdims=True)
    G = P.copy()
    G[np.arange(L.shape[0]), :, np.asarray(y)] -= 1.0
    G /= L.shape[0]
    off = offsets(hs)
    mid = np.repeat(np.arange(len(hs)), np.asarray(hs, np.int64))
    Gn = np.abs(G[:, mid, :])               # [B, N, O]: G of each unit's model
    return np.einsum("bno,bn->on", Gn, np.abs(H))


def err_dw2(g, r, hs, terms):
    """Per-model error of dW2 [O, N] relative to the size of its terms."""
    d = np.abs(np.asarray(g, np.float64) - np.asarray(r, np.float64)).max(axis=0)
    return _seg_max(d, hs) / np.maximum(_seg_max(np.asarray(terms).max(axis=0), hs), 1e-300)
