"""CPU oracle for ParallelMLPs training (fp64, plain C + OpenMP).

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and
the benchmark's CPU-baseline leg, never by the product package.  The oracle
trains every MLP on its own with ordinary matrix products, which is the
result the packed method of Section 3 is constructed to reproduce exactly.

`build()` compiles `pmlp_oracle.c` with gcc into `liboracle.so` next to
this file; the wrappers below only marshal numpy arrays through ctypes.

`head="mse"` (gradients, train, dataset_loss) replaces the softmax
cross-entropy with the mean squared error against real targets y [B, O]
(regression); the default `head="ce"` takes integer labels y [B].

`mask` (forward, gradients, train, hidden, value_ties, dataset_loss) gives
per-model input feature masks [M, F]: model m is trained on its own subset
of the input columns (feature selection); its packed W1 block keeps zeros in
the other columns.

`rounding="bf16"` (forward, gradients, train, hidden, dataset_loss) emulates
the bf16-in / fp32-accumulate variant of the two input-layer products: X,
W1 and dZ go to fp32 and then to the nearest bfloat16 before they are
multiplied; all other arithmetic stays fp64.  `rounding="bf16_store"` is
that variant with Z also kept in bfloat16: the pre-activation is stored as
the bfloat16 nearest to its fp32 value and the activation, its slope and
everything after them use the stored value; `stored_z` (forward, gradients,
train, hidden) gives the checked result's stored Z [rows, N] so that, where
two stored values are correct (a rounding midpoint within `zband` times
the size of the terms of Z), the oracle takes the checked one (see
orc_set_stored_z in pmlp_oracle.c; stored_z_conflicts counts the rest).
"""
from __future__ import annotations

import contextlib
import ctypes as C
import os
import subprocess
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pmlp_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle (plain -O2, no target-specific tuning)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
               "-ffp-contract=off", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = C.CDLL(_LIB)
        P = C.c_void_p
        i32, i64, u64, dbl = C.c_int32, C.c_int64, C.c_uint64, C.c_double
        lib.orc_splitmix64.restype = u64
        lib.orc_splitmix64.argtypes = [u64]
        lib.orc_act.restype = dbl
        lib.orc_act.argtypes = [C.c_int, dbl]
        lib.orc_act_deriv.restype = dbl
        lib.orc_act_deriv.argtypes = [C.c_int, dbl]
        lib.orc_max_threads.restype = C.c_int
        lib.orc_init_params.restype = C.c_int
        lib.orc_init_params.argtypes = [i32, i32, i32, P, u64, P, P]
        lib.orc_init_biases.restype = C.c_int
        lib.orc_init_biases.argtypes = [i32, i32, i32, P, u64, P, P]
        lib.orc_forward.restype = C.c_int
        lib.orc_forward.argtypes = [i32, i32, i32, P, P, P, P, P, P, P, i32, P, C.c_int]
        lib.orc_gradients.restype = C.c_int
        lib.orc_gradients.argtypes = [i32, i32, i32, P, P, P, P, P, P, P, P, i32,
                                      P, P, P, P, P, P, P, dbl, dbl, dbl, C.c_int]
        lib.orc_train.restype = C.c_int
        lib.orc_train.argtypes = [i32, i32, i32, P, P, P, P, P, P, P, P, i32, P, P,
                                  dbl, P, P, P, P, P, P, P, i32, P, dbl, C.c_int]
        lib.orc_hidden.restype = C.c_int
        lib.orc_hidden.argtypes = [i32, i32, P, P, P, P, P, i32, P, P]
        lib.orc_set_input_rounding.restype = C.c_int
        lib.orc_set_input_rounding.argtypes = [C.c_int]
        lib.orc_bf16.restype = C.c_float
        lib.orc_bf16.argtypes = [C.c_float]
        lib.orc_bf16_array.restype = None
        lib.orc_bf16_array.argtypes = [P, P, i64]
        lib.orc_value_ties.restype = C.c_int
        lib.orc_value_ties.argtypes = [i32, i32, P, P, P, P, P, i32, dbl, P]
        lib.orc_set_head.restype = C.c_int
        lib.orc_set_head.argtypes = [C.c_int]
        lib.orc_set_branch.restype = C.c_int
        lib.orc_set_branch.argtypes = [P, i64, dbl]
        lib.orc_branch_conflicts.restype = i64
        lib.orc_branch_conflicts.argtypes = []
        lib.orc_set_stored_z.restype = C.c_int
        lib.orc_set_stored_z.argtypes = [P, i64, dbl]
        lib.orc_stored_z_conflicts.restype = i64
        lib.orc_stored_z_conflicts.argtypes = []
        lib.orc_set_feature_mask.restype = C.c_int
        lib.orc_set_feature_mask.argtypes = [P]
        lib.orc_dataset_loss.restype = C.c_int
        lib.orc_dataset_loss.argtypes = [i32, i32, i32, P, P, P, P, P, P, P, P, i64,
                                         i32, P, C.c_int]
        _lib = lib
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _c(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


def _bias(b, n: int, what: str):
    if b is None:
        return None
    a = _c(b, np.float64).reshape(-1)
    if a.size != n:
        raise ValueError("%s needs %d entries" % (what, n))
    return a


def _check(rc: int, what: str):
    if rc != 0:
        raise RuntimeError("oracle %s failed with code %d" % (what, rc))


_ROUNDING = {"exact": 0, "bf16": 1, "bf16_store": 2}


@contextlib.contextmanager
def _rounding(mode: str):
    if mode not in _ROUNDING:
        raise ValueError("rounding must be one of %s" % sorted(_ROUNDING))
    lib = _load()
    _check(lib.orc_set_input_rounding(_ROUNDING[mode]), "set_input_rounding")
    try:
        yield
    finally:
        lib.orc_set_input_rounding(0)


_HEADS = {"ce": 0, "mse": 1}


@contextlib.contextmanager
def _head(head: str):
    if head not in _HEADS:
        raise ValueError("head must be one of %s" % sorted(_HEADS))
    lib = _load()
    _check(lib.orc_set_head(_HEADS[head]), "set_head")
    try:
        yield
    finally:
        lib.orc_set_head(0)


_last_conflicts = 0


@contextlib.contextmanager
def _branch(br, band: float, N: int):
    """Branch choices at Hardshrink's jumps for the duration of one call
    (see orc_set_branch in pmlp_oracle.c): br is [rows, N] with nonzero
    where the checked result let the value pass; None gives none."""
    global _last_conflicts
    lib = _load()
    a = None
    if br is not None:
        a = np.ascontiguousarray(np.asarray(br) != 0, dtype=np.uint8)
        if a.ndim != 2 or a.shape[1] != N:
            raise ValueError("branch choices must be [rows, %d]" % N)
    _check(lib.orc_set_branch(_p(a), 0 if a is None else N, float(band)), "set_branch")
    try:
        yield
    finally:
        _last_conflicts = int(lib.orc_branch_conflicts())
        lib.orc_set_branch(None, 0, 0.0)


_last_z_conflicts = 0


@contextlib.contextmanager
def _stored_z(zs, band: float, N: int):
    """Stored-Z choices of the bf16 storage variant for the duration of one
    call (see orc_set_stored_z in pmlp_oracle.c): zs is [rows, N] fp32, the
    stored Z of the checked result; None gives none."""
    global _last_z_conflicts
    lib = _load()
    a = None
    if zs is not None:
        a = np.ascontiguousarray(zs, dtype=np.float32)
        if a.ndim != 2 or a.shape[1] != N:
            raise ValueError("stored Z must be [rows, %d]" % N)
    _check(lib.orc_set_stored_z(_p(a), 0 if a is None else N, float(band)), "set_stored_z")
    try:
        yield
    finally:
        _last_z_conflicts = int(lib.orc_stored_z_conflicts())
        lib.orc_set_stored_z(None, 0, 0.0)


def stored_z_conflicts() -> int:
    """Number of (sample, unit) pairs in the last call given stored Z where
    the given value is not among the correct stored values (it kept its
    own there)."""
    return _last_z_conflicts


@contextlib.contextmanager
def _fmask(mask, M: int, F: int):
    """Per-model input feature masks [M, F] for the duration of one call
    (nonzero: model m sees feature f; see orc_set_feature_mask in
    pmlp_oracle.c); None: every model sees every feature."""
    lib = _load()
    a = None
    if mask is not None:
        a = np.ascontiguousarray(np.asarray(mask) != 0, dtype=np.uint8)
        if a.shape != (M, F):
            raise ValueError("feature masks must be [%d, %d]" % (M, F))
    lib.orc_set_feature_mask(_p(a))
    try:
        yield
    finally:
        lib.orc_set_feature_mask(None)


def branch_conflicts() -> int:
    """Number of (sample, unit) pairs in the last call given branch choices
    where the given side differs from the oracle's own outside the band
    (a choice that is not among the correct results)."""
    return _last_conflicts


def _labels(y, head: str, O: int, S: int) -> np.ndarray:
    """int32 labels [S] (ce) or float32 targets [S, O] (mse)."""
    if head == "mse":
        t = _c(y, np.float32)
        if t.shape != (S, O):
            raise ValueError("mse targets must be [%d, %d]" % (S, O))
        return t
    return _c(y, np.int32)


def bf16_round(x) -> np.ndarray:
    """Nearest bfloat16 (ties to even) of each fp32 value, as fp32."""
    a = _c(x, np.float32)
    out = np.empty_like(a)
    _load().orc_bf16_array(_p(a), _p(out), a.size)
    return out


def splitmix64(state: int) -> int:
    return int(_load().orc_splitmix64(C.c_uint64(state & 0xFFFFFFFFFFFFFFFF)))


def act(act_id: int, z: float) -> float:
    return float(_load().orc_act(act_id, z))


def act_deriv(act_id: int, z: float) -> float:
    return float(_load().orc_act_deriv(act_id, z))


def max_threads() -> int:
    return int(_load().orc_max_threads())


def init_params(F: int, O: int, hidden_sizes, seed: int) -> Tuple[np.ndarray, np.ndarray]:
    hs = _c(hidden_sizes, np.int32)
    N = int(hs.sum())
    W1 = np.empty((N, F), np.float32)
    W2 = np.empty((O, N), np.float32)
    _check(_load().orc_init_params(F, O, len(hs), _p(hs), C.c_uint64(seed), _p(W1), _p(W2)),
           "init_params")
    return W1, W2


def init_biases(F: int, O: int, hidden_sizes, seed: int) -> Tuple[np.ndarray, np.ndarray]:
    """b1 [N] and b2 [M, O] (fp32) from the counter-based stream, tags 3 and 4."""
    hs = _c(hidden_sizes, np.int32)
    b1 = np.empty(int(hs.sum()), np.float32)
    b2 = np.empty((len(hs), O), np.float32)
    _check(_load().orc_init_biases(F, O, len(hs), _p(hs), C.c_uint64(seed), _p(b1), _p(b2)),
           "init_biases")
    return b1, b2


def forward(hidden_sizes, act_ids, W1, W2, X, nthreads: int = 0,
            rounding: str = "exact", b1=None, b2=None, branch=None,
            band: float = 1e-6, mask=None, stored_z=None, zband: float = 1e-6) -> np.ndarray:
    """logits [B, M, O] in fp64; optional biases b1 [N] and b2 [M, O];
    optional branch choices [B, N] at Hardshrink's jumps (see _branch)."""
    hs, ac = _c(hidden_sizes, np.int32), _c(act_ids, np.int32)
    W1d, W2d, Xf = _c(W1, np.float64), _c(W2, np.float64), _c(X, np.float32)
    B, F = Xf.shape
    O, N = W2d.shape
    c1, c2 = _bias(b1, N, "b1"), _bias(b2, len(hs) * O, "b2")
    out = np.empty((B, len(hs), O), np.float64)
    with _rounding(rounding), _branch(branch, band, N), _stored_z(stored_z, zband, N), _fmask(mask, len(hs), F):
        _check(_load().orc_forward(F, O, len(hs), _p(hs), _p(ac), _p(W1d), _p(W2d), _p(c1),
                                   _p(c2), _p(Xf), B, _p(out), nthreads), "forward")
    return out


def gradients(hidden_sizes, act_ids, W1, W2, X, y, kink_rel: float = 1e-6,
              with_allowance: bool = True, nthreads: int = 0, rounding: str = "exact",
              tie_rel: float = 1e-5, cond_rel: float = 2.4e-7, b1=None, b2=None,
              head: str = "ce", branch=None, band: float = 1e-6, mask=None, stored_z=None,
              zband: float = 1e-6):
    """(dW1 [N,F], dW2 [O,N], loss [M], allow_dW1 [N,F] or None) in fp64.

    allow_dW1 bounds what a correct fp32 evaluation may differ by where a
    discrete choice is within rounding of its boundary: the derivative branch
    at a ReLU/LeakyReLU kink (|Z| <= kink_rel * sum_f |x w|) and, with
    rounding="bf16", the bfloat16 neighbour dZ rounds to (fp32 dZ within
    tie_rel * sum_o |G W2| |act'| of a rounding midpoint); and the amplified
    fp32 error of dH = G W2 where its terms cancel more than 16-fold
    (cond_rel, about 4 units in the last fp32 place, times the excess).

    The gradient is that of sum_m L_m, so each model's slice is the gradient
    of its own mean cross-entropy (or, with head="mse", mean squared error).  With biases b1 [N] and b2 [M, O] three more
    items follow: db1 [N], db2 [M, O] and the allowance of db1 [N] (that of a
    weight whose input is fixed at 1)."""
    hs, ac = _c(hidden_sizes, np.int32), _c(act_ids, np.int32)
    W1d, W2d, Xf = _c(W1, np.float64), _c(W2, np.float64), _c(X, np.float32)
    B, F = Xf.shape
    O, N = W2d.shape
    yi = _labels(y, head, O, B)
    dW1 = np.empty((N, F), np.float64)
    dW2 = np.empty((O, N), np.float64)
    loss = np.empty(len(hs), np.float64)
    allow = np.empty((N, F), np.float64) if with_allowance else None
    M = len(hs)
    c1, c2 = _bias(b1, N, "b1"), _bias(b2, M * O, "b2")
    db1 = np.empty(N, np.float64) if c1 is not None else None
    db2 = np.empty((M, O), np.float64) if c2 is not None else None
    allow_b = np.empty(N, np.float64) if (with_allowance and c1 is not None) else None
    with _rounding(rounding), _head(head), _branch(branch, band, N), _stored_z(stored_z, zband, N), _fmask(mask, M, F):
        _check(_load().orc_gradients(F, O, len(hs), _p(hs), _p(ac), _p(W1d), _p(W2d), _p(c1),
                                     _p(c2), _p(Xf), _p(yi), B, _p(dW1), _p(dW2), _p(db1),
                                     _p(db2), _p(loss), _p(allow), _p(allow_b),
                                     float(kink_rel), float(tie_rel), float(cond_rel),
                                     nthreads),
               "gradients")
    if c1 is not None or c2 is not None:
        return dW1, dW2, loss, allow, db1, db2, allow_b
    return dW1, dW2, loss, allow


def train(hidden_sizes, act_ids, W1, W2, X, y, batches: Sequence[Tuple[int, int]],
          lr: float, models: Optional[Sequence[int]] = None, nthreads: int = 0,
          rounding: str = "exact", return_ties: bool = False, tie_rel: float = 1e-6,
          b1=None, b2=None, head: str = "ce", branch=None, band: float = 1e-6, mask=None,
          stored_z=None, zband: float = 1e-6):
    """SGD over the given (offset, length) batches.

    Returns (W1' [N,F], W2' [O,N], loss_last [M]) in fp64.  With a model
    subset, entries of the other models are NaN.  With biases b1 [N] and
    b2 [M, O], the updated b1' and b2' follow loss_last.  lr is one rate for all
    models or an array of M per-model rates.  With return_ties, a fourth
    item counts per model the value ties met during training (Z within
    tie_rel * sum_f |x w| of a jump of the activation, at that step's
    weights; see value_ties)."""
    hs, ac = _c(hidden_sizes, np.int32), _c(act_ids, np.int32)
    W1d, W2d, Xf = _c(W1, np.float64), _c(W2, np.float64), _c(X, np.float32)
    F = Xf.shape[1]
    O, N = W2d.shape
    yi = _labels(y, head, O, Xf.shape[0])
    off = np.asarray([b[0] for b in batches], np.int64)
    ln = np.asarray([b[1] for b in batches], np.int32)
    if len(batches) and (off.min() < 0 or (off + ln).max() > Xf.shape[0]):
        raise ValueError("batch outside the sample arrays")
    W1o = np.full((N, F), np.nan)
    W2o = np.full((O, N), np.nan)
    loss = np.full(len(hs), np.nan)
    sel = None if models is None else _c(models, np.int32)
    ties = np.zeros(len(hs), np.int32) if return_ties else None
    c1, c2 = _bias(b1, N, "b1"), _bias(b2, len(hs) * O, "b2")
    b1o = np.full(N, np.nan) if c1 is not None else None
    b2o = np.full((len(hs), O), np.nan) if c2 is not None else None
    lr_arr = np.asarray(lr, np.float64)
    lr_m = None
    if lr_arr.ndim:
        lr_m = np.ascontiguousarray(lr_arr.reshape(-1))
        if lr_m.size != len(hs):
            raise ValueError("per-model lr needs one rate per model")
        lr = 0.0
    with _rounding(rounding), _head(head), _branch(branch, band, N), _stored_z(stored_z, zband, N), _fmask(mask, len(hs), F):
        _check(_load().orc_train(F, O, len(hs), _p(hs), _p(ac), _p(W1d), _p(W2d), _p(c1),
                                 _p(c2), _p(Xf), _p(yi), len(batches), _p(off), _p(ln),
                                 float(lr), _p(lr_m), _p(W1o), _p(W2o), _p(b1o), _p(b2o),
                                 _p(loss), _p(sel), 0 if sel is None else len(sel),
                                 _p(ties), float(tie_rel), nthreads), "train")
    out = [W1o, W2o, loss]
    if c1 is not None or c2 is not None:
        out += [b1o, b2o]
    if return_ties:
        out.append(ties)
    return tuple(out)


def hidden(hidden_sizes, act_ids, W1, X, rounding: str = "exact", b1=None,
           branch=None, band: float = 1e-6, mask=None, stored_z=None,
           zband: float = 1e-6) -> Tuple[np.ndarray, np.ndarray]:
    """Z = X W1^T and H = act(Z), both [B, N] fp64 (branch: see _branch)."""
    hs, ac = _c(hidden_sizes, np.int32), _c(act_ids, np.int32)
    W1d, Xf = _c(W1, np.float64), _c(X, np.float32)
    B, F = Xf.shape
    N = int(hs.sum())
    Z = np.empty((B, N), np.float64)
    H = np.empty((B, N), np.float64)
    with _rounding(rounding), _branch(branch, band, N), _stored_z(stored_z, zband, N), _fmask(mask, len(hs), F):
        _check(_load().orc_hidden(F, len(hs), _p(hs), _p(ac), _p(W1d), _p(_bias(b1, N, "b1")),
                                  _p(Xf), B, _p(Z), _p(H)), "hidden")
    return Z, H


def value_ties(hidden_sizes, act_ids, W1, X, rel: float = 1e-6,
               rounding: str = "exact", b1=None, mask=None) -> np.ndarray:
    """Per-model count of (sample, unit) pairs whose Z sits within rounding
    of a jump of its activation (Hardshrink at +-0.5); models with a nonzero
    count have several correct fp32 results and are left out of comparisons."""
    hs, ac = _c(hidden_sizes, np.int32), _c(act_ids, np.int32)
    W1d, Xf = _c(W1, np.float64), _c(X, np.float32)
    B, F = Xf.shape
    counts = np.empty(len(hs), np.int32)
    with _rounding(rounding), _fmask(mask, len(hs), F):
        c1 = _bias(b1, W1d.shape[0], "b1")
        _check(_load().orc_value_ties(F, len(hs), _p(hs), _p(ac), _p(W1d), _p(c1), _p(Xf), B,
                                      float(rel), _p(counts)), "value_ties")
    return counts


def dataset_loss(hidden_sizes, act_ids, W1, W2, X, y, chunk: int = 1024,
                 nthreads: int = 0, rounding: str = "exact", b1=None,
                 b2=None, head: str = "ce", mask=None) -> np.ndarray:
    hs, ac = _c(hidden_sizes, np.int32), _c(act_ids, np.int32)
    W1d, W2d, Xf = _c(W1, np.float64), _c(W2, np.float64), _c(X, np.float32)
    S, F = Xf.shape
    O = W2d.shape[0]
    yi = _labels(y, head, O, S)
    loss = np.empty(len(hs), np.float64)
    with _rounding(rounding), _head(head), _fmask(mask, len(hs), F):
        c1 = _bias(b1, W2d.shape[1], "b1")
        c2 = _bias(b2, len(hs) * O, "b2")
        _check(_load().orc_dataset_loss(F, O, len(hs), _p(hs), _p(ac), _p(W1d), _p(W2d),
                                        _p(c1), _p(c2), _p(Xf), _p(yi), S, chunk, _p(loss),
                                        nthreads),
               "dataset_loss")
    return loss


# --------------------------------------------------------------------------
# Two hidden layers per model (Section 7, Figure 3).  h1 [M], h2 [M] hidden
# sizes, one activation per model for both layers; packed W1 [N1, F],
# W12 [K] (model m's [h2_m, h1_m] block row-major at offset K_m), W2 [O, N2].
# --------------------------------------------------------------------------

def _deep_lib():
    lib = _load()
    if not getattr(lib, "_deep_ready", False):
        P = C.c_void_p
        i32, u64, dbl = C.c_int32, C.c_uint64, C.c_double
        lib.orc_deep_init.restype = C.c_int
        lib.orc_deep_init.argtypes = [i32, i32, i32, P, P, u64, P, P, P]
        lib.orc_deep_forward_all.restype = C.c_int
        lib.orc_deep_forward_all.argtypes = [i32, i32, i32, P, P, P, P, P, P, P, i32, P, C.c_int]
        lib.orc_deep_gradients.restype = C.c_int
        lib.orc_deep_gradients.argtypes = [i32, i32, i32, P, P, P, P, P, P, P, P, i32, P, P, P,
                                           P, P, P, P, dbl, dbl, dbl, C.c_int]
        lib.orc_deep_train.restype = C.c_int
        lib.orc_deep_train.argtypes = [i32, i32, i32, P, P, P, P, P, P, P, P, i32, P, P, dbl,
                                       P, P, P, P, P, i32, P, dbl, C.c_int]
        lib._deep_ready = True
    return lib


def deep_sizes(h1, h2):
    """(N1, N2, K): units of the two hidden layers and entries of all W12 blocks."""
    a, b = np.asarray(h1, np.int64), np.asarray(h2, np.int64)
    return int(a.sum()), int(b.sum()), int((a * b).sum())


def deep_init(F: int, O: int, h1, h2, seed: int):
    """W1 [N1, F], W12 [K], W2 [O, N2] (fp32) from the counter-based stream:
    tags 1 (W1, fan_in F), 5 (W12, idx K_m + i h1_m + j, fan_in h1_m) and
    2 (W2, idx o N2 + n, fan_in h2_m)."""
    a, b = _c(h1, np.int32), _c(h2, np.int32)
    N1, N2, K = deep_sizes(a, b)
    W1 = np.empty((N1, F), np.float32)
    W12 = np.empty(K, np.float32)
    W2 = np.empty((O, N2), np.float32)
    _check(_deep_lib().orc_deep_init(F, O, len(a), _p(a), _p(b), C.c_uint64(seed), _p(W1),
                                     _p(W12), _p(W2)), "deep_init")
    return W1, W12, W2


def deep_forward(h1, h2, act_ids, W1, W12, W2, X, nthreads: int = 0) -> np.ndarray:
    """logits [B, M, O] in fp64."""
    a, b, ac = _c(h1, np.int32), _c(h2, np.int32), _c(act_ids, np.int32)
    W1d, W12d, W2d, Xf = _c(W1, np.float64), _c(W12, np.float64), _c(W2, np.float64), _c(X, np.float32)
    B, F = Xf.shape
    O = W2d.shape[0]
    out = np.empty((B, len(a), O), np.float64)
    _check(_deep_lib().orc_deep_forward_all(F, O, len(a), _p(a), _p(b), _p(ac), _p(W1d), _p(W12d),
                                            _p(W2d), _p(Xf), B, _p(out), nthreads), "deep_forward")
    return out


def deep_gradients(h1, h2, act_ids, W1, W12, W2, X, y, kink_rel: float = 1e-6,
                   cond_rel: float = 2.4e-7, tie_rel: float = 1e-6, nthreads: int = 0):
    """(dW1 [N1,F], dW12 [K], dW2 [O,N2], loss [M], allow_dW1, allow_dW12,
    ties [M]) in fp64: gradients of sum_m L_m, the allowances of what a
    correct fp32 evaluation may differ by (kink ties of either layer and the
    cancellation of dH2 = G W2), and the count of Hardshrink value ties."""
    a, b, ac = _c(h1, np.int32), _c(h2, np.int32), _c(act_ids, np.int32)
    W1d, W12d, W2d, Xf = _c(W1, np.float64), _c(W12, np.float64), _c(W2, np.float64), _c(X, np.float32)
    B, F = Xf.shape
    O = W2d.shape[0]
    N1, N2, K = deep_sizes(a, b)
    yi = _c(y, np.int32)
    dW1, dW12, dW2 = np.empty((N1, F)), np.empty(K), np.empty((O, N2))
    loss = np.empty(len(a))
    al1, al12 = np.empty((N1, F)), np.empty(K)
    ties = np.empty(len(a), np.int32)
    _check(_deep_lib().orc_deep_gradients(F, O, len(a), _p(a), _p(b), _p(ac), _p(W1d), _p(W12d),
                                          _p(W2d), _p(Xf), _p(yi), B, _p(dW1), _p(dW12), _p(dW2),
                                          _p(loss), _p(al1), _p(al12), _p(ties), float(kink_rel),
                                          float(cond_rel), float(tie_rel), nthreads),
           "deep_gradients")
    return dW1, dW12, dW2, loss, al1, al12, ties


def deep_train(h1, h2, act_ids, W1, W12, W2, X, y, batches, lr: float, models=None,
               tie_rel: float = 1e-6, nthreads: int = 0):
    """SGD over the (offset, length) batches: (W1', W12', W2', loss_last [M],
    ties [M]) in fp64; with a model subset the other entries are NaN."""
    a, b, ac = _c(h1, np.int32), _c(h2, np.int32), _c(act_ids, np.int32)
    W1d, W12d, W2d, Xf = _c(W1, np.float64), _c(W12, np.float64), _c(W2, np.float64), _c(X, np.float32)
    F = Xf.shape[1]
    O = W2d.shape[0]
    N1, N2, K = deep_sizes(a, b)
    yi = _c(y, np.int32)
    off = np.asarray([t[0] for t in batches], np.int64)
    ln = np.asarray([t[1] for t in batches], np.int32)
    if len(batches) and (off.min() < 0 or (off + ln).max() > Xf.shape[0]):
        raise ValueError("batch outside the sample arrays")
    W1o, W12o, W2o = np.full((N1, F), np.nan), np.full(K, np.nan), np.full((O, N2), np.nan)
    loss = np.full(len(a), np.nan)
    ties = np.zeros(len(a), np.int32)
    sel = None if models is None else _c(models, np.int32)
    _check(_deep_lib().orc_deep_train(F, O, len(a), _p(a), _p(b), _p(ac), _p(W1d), _p(W12d),
                                      _p(W2d), _p(Xf), _p(yi), len(batches), _p(off), _p(ln),
                                      float(lr), _p(W1o), _p(W12o), _p(W2o), _p(loss), _p(sel),
                                      0 if sel is None else len(sel), _p(ties), float(tie_rel),
                                      nthreads), "deep_train")
    return W1o, W12o, W2o, loss, ties
