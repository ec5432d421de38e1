"""ParallelMLPs training on AMD MI355X: Python binding of libpmlp.

Every step of the packed training path runs in the HIP kernels of
``libpmlp.so`` (built in-tree by ``paper_2206_08369_amd.build``).  This
module only marshals arguments: the ``pmlp_*`` functions mirror the C ABI
of ``include/pmlp.h`` one to one and take device pointers as integers;
:class:`PackedMLP` adds shape/dtype checks for torch tensors and passes
torch's current HIP stream.  There is no fallback: if the library is not
built, loading it raises.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "PMLP_OK", "PMLP_EINVAL", "PMLP_ENOMEM", "PMLP_EDEVICE", "PMLP_ESTATE",
    "PMLP_FP32", "PMLP_BF16_GEMM", "PMLP_BF16_STORE", "PMLP_BIAS", "PMLP_NUM_KERNELS", "ACT_IDS", "PmlpError",
    "library_path", "load_library", "pmlp_create", "pmlp_destroy", "pmlp_set_stream",
    "pmlp_set_precision", "pmlp_forward", "pmlp_train_step", "pmlp_train_step_lr",
    "pmlp_losses",
    "pmlp_gradients", "pmlp_hidden", "pmlp_get_params", "pmlp_set_params", "pmlp_info",
    "pmlp_set_profiling", "pmlp_kernel_time", "pmlp_profile_reset", "pmlp_kernel_name",
    "pmlp_last_error", "pmlp_gradients_ex", "pmlp_get_biases", "pmlp_set_biases",
    "PMLP_MSE", "pmlp_train_step_mse", "pmlp_gradients_mse", "pmlp_nonfinite", "pmlp_train_step_noalloc",
    "pmlp_set_feature_mask", "pmlp_get_models", "pmlp_create_deep", "pmlp_gradients_deep",
    "pmlp_get_params_deep", "pmlp_set_params_deep", "pmlp_info_deep", "pmlp_kernel_variant",
    "PMLP_ARITH_NONE", "PMLP_ARITH_FP32", "PMLP_ARITH_X3", "PMLP_ARITH_BF16", "PackedMLP",
    "DeepPackedMLP",
]

PMLP_OK = 0
PMLP_EINVAL = -1
PMLP_ENOMEM = -2
PMLP_EDEVICE = -3
PMLP_ESTATE = -4
PMLP_FP32 = 0
PMLP_BF16_GEMM = 1
PMLP_BF16_STORE = 2
PMLP_BIAS = 1
PMLP_MSE = 2
PMLP_NUM_KERNELS = 11

ACT_IDS = {
    "identity": 0, "relu": 1, "tanh": 2, "sigmoid": 3, "elu": 4, "leaky_relu": 5,
    "gelu": 6, "silu": 7, "softplus": 8, "swish2": 9,
    "selu": 10, "hardshrink": 11, "mish": 12,
}

_HERE = os.path.dirname(os.path.abspath(__file__))
_lib = None


def library_path() -> str:
    return os.path.join(_HERE, "libpmlp.so")


class PmlpError(RuntimeError):
    def __init__(self, code: int, what: str, msg: str):
        super().__init__("%s failed (code %d): %s" % (what, code, msg))
        self.code = code


def load_library():
    """Load libpmlp.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        raise ImportError("libpmlp.so is not built; run paper_2206_08369_amd.build.build()")
    lib = C.CDLL(path)
    P, i32, i64, u64, f32 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_float
    sig = {
        "pmlp_create": [C.POINTER(P), i32, i32, i32, P, P, u64],
        "pmlp_create_ex": [C.POINTER(P), i32, i32, i32, P, P, u64, i32],
        "pmlp_gradients_ex": [P, P, P, i32, P, P, P, P],
        "pmlp_train_step_mse": [P, P, P, i32, f32],
        "pmlp_gradients_mse": [P, P, P, i32, P, P],
        "pmlp_get_biases": [P, P, P],
        "pmlp_set_biases": [P, P, P],
        "pmlp_destroy": [P],
        "pmlp_set_stream": [P, P],
        "pmlp_set_precision": [P, i32],
        "pmlp_forward": [P, P, i32, P],
        "pmlp_train_step": [P, P, P, i32, f32],
        "pmlp_train_step_lr": [P, P, P, i32, P],
        "pmlp_losses": [P, P],
        "pmlp_gradients": [P, P, P, i32, P, P],
        "pmlp_hidden": [P, P, i32, P, P],
        "pmlp_get_params": [P, P, P],
        "pmlp_set_params": [P, P, P],
        "pmlp_info": [P, C.POINTER(i64), C.POINTER(i32), C.POINTER(i32), C.POINTER(i32)],
        "pmlp_set_profiling": [P, i32],
        "pmlp_kernel_time": [P, i32, C.POINTER(C.c_double), C.POINTER(i64)],
        "pmlp_profile_reset": [P],
        "pmlp_nonfinite": [P, C.POINTER(i32)],
        "pmlp_train_step_noalloc": [P, P, P, i32, f32],
        "pmlp_set_feature_mask": [P, P],
        "pmlp_get_models": [P, P, i32, P, P],
        "pmlp_create_deep": [C.POINTER(P), i32, i32, i32, P, P, P, u64],
        "pmlp_gradients_deep": [P, P, P, i32, P, P, P],
        "pmlp_get_params_deep": [P, P, P, P],
        "pmlp_set_params_deep": [P, P, P, P],
        "pmlp_info_deep": [P, C.POINTER(i64), C.POINTER(i64)],
        "pmlp_kernel_variant": [P, i32, C.POINTER(C.c_char_p), C.POINTER(i32)],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = C.c_int
    lib.pmlp_kernel_name.argtypes = [i32]
    lib.pmlp_kernel_name.restype = C.c_char_p
    lib.pmlp_last_error.argtypes = []
    lib.pmlp_last_error.restype = C.c_char_p
    _lib = lib
    return lib


def pmlp_last_error() -> str:
    return load_library().pmlp_last_error().decode()


def pmlp_kernel_name(k: int) -> str:
    return load_library().pmlp_kernel_name(int(k)).decode()


def _check(rc: int, what: str) -> int:
    if rc != PMLP_OK:
        raise PmlpError(rc, what, pmlp_last_error())
    return rc


def _host(a: np.ndarray, dtype) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


def _ptr(x) -> Optional[int]:
    """Device pointer of an int, a torch tensor or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


# --- raw C ABI (device pointers as integers) ------------------------------

def pmlp_create(F: int, O: int, hidden_sizes: Sequence[int], act_ids: Sequence[int],
                seed: int, flags: int = 0) -> int:
    hs = _host(hidden_sizes, np.int32)
    ac = _host(act_ids, np.int32)
    if hs.shape != ac.shape or hs.ndim != 1:
        raise ValueError("hidden_sizes and act_ids must be 1-D of equal length")
    h = C.c_void_p()
    _check(load_library().pmlp_create_ex(C.byref(h), int(F), int(O), int(hs.size),
                                         hs.ctypes.data, ac.ctypes.data,
                                         int(seed) & 0xFFFFFFFFFFFFFFFF, int(flags)),
           "pmlp_create_ex")
    return h.value


def pmlp_gradients_ex(h: int, X, y, B: int, dW1, dW2, db1, db2) -> None:
    _check(load_library().pmlp_gradients_ex(h, _ptr(X), _ptr(y), int(B), _ptr(dW1), _ptr(dW2),
                                            _ptr(db1), _ptr(db2)), "pmlp_gradients_ex")


def pmlp_get_biases(h: int, N: int, M: int, O: int) -> Tuple[np.ndarray, np.ndarray]:
    b1 = np.empty(N, np.float32)
    b2 = np.empty((M, O), np.float32)
    _check(load_library().pmlp_get_biases(h, b1.ctypes.data, b2.ctypes.data), "pmlp_get_biases")
    return b1, b2


def pmlp_set_biases(h: int, b1=None, b2=None) -> None:
    c1 = None if b1 is None else _host(b1, np.float32)
    c2 = None if b2 is None else _host(b2, np.float32)
    _check(load_library().pmlp_set_biases(h, None if c1 is None else c1.ctypes.data,
                                          None if c2 is None else c2.ctypes.data),
           "pmlp_set_biases")


def pmlp_destroy(h: int) -> None:
    _check(load_library().pmlp_destroy(h), "pmlp_destroy")


def pmlp_set_stream(h: int, stream: int) -> None:
    _check(load_library().pmlp_set_stream(h, stream or None), "pmlp_set_stream")


def pmlp_set_precision(h: int, mode: int) -> None:
    _check(load_library().pmlp_set_precision(h, int(mode)), "pmlp_set_precision")


def pmlp_forward(h: int, X, B: int, logits) -> None:
    _check(load_library().pmlp_forward(h, _ptr(X), int(B), _ptr(logits)), "pmlp_forward")


def pmlp_train_step(h: int, X, y, B: int, lr: float) -> None:
    _check(load_library().pmlp_train_step(h, _ptr(X), _ptr(y), int(B), float(lr)),
           "pmlp_train_step")


def pmlp_train_step_noalloc(h: int, X, y, B: int, lr: float) -> None:
    _check(load_library().pmlp_train_step_noalloc(h, _ptr(X), _ptr(y), int(B), float(lr)),
           "pmlp_train_step_noalloc")


def pmlp_train_step_lr(h: int, X, y, B: int, lr) -> None:
    _check(load_library().pmlp_train_step_lr(h, _ptr(X), _ptr(y), int(B), _ptr(lr)),
           "pmlp_train_step_lr")


def pmlp_train_step_mse(h: int, X, Y, B: int, lr: float) -> None:
    _check(load_library().pmlp_train_step_mse(h, _ptr(X), _ptr(Y), int(B), float(lr)),
           "pmlp_train_step_mse")


def pmlp_gradients_mse(h: int, X, Y, B: int, dW1, dW2) -> None:
    _check(load_library().pmlp_gradients_mse(h, _ptr(X), _ptr(Y), int(B), _ptr(dW1), _ptr(dW2)),
           "pmlp_gradients_mse")


def pmlp_losses(h: int) -> np.ndarray:
    M = pmlp_info(h)[1]
    out = np.empty(M, np.float32)
    _check(load_library().pmlp_losses(h, out.ctypes.data), "pmlp_losses")
    return out


def pmlp_gradients(h: int, X, y, B: int, dW1, dW2) -> None:
    _check(load_library().pmlp_gradients(h, _ptr(X), _ptr(y), int(B), _ptr(dW1), _ptr(dW2)),
           "pmlp_gradients")


def pmlp_hidden(h: int, X, B: int, Z=None, H=None) -> None:
    _check(load_library().pmlp_hidden(h, _ptr(X), int(B), _ptr(Z), _ptr(H)), "pmlp_hidden")


def pmlp_nonfinite(h: int) -> int:
    n = C.c_int32()
    _check(load_library().pmlp_nonfinite(h, C.byref(n)), "pmlp_nonfinite")
    return n.value


def pmlp_get_params(h: int) -> Tuple[np.ndarray, np.ndarray]:
    N, _, F, O = pmlp_info(h)
    W1 = np.empty((N, F), np.float32)
    W2 = np.empty((O, N), np.float32)
    _check(load_library().pmlp_get_params(h, W1.ctypes.data, W2.ctypes.data), "pmlp_get_params")
    return W1, W2


def pmlp_set_params(h: int, W1: Optional[np.ndarray], W2: Optional[np.ndarray]) -> None:
    N, _, F, O = pmlp_info(h)
    a = b = None
    if W1 is not None:
        a = _host(W1, np.float32)
        if a.shape != (N, F):
            raise ValueError("W1 must be [N, F] = [%d, %d]" % (N, F))
    if W2 is not None:
        b = _host(W2, np.float32)
        if b.shape != (O, N):
            raise ValueError("W2 must be [O, N] = [%d, %d]" % (O, N))
    _check(load_library().pmlp_set_params(h, None if a is None else a.ctypes.data,
                                          None if b is None else b.ctypes.data),
           "pmlp_set_params")


def pmlp_get_models(h: int, models, hidden_sizes) -> Tuple[np.ndarray, np.ndarray]:
    """W1 rows [R, F] and W2 columns [O, R] of the given models, in order."""
    _, _, F, O = pmlp_info(h)
    idx = _host(models, np.int32)
    hs = np.asarray(hidden_sizes, np.int64)
    ok = (idx >= 0) & (idx < hs.size)
    if not ok.all():   # the library rejects the list before copying anything
        _check(load_library().pmlp_get_models(h, idx.ctypes.data, int(idx.size), None, None),
               "pmlp_get_models")
    R = int(hs[idx].sum())
    W1 = np.empty((R, F), np.float32)
    W2 = np.empty((O, R), np.float32)
    _check(load_library().pmlp_get_models(h, idx.ctypes.data, int(idx.size), W1.ctypes.data,
                                          W2.ctypes.data), "pmlp_get_models")
    return W1, W2


def pmlp_create_deep(F: int, O: int, h1: Sequence[int], h2: Sequence[int],
                     act_ids: Sequence[int], seed: int) -> int:
    a, b, ac = _host(h1, np.int32), _host(h2, np.int32), _host(act_ids, np.int32)
    if not (a.shape == b.shape == ac.shape and a.ndim == 1):
        raise ValueError("h1, h2 and act_ids must be 1-D of equal length")
    h = C.c_void_p()
    _check(load_library().pmlp_create_deep(C.byref(h), int(F), int(O), int(a.size), a.ctypes.data,
                                           b.ctypes.data, ac.ctypes.data,
                                           int(seed) & 0xFFFFFFFFFFFFFFFF), "pmlp_create_deep")
    return h.value


def pmlp_gradients_deep(h: int, X, y, B: int, dW1, dW12, dW2) -> None:
    _check(load_library().pmlp_gradients_deep(h, _ptr(X), _ptr(y), int(B), _ptr(dW1), _ptr(dW12),
                                              _ptr(dW2)), "pmlp_gradients_deep")


def pmlp_info_deep(h: int) -> Tuple[int, int]:
    n2, k = C.c_int64(), C.c_int64()
    _check(load_library().pmlp_info_deep(h, C.byref(n2), C.byref(k)), "pmlp_info_deep")
    return n2.value, k.value


def pmlp_get_params_deep(h: int) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    N1, _, F, O = pmlp_info(h)
    N2, K = pmlp_info_deep(h)
    W1 = np.empty((N1, F), np.float32)
    W12 = np.empty(K, np.float32)
    W2 = np.empty((O, N2), np.float32)
    _check(load_library().pmlp_get_params_deep(h, W1.ctypes.data, W12.ctypes.data, W2.ctypes.data),
           "pmlp_get_params_deep")
    return W1, W12, W2


def pmlp_set_params_deep(h: int, W1=None, W12=None, W2=None) -> None:
    N1, _, F, O = pmlp_info(h)
    N2, K = pmlp_info_deep(h)
    arrs = []
    for a, shape, what in ((W1, (N1, F), "W1"), (W12, (K,), "W12"), (W2, (O, N2), "W2")):
        if a is None:
            arrs.append(None)
            continue
        c = _host(a, np.float32)
        if c.shape != shape:
            raise ValueError("%s must be %s" % (what, shape))
        arrs.append(c)
    _check(load_library().pmlp_set_params_deep(h, *[None if c is None else c.ctypes.data
                                                    for c in arrs]), "pmlp_set_params_deep")


def pmlp_set_feature_mask(h: int, mask: Optional[np.ndarray]) -> None:
    if mask is None:
        _check(load_library().pmlp_set_feature_mask(h, None), "pmlp_set_feature_mask")
        return
    _, M, F, _ = pmlp_info(h)
    a = np.ascontiguousarray(np.asarray(mask) != 0, dtype=np.uint8)
    if a.shape != (M, F):
        raise ValueError("feature masks must be [M, F] = [%d, %d]" % (M, F))
    _check(load_library().pmlp_set_feature_mask(h, a.ctypes.data), "pmlp_set_feature_mask")


def pmlp_info(h: int) -> Tuple[int, int, int, int]:
    N, M, F, O = C.c_int64(), C.c_int32(), C.c_int32(), C.c_int32()
    _check(load_library().pmlp_info(h, C.byref(N), C.byref(M), C.byref(F), C.byref(O)),
           "pmlp_info")
    return N.value, M.value, F.value, O.value


def pmlp_set_profiling(h: int, enable: bool) -> None:
    _check(load_library().pmlp_set_profiling(h, 1 if enable else 0), "pmlp_set_profiling")


def pmlp_kernel_time(h: int, k: int) -> Tuple[float, int]:
    ms, n = C.c_double(), C.c_int64()
    _check(load_library().pmlp_kernel_time(h, int(k), C.byref(ms), C.byref(n)),
           "pmlp_kernel_time")
    return ms.value, n.value


PMLP_ARITH_NONE, PMLP_ARITH_FP32, PMLP_ARITH_X3, PMLP_ARITH_BF16 = 0, 1, 2, 3


def pmlp_kernel_variant(h: int, k: int) -> Tuple[str, int]:
    """(kernel name, PMLP_ARITH_*) of role k's last launch."""
    name, arith = C.c_char_p(), C.c_int32()
    _check(load_library().pmlp_kernel_variant(h, int(k), C.byref(name), C.byref(arith)),
           "pmlp_kernel_variant")
    return (name.value or b"").decode(), arith.value


def pmlp_profile_reset(h: int) -> None:
    _check(load_library().pmlp_profile_reset(h), "pmlp_profile_reset")


# --- torch-facing wrapper -------------------------------------------------

class PackedMLP:
    """M independent one-hidden-layer MLPs packed into one wide network.

    Tensors passed in must be contiguous CUDA (HIP) tensors on the device
    that was current at construction: X float32 [B, F], and y int32 [B]
    labels (head "ce", classification) or float32 [B, O] targets (head
    "mse", regression).  Work is enqueued on torch's current stream of that
    device."""

    def __init__(self, F: int, O: int, hidden_sizes: Sequence[int], act_ids: Sequence[int],
                 seed: int = 0, precision: int = PMLP_FP32, biases: bool = False,
                 head: str = "ce"):
        import torch
        if head not in ("ce", "mse"):
            raise ValueError("head must be 'ce' or 'mse'")
        self._torch = torch
        self.device = torch.device("cuda", torch.cuda.current_device())
        self.biases = bool(biases)
        self.head = head
        self.handle = pmlp_create(F, O, hidden_sizes, act_ids, seed,
                                  (PMLP_BIAS if biases else 0) | (PMLP_MSE if head == "mse" else 0))
        self.N, self.M, self.F, self.O = pmlp_info(self.handle)
        self.hidden_sizes = _host(hidden_sizes, np.int32)
        self.act_ids = _host(act_ids, np.int32)
        if precision != PMLP_FP32:
            pmlp_set_precision(self.handle, precision)

    def close(self) -> None:
        if getattr(self, "handle", None):
            pmlp_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _stream(self) -> None:
        pmlp_set_stream(self.handle, self._torch.cuda.current_stream(self.device).cuda_stream)

    def _x(self, X):
        t = self._torch
        if not (X.is_cuda and X.dtype == t.float32 and X.is_contiguous() and X.dim() == 2
                and X.shape[1] == self.F and X.device == self.device):
            raise ValueError("X must be a contiguous float32 [B, %d] tensor on %s"
                             % (self.F, self.device))
        return X.shape[0]

    def _y(self, y, B):
        t = self._torch
        if self.head == "mse":
            if not (y.is_cuda and y.dtype == t.float32 and y.is_contiguous()
                    and tuple(y.shape) == (B, self.O) and y.device == self.device):
                raise ValueError("targets must be a contiguous float32 [B, %d] tensor on %s"
                                 % (self.O, self.device))
            return
        if not (y.is_cuda and y.dtype == t.int32 and y.is_contiguous() and y.shape == (B,)
                and y.device == self.device):
            raise ValueError("y must be a contiguous int32 [B] tensor on %s" % self.device)

    def set_precision(self, mode: int) -> None:
        pmlp_set_precision(self.handle, mode)

    def forward(self, X, out=None):
        B = self._x(X)
        if out is None:
            out = self._torch.empty((B, self.M, self.O), dtype=self._torch.float32,
                                    device=self.device)
        elif not (out.is_contiguous() and out.shape == (B, self.M, self.O)
                  and out.dtype == self._torch.float32):
            raise ValueError("out must be a contiguous float32 [B, M, O] tensor")
        self._stream()
        pmlp_forward(self.handle, X, B, out)
        return out

    def train_step(self, X, y, lr) -> None:
        """One SGD step; lr is one rate, or a float32 device tensor of M
        per-model rates."""
        B = self._x(X)
        self._y(y, B)
        self._stream()
        if self.head == "mse":
            if isinstance(lr, self._torch.Tensor):
                raise ValueError("per-model learning rates are not provided for the mse head")
            pmlp_train_step_mse(self.handle, X, y, B, lr)
            return
        if isinstance(lr, self._torch.Tensor):
            if not (lr.is_cuda and lr.dtype == self._torch.float32 and lr.is_contiguous()
                    and lr.numel() == self.M):
                raise ValueError("per-model lr must be a contiguous float32 device tensor of M rates")
            pmlp_train_step_lr(self.handle, X, y, B, lr)
        else:
            pmlp_train_step(self.handle, X, y, B, lr)

    def gradients(self, X, y):
        B = self._x(X)
        self._y(y, B)
        t = self._torch
        dW1 = t.empty((self.N, self.F), dtype=t.float32, device=self.device)
        dW2 = t.empty((self.O, self.N), dtype=t.float32, device=self.device)
        self._stream()
        if self.head == "mse":
            if self.biases:
                raise ValueError("bias gradients are not provided for the mse head")
            pmlp_gradients_mse(self.handle, X, y, B, dW1, dW2)
            return dW1, dW2
        if not self.biases:
            pmlp_gradients(self.handle, X, y, B, dW1, dW2)
            return dW1, dW2
        db1 = t.empty(self.N, dtype=t.float32, device=self.device)
        db2 = t.empty((self.M, self.O), dtype=t.float32, device=self.device)
        pmlp_gradients_ex(self.handle, X, y, B, dW1, dW2, db1, db2)
        return dW1, dW2, db1, db2

    def hidden(self, X):
        B = self._x(X)
        t = self._torch
        Z = t.empty((B, self.N), dtype=t.float32, device=self.device)
        H = t.empty((B, self.N), dtype=t.float32, device=self.device)
        self._stream()
        pmlp_hidden(self.handle, X, B, Z, H)
        return Z, H

    def losses(self) -> np.ndarray:
        return pmlp_losses(self.handle)

    def nonfinite_count(self) -> int:
        """(step, model) pairs with a non-finite loss since the last call."""
        return pmlp_nonfinite(self.handle)

    def get_params(self) -> Tuple[np.ndarray, np.ndarray]:
        return pmlp_get_params(self.handle)

    def get_models(self, models) -> Tuple[np.ndarray, np.ndarray]:
        """W1 [R, F] and W2 [O, R] of the given models (R: their hidden units)."""
        return pmlp_get_models(self.handle, models, self.hidden_sizes)

    def set_params(self, W1=None, W2=None) -> None:
        pmlp_set_params(self.handle, W1, W2)

    def set_feature_mask(self, mask) -> None:
        """Per-model input feature masks [M, F] (nonzero: the model sees the
        feature), or None to remove them."""
        pmlp_set_feature_mask(self.handle, mask)

    def get_biases(self) -> Tuple[np.ndarray, np.ndarray]:
        """b1 [N], b2 [M, O] of a handle made with biases=True."""
        return pmlp_get_biases(self.handle, self.N, self.M, self.O)

    def set_biases(self, b1=None, b2=None) -> None:
        pmlp_set_biases(self.handle, b1, b2)

    def set_profiling(self, enable: bool) -> None:
        pmlp_set_profiling(self.handle, enable)

    def kernel_times(self):
        """{kernel name: (total ms, launches)} since the last reset."""
        return {pmlp_kernel_name(k): pmlp_kernel_time(self.handle, k)
                for k in range(PMLP_NUM_KERNELS)}

    def kernel_variants(self):
        """{kernel role: (kernel name, PMLP_ARITH_*)} of the last launches."""
        return {pmlp_kernel_name(k): pmlp_kernel_variant(self.handle, k)
                for k in range(PMLP_NUM_KERNELS)}

    def profile_reset(self) -> None:
        pmlp_profile_reset(self.handle)


class DeepPackedMLP(PackedMLP):
    """M independent MLPs with two hidden layers each (h1[m] then h2[m]
    units, one activation per model), packed as one network.  Takes the
    forward, train_step, losses and nonfinite_count calls of PackedMLP;
    gradients and parameters carry the hidden-to-hidden blocks W12."""

    def __init__(self, F: int, O: int, h1: Sequence[int], h2: Sequence[int],
                 act_ids: Sequence[int], seed: int = 0):
        import torch
        self._torch = torch
        self.device = torch.device("cuda", torch.cuda.current_device())
        self.biases = False
        self.head = "ce"
        self.handle = pmlp_create_deep(F, O, h1, h2, act_ids, seed)
        self.N, self.M, self.F, self.O = pmlp_info(self.handle)
        self.N2, self.K = pmlp_info_deep(self.handle)
        self.hidden_sizes = _host(h1, np.int32)
        self.hidden_sizes2 = _host(h2, np.int32)
        self.act_ids = _host(act_ids, np.int32)

    def gradients(self, X, y):
        B = self._x(X)
        self._y(y, B)
        t = self._torch
        dW1 = t.empty((self.N, self.F), dtype=t.float32, device=self.device)
        dW12 = t.empty(max(self.K, 1), dtype=t.float32, device=self.device)
        dW2 = t.empty((self.O, self.N2), dtype=t.float32, device=self.device)
        self._stream()
        pmlp_gradients_deep(self.handle, X, y, B, dW1, dW12, dW2)
        return dW1, dW12[:self.K], dW2

    def get_params(self):
        return pmlp_get_params_deep(self.handle)

    def set_params(self, W1=None, W12=None, W2=None) -> None:
        pmlp_set_params_deep(self.handle, W1, W12, W2)
