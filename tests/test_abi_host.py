"""Host-side checks of the C ABI that need no GPU: the library loads, it
exports every function include/pmlp.h declares, and argument errors are
reported before any device work."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "pmlp.h")


@pytest.fixture(scope="module")
def pm():
    import paper_2206_08369_amd as pm
    if not os.path.exists(pm.library_path()):
        from paper_2206_08369_amd import build
        build.build()
    pm.load_library()
    return pm


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pmlp_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("pmlp_create", "pmlp_destroy", "pmlp_forward", "pmlp_train_step",
                     "pmlp_losses", "pmlp_gradients", "pmlp_get_params", "pmlp_set_params"):
        assert required in names


def test_library_exports_every_declared_symbol(pm):
    lib = C.CDLL(pm.library_path())
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_kernel_names(pm):
    names = [pm.pmlp_kernel_name(k) for k in range(pm.PMLP_NUM_KERNELS)]
    assert names[1] == "gemm_fwd" and names[3] == "m3_fwd" and names[5] == "m3_bwd"
    assert pm.pmlp_kernel_name(99) == ""


@pytest.mark.parametrize("F,O,hs,acts,msg", [
    (0, 2, [1], [0], "F must be"),
    (3, 1, [1], [0], "O must be"),
    (3, 17, [1], [0], "O must be"),
    (3, 2, [0], [0], "hidden size"),
    (3, 2, [2, -1], [0, 0], "hidden size"),
    (3, 2, [1], [13], "activation id"),
    (3, 2, [1], [-1], "activation id"),
])
def test_create_rejects_bad_arguments(pm, F, O, hs, acts, msg):
    with pytest.raises(pm.PmlpError) as e:
        pm.pmlp_create(F, O, hs, acts, 0)
    assert e.value.code == pm.PMLP_EINVAL
    assert msg in str(e.value)


def test_null_arguments_rejected(pm):
    lib = pm.load_library()
    h = C.c_void_p()
    hs = np.ones(2, np.int32)
    assert lib.pmlp_create(None, 3, 2, 2, hs.ctypes.data, hs.ctypes.data, 0) == pm.PMLP_EINVAL
    assert lib.pmlp_create(C.byref(h), 3, 2, 2, None, hs.ctypes.data, 0) == pm.PMLP_EINVAL
    assert lib.pmlp_create(C.byref(h), 3, 2, 0, hs.ctypes.data, hs.ctypes.data, 0) == pm.PMLP_EINVAL
    assert h.value is None
    for fn, args in [("pmlp_forward", (None, None, 1, None)),
                     ("pmlp_train_step", (None, None, None, 1, C.c_float(0.1))),
                     ("pmlp_losses", (None, None)),
                     ("pmlp_info", (None, None, None, None, None)),
                     ("pmlp_set_precision", (None, 0)),
                     ("pmlp_kernel_time", (None, 0, None, None))]:
        assert getattr(lib, fn)(*args) == pm.PMLP_EINVAL, fn
    assert "null handle" in pm.pmlp_last_error()
    assert lib.pmlp_destroy(None) == pm.PMLP_OK


def test_package_fails_loudly_without_library(tmp_path, monkeypatch):
    """The binding has no CPU fallback: a missing library is an error."""
    import paper_2206_08369_amd as pm
    monkeypatch.setattr(pm, "_lib", None)
    monkeypatch.setattr(pm, "library_path", lambda: str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        pm.load_library()


def test_create_rejects_unknown_flags(pm):
    with pytest.raises(pm.PmlpError) as e:
        pm.pmlp_create(3, 2, [1], [0], 0, flags=4)
    assert e.value.code == pm.PMLP_EINVAL and "unknown flags" in str(e.value)
