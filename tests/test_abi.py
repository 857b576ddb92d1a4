"""The C-ABI library: it loads, exports every declared entry point, and
rejects invalid arguments before touching a device (no GPU needed)."""

import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2608_30384_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    txt = open(os.path.join(ROOT, "include", "rslm.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    names = re.findall(r"\b(?:int|size_t|const char \*)\s*\*?\s*(\w+)\s*\(", txt)
    return sorted(set(n for n in names if n.startswith(("rslm_", "ivf_"))))


def test_library_exports_every_declared_symbol():
    lib = L.lib()
    declared = _declared()
    assert len(declared) >= 15
    for name in declared:
        assert hasattr(lib, name), name
    assert set(declared) == set(L.EXPORTS)


def test_status_strings():
    lib = L.lib()
    for s, txt in L.STATUS.items():
        assert lib.rslm_status_string(s).decode() == txt
    assert lib.rslm_status_string(99).decode() == "unknown status"
    assert lib.rslm_version().decode().count(".") == 2


def _desc(dim=96, bits=4, passes=-1, mode=1, signs=None, perm=None, cb=None):
    import synth
    signs = np.ascontiguousarray(synth.sign_table() if signs is None else signs, dtype=np.int8)
    perm = np.ascontiguousarray(synth.permutation_table() if perm is None else perm, dtype=np.int32)
    cb = np.ascontiguousarray(synth.codebook(bits if 1 <= bits <= 4 else 4) if cb is None else cb,
                              dtype=np.float32)
    keep = (signs, perm, cb)
    d = L.PlanDesc(dim, bits, passes, mode, signs.ctypes.data_as(C.POINTER(C.c_int8)),
                   perm.ctypes.data_as(C.POINTER(C.c_int32)), cb.ctypes.data_as(C.POINTER(C.c_float)))
    return d, keep


@pytest.mark.parametrize("kw", [
    dict(dim=0), dict(dim=5000), dict(bits=5), dict(bits=0), dict(passes=3), dict(mode=2),
    dict(signs=np.zeros(256)), dict(perm=np.zeros(128)),
    dict(cb=np.linspace(-2, 2, 16) + 1e-4),          # not float16-exact
    dict(cb=np.linspace(2, -2, 16).astype(np.float16).astype(np.float32)),   # not ascending
])
def test_plan_create_validates_before_device(kw):
    d, keep = _desc(**kw)
    h = C.c_void_p()
    assert L.lib().rslm_plan_create(C.byref(d), C.byref(h)) == 1


def test_calls_validate_arguments_without_device():
    lib = L.lib()
    null = C.c_void_p(0)
    assert lib.rslm_fwht(null, null, null, 4, 0, null) == 1
    assert lib.ivf_assign_probe(null, 4, 8, null, 0, 1, 0, null, null, null, 0, null) == 1
    assert lib.ivf_assign_probe(null, 4, 8, null, 16, 2, 0, null, null, null, 0, null) == 1
    assert lib.ivf_assign_probe(null, 4, 8, null, 16, 17, 1, null, null, null, 0, null) == 1
    assert lib.rslm_sq8_fit(null, 4, 0, null, null, 0, null) == 1
    assert lib.rslm_encode(null, null, 0, null, null, 0, null, null, 0, null, null, null, null) == 1
    assert lib.ivf_kmeans_update(null, 4, 8, null, 0, null, null, 0, null) == 1      # nlist 0
    assert lib.ivf_kmeans_update(null, 4, 8, null, 16, null, null, 0, null) == 1     # no centres
    assert lib.ivf_kmeans_update(null, 4, 0, null, 16, C.c_void_p(256), null, 0, null) == 1
    assert lib.ivf_kmeans_update(C.c_void_p(0x1002), 4, 8, C.c_void_p(256), 16, C.c_void_p(256),
                                 C.c_void_p(256), 1 << 20, null) == 1              # misaligned
    assert lib.ivf_kmeans_update(C.c_void_p(256), 4, 8, C.c_void_p(256), 16, C.c_void_p(256),
                                 C.c_void_p(256), 16, null) == 4                   # workspace
    assert lib.ivf_kmeans_update(null, 0, 8, null, 16, C.c_void_p(256), null, 0, null) == 0
    codec = L.RescoreCodec(7, 8, 10, 0, 0, 0)
    assert lib.rslm_rescore(C.byref(codec), null, 1, null, null, 10, 10, null, null, null) == 2
    codec = L.RescoreCodec(0, 8, 10, 0, 0, 0)
    assert lib.rslm_rescore(C.byref(codec), null, 1, null, null, 10, 20, null, null, null) == 1


def test_workspace_sizes_are_host_side():
    lib = L.lib()
    assert lib.ivf_assign_probe_workspace(256, 768, 4096, 64, 1) >= 256 * 4096 * 4
    assert lib.ivf_assign_probe_workspace(256, 768, 4096, 1, 0) >= 4096 * 4
    assert lib.ivf_kmeans_update_workspace(1000, 16) >= 1000 * 4 + 3 * 16 * 4
    # the unified query answers as the per-call functions
    assert lib.rslm_workspace_size(2, None, None, 256, 768, 4096, 64, 0) == \
        lib.ivf_assign_probe_workspace(256, 768, 4096, 64, 1)
    assert lib.rslm_workspace_size(1, None, None, 5000, 96, 1024, 7, 0) == \
        lib.ivf_assign_probe_workspace(5000, 96, 1024, 1, 0)
    assert lib.rslm_workspace_size(3, None, None, 1000, 0, 16, 0, 0) == \
        lib.ivf_kmeans_update_workspace(1000, 16)
    assert lib.rslm_workspace_size(0, None, None, 256, 0, 0, 64, 100) == 0   # no plan
    assert lib.rslm_workspace_size(9, None, None, 256, 768, 4096, 64, 100) == 0
