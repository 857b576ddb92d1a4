"""ctypes declarations of librslm's C ABI (include/rslm.h).

Loading fails loudly when the shared library has not been built: there is no
fallback implementation anywhere in this package.
"""

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librslm.so")

RSLM_OK = 0
STATUS = {0: "ok", 1: "invalid argument", 2: "unsupported", 3: "HIP error",
          4: "workspace too small", 5: "no gfx950 device"}
IVF_ASSIGN_L2 = 0
IVF_PROBE_IP = 1
RSLM_RESCORE_SQ8 = 0
RSLM_RESCORE_RSLM = 1

EXPORTS = [
    "rslm_status_string", "rslm_last_hip_error", "rslm_version",
    "rslm_plan_create", "rslm_plan_destroy", "rslm_plan_get_info",
    "rslm_fwht", "rslm_encode", "rslm_encode_two_stage", "rslm_encode_sq8", "rslm_pack_codes",
    "rslm_pack_records", "rslm_score", "rslm_decode", "rslm_unpack_codes",
    "ivf_assign_probe_workspace", "ivf_assign_probe", "ivf_assign_probe_noalloc",
    "ivf_assign_probe_noalloc_limit", "ivf_kmeans_update_workspace",
    "ivf_kmeans_update",
    "rslm_scan_topk_workspace", "rslm_scan_topk", "rslm_workspace_size",
    "rslm_sq8_fit", "rslm_sq8_encode", "rslm_rescore", "rslm_set_timer", "rslm_calibrate_read",
    "rslm_grid2_lists",
]


class PlanDesc(C.Structure):
    _fields_ = [("dim", C.c_int32), ("bits", C.c_int32), ("passes", C.c_int32),
                ("scale_mode", C.c_int32), ("signs", C.POINTER(C.c_int8)),
                ("perm", C.POINTER(C.c_int32)), ("codebook", C.POINTER(C.c_float)),
                ("lite", C.c_int32), ("codebook_lead", C.POINTER(C.c_float))]


class PlanInfo(C.Structure):
    _fields_ = [("dim", C.c_int32), ("bits", C.c_int32), ("passes", C.c_int32),
                ("scale_mode", C.c_int32), ("K", C.c_int32), ("g", C.c_int32),
                ("block", C.c_int32), ("n_full_blocks", C.c_int32), ("d_pad", C.c_int32),
                ("canon_bytes", C.c_int32), ("tile_records", C.c_int32),
                ("tile_bytes", C.c_int32), ("emax", C.c_double), ("lite", C.c_int32),
                ("record_bytes", C.c_int32)]


class Index(C.Structure):
    _fields_ = [("nlist", C.c_int32), ("max_list_size", C.c_int32),
                ("list_offsets", C.c_void_p), ("list_sizes", C.c_void_p),
                ("ids", C.c_void_p), ("codes", C.c_void_p), ("scales", C.c_void_p)]


class RescoreCodec(C.Structure):
    _fields_ = [("kind", C.c_int32), ("dim", C.c_int32), ("n_vectors", C.c_int64),
                ("codes", C.c_void_p), ("lo", C.c_void_p), ("hi", C.c_void_p),
                ("scales", C.c_void_p), ("plan", C.c_void_p)]


_lib = None

P = C.c_void_p
I32 = C.c_int32
I64 = C.c_int64
SZ = C.c_size_t


def _declare(lib):
    sig = {
        "rslm_status_string": (C.c_char_p, [C.c_int]),
        "rslm_last_hip_error": (C.c_int, []),
        "rslm_version": (C.c_char_p, []),
        "rslm_plan_create": (C.c_int, [C.POINTER(PlanDesc), C.POINTER(C.c_void_p)]),
        "rslm_plan_destroy": (C.c_int, [P]),
        "rslm_plan_get_info": (C.c_int, [P, C.POINTER(PlanInfo)]),
        "rslm_fwht": (C.c_int, [P, P, P, I64, C.c_int, P]),
        "rslm_encode": (C.c_int, [P, P, I64, P, P, I64, P, P, I32, P, P, P, P]),
        "rslm_encode_two_stage": (C.c_int, [P, P, P, I64, P, P, I64, P, P, I32, P, P, P, P,
                                            P]),
        "rslm_encode_sq8": (C.c_int, [P, P, I64, P, P, I64, P, P, I32, P, P, P, P, P, P]),
        "rslm_pack_codes": (C.c_int, [P, P, I64, P, P]),
        "rslm_pack_records": (C.c_int, [P, P, P, I64, P, P]),
        "rslm_score": (C.c_int, [P, P, I64, P, I64, P, I32, P, P]),
        "rslm_decode": (C.c_int, [P, P, P, I64, P, P, I32, P, P]),
        "rslm_unpack_codes": (C.c_int, [P, P, I64, P, P]),
        "ivf_assign_probe_workspace": (SZ, [I64, I32, I32, I32, C.c_int]),
        "ivf_assign_probe": (C.c_int, [P, I64, I32, P, I32, I32, C.c_int, P, P, P, SZ, P]),
        "ivf_assign_probe_noalloc": (C.c_int, [P, I64, I32, P, I32, I32, C.c_int, P, P, P]),
        "ivf_assign_probe_noalloc_limit": (SZ, []),
        "ivf_kmeans_update_workspace": (SZ, [I64, I32]),
        "ivf_kmeans_update": (C.c_int, [P, I64, I32, P, I32, P, P, SZ, P]),
        "rslm_scan_topk_workspace": (SZ, [P, C.POINTER(Index), I32, I32, I32]),
        "rslm_workspace_size": (SZ, [C.c_int, P, C.POINTER(Index), I64, I32, I32, I32, I32]),
        "rslm_scan_topk": (C.c_int, [P, C.POINTER(Index), P, I32, P, P, I32, I32, P, P, P,
                                     SZ, P]),
        "rslm_sq8_fit": (C.c_int, [P, I64, I32, P, P, C.c_int, P]),
        "rslm_sq8_encode": (C.c_int, [P, I64, I32, P, P, P, I64, P, P]),
        "rslm_rescore": (C.c_int, [C.POINTER(RescoreCodec), P, I32, P, P, I32, I32, P, P, P]),
        "rslm_set_timer": (C.c_int, [C.c_int, P, P]),
        "rslm_calibrate_read": (C.c_int, [P, I64, P, I32, C.c_int, P]),
        "rslm_grid2_lists": (C.c_int, [P, I32, C.c_float, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args


def lib():
    """Load librslm.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2608_30384_amd.build`"
                " (librslm is the only implementation; there is no fallback)")
        handle = C.CDLL(LIB_PATH, mode=C.RTLD_GLOBAL)
        _declare(handle)
        _lib = handle
    return _lib


class RslmError(RuntimeError):
    def __init__(self, fn, status):
        msg = f"{fn}: {STATUS.get(status, status)}"
        if status == 3:
            msg += f" (hipError {lib().rslm_last_hip_error()})"
        super().__init__(msg)
        self.status = status


def check(fn, status):
    if status != RSLM_OK:
        raise RslmError(fn, status)
