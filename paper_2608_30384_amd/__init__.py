"""MI355X-native RSLM IVF scan and encoder (arXiv 2608.30384).

The computation lives in ``librslm.so`` (HIP kernels for gfx950, C ABI in
``include/rslm.h``); this package only binds it.  Build it with
``python -m paper_2608_30384_amd.build``.
"""

from ._lib import IVF_ASSIGN_L2, IVF_PROBE_IP, RslmError, lib
from .api import (
    Index, Plan, ivf_assign_probe, ivf_kmeans_update, rslm_decode, rslm_encode, rslm_encode_sq8, rslm_encode_two_stage, rslm_fwht,
    rslm_pack_codes, rslm_pack_records, rslm_score,
    rslm_rescore, rslm_rescore_rslm, rslm_scan_topk, rslm_scan_topk_workspace, rslm_sq8_encode,
    rslm_sq8_fit, rslm_unpack_codes,
)

__all__ = [
    "IVF_ASSIGN_L2", "IVF_PROBE_IP", "RslmError", "lib", "Index", "Plan", "ivf_assign_probe", "ivf_kmeans_update",
    "rslm_decode", "rslm_encode", "rslm_encode_sq8", "rslm_encode_two_stage", "rslm_fwht", "rslm_pack_codes",
    "rslm_pack_records", "rslm_rescore", "rslm_rescore_rslm", "rslm_scan_topk",
    "rslm_scan_topk_workspace", "rslm_score", "rslm_sq8_encode", "rslm_sq8_fit",
    "rslm_unpack_codes",
]
