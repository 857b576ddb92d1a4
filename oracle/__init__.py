"""CPU oracle for the RSLM IVF scan / encode path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 NumPy restatement of what the RSLM paper (arXiv
2608.30384, "RSLM: Training-Free Vector Quantization for Approximate Nearest
Neighbor Search") computes.  It exists to check the HIP library; it is not
part of the product.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it.  It shares no code with
the HIP library (``paper_2608_30384_amd``) and imports nothing from it; the
two meet only through the seeded inputs of the ``synth`` package.

Every function cites the passage of the paper it follows; where the paper is
silent the reading taken is stated in the docstring.

Parity status: every function is pinned by ``tests/test_oracle_*.py``
against closed forms, library routines, invariants or brute force, except
the 2-D/4-D codebook *values* (unique only up to an orthogonal map; pinned
only through the Lloyd optimality conditions), see ``tests``.
"""

from .rotation import (
    block_size, block_list, resolve_passes, hadamard, intra_block_perm,
    rotate, rotation_matrix,
)
from .codec import (
    codec_shape, e_max, enc_ue7m9, dec_ue7m9, enc_ue4m12, dec_ue4m12,
    encode, pack_canonical, unpack_canonical, canonical_code_bytes,
    decode_rotated, reconstruct, first_stage_rotated, encode_rescore, reconstruct_rescore,
    lite_lead, record_bytes, pack_records, unpack_records,
)
from .search import (
    assign_l2, assign_l2_expanded, probe_ip, kmeans, scan_scores_lut, scan_scores_dense, topk,
    ivf_candidates, ivf_search, sq8_fit, sq8_encode, sq8_decode, rescore_sq8, rescore_sq8_scores,
    rescore_rslm, rescore_rslm_scores, brute_force_mips,
)

__all__ = [n for n in dir() if not n.startswith("_")]
