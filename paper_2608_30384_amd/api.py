"""Thin Python binding of librslm: torch tensors in, C ABI calls out.

Every function marshals arguments (device pointers, sizes, the current HIP
stream) and calls the entry point of the same name in ``include/rslm.h``;
all computation happens in the HIP kernels.  Tensors must be contiguous,
on the plan's device, with the dtypes stated in the C header.
"""

import ctypes as C

import numpy as np
import torch

from . import _lib as L


def _ptr(t):
    return C.c_void_p(t.data_ptr()) if t is not None else C.c_void_p(0)


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _need(t, dtype, name):
    if t is None:
        return
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


class _Workspace:
    """Grow-only scratch buffer per device, stream and purpose.

    Keyed by stream as well: calls on different streams never share a buffer
    (they would race), and a buffer is allocated while its stream is current,
    so torch's caching allocator ties it to that stream and does not hand its
    memory to another stream while a kernel there may still use it."""

    def __init__(self):
        self._bufs = {}

    def get(self, nbytes, device, key, stream=None):
        s = stream if stream is not None else torch.cuda.current_stream(device)
        k = (str(device), s.cuda_stream, key)
        b = self._bufs.get(k)
        if b is None or b.numel() < nbytes:
            with torch.cuda.stream(s):
                b = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
            self._bufs[k] = b
        return b


_WS = _Workspace()


class Plan:
    """An RSLM codec plan (``rslm_plan_create``) on the current device."""

    def __init__(self, dim, bits, passes=-1, scale_mode="global", signs=None, perm=None,
                 codebook=None, lite=False):
        import synth  # the fixed tables are inputs shared as data

        signs = synth.sign_table() if signs is None else np.asarray(signs, dtype=np.int8)
        perm = synth.permutation_table() if perm is None else np.asarray(perm, dtype=np.int32)
        cb = synth.codebook(bits) if codebook is None else np.asarray(codebook, dtype=np.float32)
        self._signs = np.ascontiguousarray(signs, dtype=np.int8)
        self._perm = np.ascontiguousarray(perm, dtype=np.int32)
        self._cb = np.ascontiguousarray(cb, dtype=np.float32).reshape(-1)
        # Rslm4Lite: the K = 8 (3-bit) codebook for the leading coordinates
        self._cbl = np.ascontiguousarray(synth.codebook(3), dtype=np.float32).reshape(-1)
        mode = {"local": 0, "global": 1}.get(scale_mode, scale_mode)
        desc = L.PlanDesc(dim, bits, passes, int(mode),
                          self._signs.ctypes.data_as(C.POINTER(C.c_int8)),
                          self._perm.ctypes.data_as(C.POINTER(C.c_int32)),
                          self._cb.ctypes.data_as(C.POINTER(C.c_float)), int(bool(lite)),
                          self._cbl.ctypes.data_as(C.POINTER(C.c_float)))
        h = C.c_void_p()
        L.check("rslm_plan_create", L.lib().rslm_plan_create(C.byref(desc), C.byref(h)))
        self.handle = h
        info = L.PlanInfo()
        L.check("rslm_plan_get_info", L.lib().rslm_plan_get_info(h, C.byref(info)))
        self.info = info
        self.dim, self.bits = dim, bits
        self.passes = info.passes
        self.d_pad = info.d_pad
        self.tile_bytes = info.tile_bytes
        self.canon_bytes = info.canon_bytes
        self.record_bytes = info.record_bytes
        self.lite = bool(info.lite)
        self.emax = info.emax
        self.device = torch.device("cuda", torch.cuda.current_device())

    def code_bytes(self, n_records):
        return (n_records + 15) // 16 * self.tile_bytes

    def close(self):
        if self.handle:
            L.lib().rslm_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def rslm_fwht(plan, x, y=None, inverse=False, stream=None):
    _need(x, torch.float32, "x")
    n = x.shape[0] if x.dim() > 1 else 1
    if x.numel() != n * plan.dim:
        raise ValueError("x must be n x dim")
    if y is None:
        y = torch.empty_like(x)
    _need(y, torch.float32, "y")
    L.check("rslm_fwht", L.lib().rslm_fwht(plan.handle, _ptr(x), _ptr(y), n, int(inverse),
                                           _stream(stream)))
    return y


def rslm_encode(plan, x, codes, scales, n_records=None, src_row=None, rec_list=None,
                centroids=None, centroids_rot=None, resid_rot=None, stream=None):
    _need(x, torch.float32, "x")
    _need(codes, torch.uint8, "codes")
    _need(scales, torch.int32, "scales")
    _need(src_row, torch.int64, "src_row")
    _need(rec_list, torch.int32, "rec_list")
    _need(centroids, torch.float32, "centroids")
    _need(centroids_rot, torch.float32, "centroids_rot")
    _need(resid_rot, torch.float32, "resid_rot")
    n_rows = x.shape[0]
    if n_records is None:
        n_records = src_row.shape[0] if src_row is not None else n_rows
    if codes.numel() < plan.code_bytes(n_records) or scales.numel() < n_records:
        raise ValueError("codes / scales too small")
    if resid_rot is not None and resid_rot.numel() < n_rows * plan.dim:
        raise ValueError("resid_rot too small")
    nlist = centroids.shape[0] if centroids is not None else 0
    L.check("rslm_encode", L.lib().rslm_encode(
        plan.handle, _ptr(x), n_rows, _ptr(src_row), _ptr(rec_list), n_records,
        _ptr(centroids), _ptr(centroids_rot), nlist, _ptr(codes), _ptr(scales),
        _ptr(resid_rot), _stream(stream)))


def rslm_encode_two_stage(plan, plan2, x, codes, scales, codes2, scales2, n_records=None,
                          src_row=None, rec_list=None, centroids=None, centroids_rot=None,
                          stream=None):
    """``rslm_encode`` plus the rescoring codec ``plan2`` on the second
    residual; codes2 (n_rows x plan2.canon_bytes uint8) and scales2 (n_rows
    int32) are indexed by row of x."""
    _need(x, torch.float32, "x")
    _need(codes, torch.uint8, "codes")
    _need(scales, torch.int32, "scales")
    _need(codes2, torch.uint8, "codes2")
    _need(scales2, torch.int32, "scales2")
    _need(src_row, torch.int64, "src_row")
    _need(rec_list, torch.int32, "rec_list")
    _need(centroids, torch.float32, "centroids")
    _need(centroids_rot, torch.float32, "centroids_rot")
    n_rows = x.shape[0]
    if n_records is None:
        n_records = src_row.shape[0] if src_row is not None else n_rows
    if codes.numel() < plan.code_bytes(n_records) or scales.numel() < n_records:
        raise ValueError("codes / scales too small")
    if codes2.numel() < n_rows * plan2.canon_bytes or scales2.numel() < n_rows:
        raise ValueError("codes2 / scales2 too small")
    nlist = centroids.shape[0] if centroids is not None else 0
    L.check("rslm_encode_two_stage", L.lib().rslm_encode_two_stage(
        plan.handle, plan2.handle, _ptr(x), n_rows, _ptr(src_row), _ptr(rec_list), n_records,
        _ptr(centroids), _ptr(centroids_rot), nlist, _ptr(codes), _ptr(scales), _ptr(codes2),
        _ptr(scales2), _stream(stream)))


def rslm_encode_sq8(plan, x, codes, scales, lo, hi, codes2, n_records=None, src_row=None,
                    rec_list=None, centroids=None, centroids_rot=None, stream=None):
    """``rslm_encode`` with the second residual written as SQ8 codes (ranges
    lo / hi); codes2 (n_rows x dim uint8) is indexed by row of x."""
    _need(x, torch.float32, "x")
    _need(codes, torch.uint8, "codes")
    _need(scales, torch.int32, "scales")
    _need(lo, torch.float32, "lo")
    _need(hi, torch.float32, "hi")
    _need(codes2, torch.uint8, "codes2")
    _need(src_row, torch.int64, "src_row")
    _need(rec_list, torch.int32, "rec_list")
    _need(centroids, torch.float32, "centroids")
    _need(centroids_rot, torch.float32, "centroids_rot")
    n_rows = x.shape[0]
    if n_records is None:
        n_records = src_row.shape[0] if src_row is not None else n_rows
    if codes.numel() < plan.code_bytes(n_records) or scales.numel() < n_records:
        raise ValueError("codes / scales too small")
    if codes2.numel() < n_rows * plan.dim or lo.numel() < plan.dim or hi.numel() < plan.dim:
        raise ValueError("codes2 / lo / hi too small")
    nlist = centroids.shape[0] if centroids is not None else 0
    L.check("rslm_encode_sq8", L.lib().rslm_encode_sq8(
        plan.handle, _ptr(x), n_rows, _ptr(src_row), _ptr(rec_list), n_records,
        _ptr(centroids), _ptr(centroids_rot), nlist, _ptr(codes), _ptr(scales), _ptr(lo),
        _ptr(hi), _ptr(codes2), _stream(stream)))


def rslm_pack_codes(plan, canon, n, stream=None):
    _need(canon, torch.uint8, "canon")
    tiles = torch.empty(plan.code_bytes(n), dtype=torch.uint8, device=canon.device)
    L.check("rslm_pack_codes", L.lib().rslm_pack_codes(plan.handle, _ptr(canon), n,
                                                       _ptr(tiles), _stream(stream)))
    return tiles


def rslm_decode(plan, codes, scales, n, rec_list=None, centroids=None, out=None, stream=None):
    """Reconstructions x~ = g^ (c + R^T s^ C[code]) of n records (n x dim)."""
    _need(codes, torch.uint8, "codes")
    _need(scales, torch.int32, "scales")
    _need(rec_list, torch.int32, "rec_list")
    _need(centroids, torch.float32, "centroids")
    if out is None:
        out = torch.empty((n, plan.dim), dtype=torch.float32, device=codes.device)
    _need(out, torch.float32, "out")
    nlist = centroids.shape[0] if centroids is not None else 0
    L.check("rslm_decode", L.lib().rslm_decode(plan.handle, _ptr(codes), _ptr(scales), n,
                                               _ptr(rec_list), _ptr(centroids), nlist, _ptr(out),
                                               _stream(stream)))
    return out


def rslm_pack_records(plan, tiles, scales, n, stream=None):
    """Packed records (codes + scale suffix; Lite: codes alone), n x record_bytes."""
    _need(tiles, torch.uint8, "tiles")
    _need(scales, torch.int32, "scales")
    records = torch.empty((n, plan.record_bytes), dtype=torch.uint8, device=tiles.device)
    L.check("rslm_pack_records", L.lib().rslm_pack_records(plan.handle, _ptr(tiles), _ptr(scales),
                                                           n, _ptr(records), _stream(stream)))
    return records


def rslm_score(plan, records, q_rot, ids=None, n=None, out=None, stream=None):
    """OneToMany scores (Q x n) of packed records, contiguous (ids None) or
    gathered by int64 ids."""
    _need(records, torch.uint8, "records")
    _need(q_rot, torch.float32, "q_rot")
    _need(ids, torch.int64, "ids")
    n_pool = records.numel() // plan.record_bytes
    if n is None:
        n = ids.numel() if ids is not None else n_pool
    Q = q_rot.shape[0]
    if out is None:
        out = torch.empty((Q, n), dtype=torch.float32, device=q_rot.device)
    _need(out, torch.float32, "out")
    L.check("rslm_score", L.lib().rslm_score(plan.handle, _ptr(records), n_pool, _ptr(ids), n,
                                             _ptr(q_rot), Q, _ptr(out), _stream(stream)))
    return out


def rslm_unpack_codes(plan, tiles, n, stream=None):
    _need(tiles, torch.uint8, "tiles")
    canon = torch.empty((n, plan.canon_bytes), dtype=torch.uint8, device=tiles.device)
    L.check("rslm_unpack_codes", L.lib().rslm_unpack_codes(plan.handle, _ptr(tiles), n,
                                                           _ptr(canon), _stream(stream)))
    return canon


def ivf_assign_probe(x, centroids, nprobe=1, mode=L.IVF_ASSIGN_L2, out_ids=None,
                     out_scores=None, stream=None):
    _need(x, torch.float32, "x")
    _need(centroids, torch.float32, "centroids")
    n, dim = x.shape
    nlist = centroids.shape[0]
    shape = (n,) if mode == L.IVF_ASSIGN_L2 else (n, nprobe)
    if out_ids is None:
        out_ids = torch.empty(shape, dtype=torch.int32, device=x.device)
    if out_scores is None:
        out_scores = torch.empty(shape, dtype=torch.float32, device=x.device)
    nb = L.lib().ivf_assign_probe_workspace(n, dim, nlist, nprobe, mode)
    ws = _WS.get(nb, x.device, "probe", stream)
    L.check("ivf_assign_probe", L.lib().ivf_assign_probe(
        _ptr(x), n, dim, _ptr(centroids), nlist, nprobe, mode, _ptr(out_ids),
        _ptr(out_scores), _ptr(ws), ws.numel(), _stream(stream)))
    return out_ids, out_scores


def ivf_assign_probe_noalloc(x, centroids, nprobe, mode, out_ids, out_scores, stream=None):
    """``ivf_assign_probe`` through the entry point that allocates nothing
    (fixed per-GPU scratch); the caller provides the outputs."""
    _need(x, torch.float32, "x")
    _need(centroids, torch.float32, "centroids")
    _need(out_ids, torch.int32, "out_ids")
    _need(out_scores, torch.float32, "out_scores")
    n, dim = x.shape
    L.check("ivf_assign_probe_noalloc", L.lib().ivf_assign_probe_noalloc(
        _ptr(x), n, dim, _ptr(centroids), centroids.shape[0], nprobe, mode, _ptr(out_ids),
        _ptr(out_scores), _stream(stream)))
    return out_ids, out_scores


def ivf_kmeans_update(x, assign, centroids, stream=None):
    """One Lloyd centre update in place: centroids[p] = mean of the rows of x
    assigned to p (an empty centre keeps its value)."""
    _need(x, torch.float32, "x")
    _need(assign, torch.int32, "assign")
    _need(centroids, torch.float32, "centroids")
    n, dim = x.shape
    if assign.numel() != n or centroids.dim() != 2 or centroids.shape[1] != dim:
        raise ValueError("assign must have n entries and centroids nlist x dim")
    nlist = centroids.shape[0]
    nb = L.lib().ivf_kmeans_update_workspace(n, nlist)
    ws = _WS.get(nb, x.device, "kmeans", stream)
    L.check("ivf_kmeans_update", L.lib().ivf_kmeans_update(
        _ptr(x), n, dim, _ptr(assign), nlist, _ptr(centroids), _ptr(ws), ws.numel(),
        _stream(stream)))
    return centroids


class Index:
    """Device arrays of an IVF index of RSLM records (``rslm_index``)."""

    def __init__(self, list_offsets, list_sizes, ids, codes, scales, max_list_size=None):
        _need(list_offsets, torch.int64, "list_offsets")
        _need(list_sizes, torch.int32, "list_sizes")
        _need(ids, torch.int32, "ids")
        _need(codes, torch.uint8, "codes")
        _need(scales, torch.int32, "scales")
        self.list_offsets, self.list_sizes = list_offsets, list_sizes
        self.ids, self.codes, self.scales = ids, codes, scales
        self.nlist = list_sizes.numel()
        self.max_list_size = int(list_sizes.max().item()) if max_list_size is None else int(max_list_size)

    def c_struct(self):
        return L.Index(self.nlist, self.max_list_size, self.list_offsets.data_ptr(),
                       self.list_sizes.data_ptr(), self.ids.data_ptr(), self.codes.data_ptr(),
                       self.scales.data_ptr())


def rslm_scan_topk_workspace(plan, index, Q, nprobe, k):
    cs = index.c_struct()
    return L.lib().rslm_scan_topk_workspace(plan.handle, C.byref(cs), Q, nprobe, k)


def rslm_scan_topk(plan, index, q_rot, probe_ids, probe_dots, k, out_scores=None, out_ids=None,
                   ws=None, stream=None):
    _need(q_rot, torch.float32, "q_rot")
    _need(probe_ids, torch.int32, "probe_ids")
    _need(probe_dots, torch.float32, "probe_dots")
    Q, nprobe = probe_ids.shape
    if out_scores is None:
        out_scores = torch.empty((Q, k), dtype=torch.float32, device=q_rot.device)
    if out_ids is None:
        out_ids = torch.empty((Q, k), dtype=torch.int32, device=q_rot.device)
    cs = index.c_struct()
    nb = L.lib().rslm_scan_topk_workspace(plan.handle, C.byref(cs), Q, nprobe, k)
    if ws is None:
        ws = _WS.get(nb, q_rot.device, "scan", stream)
    L.check("rslm_scan_topk", L.lib().rslm_scan_topk(
        plan.handle, C.byref(cs), _ptr(q_rot), Q, _ptr(probe_ids), _ptr(probe_dots), nprobe, k,
        _ptr(out_scores), _ptr(out_ids), _ptr(ws), ws.numel(), _stream(stream)))
    return out_scores, out_ids


def rslm_sq8_fit(v, lo=None, hi=None, accumulate=False, stream=None):
    _need(v, torch.float32, "v")
    n, dim = v.shape
    if lo is None:
        lo = torch.empty(dim, dtype=torch.float32, device=v.device)
    if hi is None:
        hi = torch.empty(dim, dtype=torch.float32, device=v.device)
    L.check("rslm_sq8_fit", L.lib().rslm_sq8_fit(_ptr(v), n, dim, _ptr(lo), _ptr(hi),
                                                 int(accumulate), _stream(stream)))
    return lo, hi


def rslm_sq8_encode(v, lo, hi, codes=None, dest_row=None, stream=None):
    _need(v, torch.float32, "v")
    _need(dest_row, torch.int32, "dest_row")
    n, dim = v.shape
    if codes is None:
        codes = torch.empty((n, dim), dtype=torch.uint8, device=v.device)
    _need(codes, torch.uint8, "codes")
    n_dest = codes.numel() // dim
    L.check("rslm_sq8_encode", L.lib().rslm_sq8_encode(_ptr(v), n, dim, _ptr(lo), _ptr(hi),
                                                       _ptr(dest_row), n_dest, _ptr(codes),
                                                       _stream(stream)))
    return codes


def rslm_rescore(codes2, lo, hi, q_rot, cand_scores, cand_ids, k_out, out_scores=None,
                 out_ids=None, stream=None):
    _need(codes2, torch.uint8, "codes2")
    _need(q_rot, torch.float32, "q_rot")
    _need(cand_scores, torch.float32, "cand_scores")
    _need(cand_ids, torch.int32, "cand_ids")
    Q, k_in = cand_ids.shape
    dim = q_rot.shape[1]
    if out_scores is None:
        out_scores = torch.empty((Q, k_out), dtype=torch.float32, device=q_rot.device)
    if out_ids is None:
        out_ids = torch.empty((Q, k_out), dtype=torch.int32, device=q_rot.device)
    codec = L.RescoreCodec(L.RSLM_RESCORE_SQ8, dim, codes2.numel() // dim, codes2.data_ptr(),
                           lo.data_ptr(), hi.data_ptr(), None, None)
    L.check("rslm_rescore", L.lib().rslm_rescore(C.byref(codec), _ptr(q_rot), Q,
                                                 _ptr(cand_scores), _ptr(cand_ids), k_in, k_out,
                                                 _ptr(out_scores), _ptr(out_ids),
                                                 _stream(stream)))
    return out_scores, out_ids


def rslm_rescore_rslm(plan2, codes2, scales2, q_rot, cand_scores, cand_ids, k_out,
                      out_scores=None, out_ids=None, stream=None):
    """``rslm_rescore`` with the RSLM rescoring codec (``rslm_encode_two_stage``
    records, indexed by vector id)."""
    _need(codes2, torch.uint8, "codes2")
    _need(scales2, torch.int32, "scales2")
    _need(q_rot, torch.float32, "q_rot")
    _need(cand_scores, torch.float32, "cand_scores")
    _need(cand_ids, torch.int32, "cand_ids")
    Q, k_in = cand_ids.shape
    if out_scores is None:
        out_scores = torch.empty((Q, k_out), dtype=torch.float32, device=q_rot.device)
    if out_ids is None:
        out_ids = torch.empty((Q, k_out), dtype=torch.int32, device=q_rot.device)
    n_vec = scales2.numel()
    if codes2.numel() < n_vec * plan2.canon_bytes:
        raise ValueError("codes2 smaller than scales2's vectors")
    codec = L.RescoreCodec(L.RSLM_RESCORE_RSLM, plan2.dim, n_vec, codes2.data_ptr(), None, None,
                           scales2.data_ptr(), plan2.handle.value)
    L.check("rslm_rescore", L.lib().rslm_rescore(C.byref(codec), _ptr(q_rot), Q,
                                                 _ptr(cand_scores), _ptr(cand_ids), k_in, k_out,
                                                 _ptr(out_scores), _ptr(out_ids),
                                                 _stream(stream)))
    return out_scores, out_ids
