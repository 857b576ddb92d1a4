"""Parity of packed records, Rslm4Lite encoding and OneToMany scoring on the
GPU with the float64 oracle.

* Rslm4Lite encoding (register and general encoders): codes, embedded
  scales and scale codes against ``oracle.encode(..., C_lead=...)`` with the
  near-tie and rounding-boundary allowances of the other encoder tests.
* ``rslm_pack_records``: byte-identical to ``oracle.pack_records`` of the
  library's own codes and scales (a pure layout operation).
* ``rslm_score``: records written by the oracle, scored for several queries,
  contiguous and gathered by ids (including ids outside the pool), against
  the oracle's LUT route with no partition centre; every bit width, local
  and global scales, Lite, ragged record sizes.
"""

import numpy as np
import pytest

import oracle
import synth
from tests import helpers as H

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def R():
    import paper_2608_30384_amd as R
    return R


def _t(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(DEV)


LITE_CASES = [(256, 1, "local", 333), (768, 2, "global", 300), (96, 2, "global", 200),
              (200, 2, "local", 150), (128, 1, "global", 170), (1536, 2, "global", 150)]


@pytest.mark.parametrize("D,passes,mode,n", LITE_CASES)
def test_lite_encode_parity(R, D, passes, mode, n):
    nlist = 4
    x = synth.aniso(n, D, seed=D + 3)
    cen = x[np.random.default_rng(D).choice(n, nlist, replace=False)] * 0.9
    assign, _ = oracle.assign_l2(x, cen)
    Rm = H.rot(D, passes)
    C16, C8 = synth.codebook(4), synth.codebook(3)
    lead = oracle.lite_lead(mode)
    ref = oracle.encode(x, Rm, C16, 4, centroids=cen[assign], scale_mode=mode, C_lead=C8)
    plan = R.Plan(D, 4, passes=passes, scale_mode=mode, lite=True)
    assert plan.lite and plan.record_bytes == oracle.record_bytes(D, 4, mode, lite=True)
    xt, ct = _t(x), _t(cen.astype(np.float32))
    crot = R.rslm_fwht(plan, ct)
    codes = torch.zeros(plan.code_bytes(n), dtype=torch.uint8, device=DEV)
    scales = torch.zeros(n, dtype=torch.int32, device=DEV)
    R.rslm_encode(plan, xt, codes, scales, rec_list=_t(assign, torch.int32), centroids=ct,
                  centroids_rot=crot)
    sc = scales.cpu().numpy().astype(np.uint32)
    su, gu = sc & 0xFFFF, sc >> 16
    recs = R.rslm_pack_records(plan, codes, scales, n).cpu().numpy()
    g, es, eg = oracle.unpack_records(recs, 4, D, mode, lite=True)
    # the embedded scales are the scale codes
    assert np.array_equal(es, su)
    if mode == "global":
        assert np.array_equal(eg, gu)
    # codes: leading coordinates on the K = 8 thresholds, the rest on K = 16
    u = ref["u"]
    near = H.near_threshold(u, C16)
    near[:, :lead] = H.near_threshold(u[:, :lead], C8)
    mism = g != ref["codes"]
    assert not np.any(mism & ~near), np.argwhere(mism & ~near)[:5]
    assert mism.sum() <= max(2, 1e-4 * mism.size)
    ok = ~mism.any(1)
    s_near = H.near_rounding(ref["s"], oracle.dec_ue7m9, oracle.enc_ue7m9)
    assert not np.any(ok & ~s_near & (su != ref["s_code"]))
    if mode == "global":
        g_near = H.near_rounding(ref["g"], oracle.dec_ue4m12, oracle.enc_ue4m12)
        okg = ok & ~g_near & (su == ref["s_code"])
        assert np.all(gu[okg] == ref["g_code"][okg])
    # packed records equal the oracle's packing of the library's codes
    assert np.array_equal(recs, oracle.pack_records(g, su, gu, 4, mode, lite=True))


@pytest.mark.parametrize("D,bits,mode", [(256, 4, "local"), (100, 1, "global"), (98, 2, "local"),
                                         (101, 3, "global")])
def test_pack_records_layout(R, D, bits, mode):
    n = 77
    x = synth.aniso(n, D, seed=D)
    plan = R.Plan(D, bits, passes=2, scale_mode=mode)
    codes = torch.zeros(plan.code_bytes(n), dtype=torch.uint8, device=DEV)
    scales = torch.zeros(n, dtype=torch.int32, device=DEV)
    R.rslm_encode(plan, _t(x), codes, scales)
    recs = R.rslm_pack_records(plan, codes, scales, n).cpu().numpy()
    assert recs.shape == (n, oracle.record_bytes(D, bits, mode))
    K, g = oracle.codec_shape(bits)
    canon = R.rslm_unpack_codes(plan, codes, n).cpu().numpy()
    c = oracle.unpack_canonical(canon, bits, -(-D // g))
    sc = scales.cpu().numpy().astype(np.uint32)
    assert np.array_equal(recs, oracle.pack_records(c, sc & 0xFFFF, sc >> 16, bits, mode))


SCORE_CASES = [
    # D, bits, mode, lite, n_pool, n (gathered), Q
    (256, 4, "local", False, 3000, 1000, 3),
    (256, 4, "local", True, 3000, 1000, 3),
    (768, 4, "global", True, 1200, 700, 2),
    (100, 1, "local", False, 2500, 900, 2),
    (98, 2, "global", False, 2000, 513, 4),
    (101, 3, "global", False, 2000, 777, 2),
    (101, 4, "local", False, 1500, 300, 1),
    (1536, 1, "global", False, 600, 333, 2),
    (2049, 4, "local", False, 300, 200, 2),     # query beyond the register path: LDS path
    (1100, 4, "global", True, 300, 150, 1),     # Lite on the LDS path
]


@pytest.mark.parametrize("D,bits,mode,lite,n_pool,n,Q", SCORE_CASES)
def test_score_parity(R, D, bits, mode, lite, n_pool, n, Q):
    rng = np.random.default_rng(D + bits + lite)
    x = synth.aniso(n_pool, D, seed=D + 1, normalize=(bits < 4))
    Rm = H.rot(D, 2)
    C = synth.codebook(bits)
    C8 = synth.codebook(3) if lite else None
    lead = oracle.lite_lead(mode) if lite else 0
    enc = oracle.encode(x, Rm, C, bits, scale_mode=mode, C_lead=C8)
    recs = oracle.pack_records(enc["codes"], enc["s_code"], enc["g_code"], bits, mode, lite)
    plan = R.Plan(D, bits, passes=2, scale_mode=mode, lite=lite)
    assert plan.record_bytes == recs.shape[1]
    q = synth.queries_like("aniso", Q, D, data_seed=D + 1, query_seed=9)
    qr = q.astype(np.float64) @ Rm.T
    sh, gh = H.dec_scales(enc["s_code"].astype(np.uint32) | (enc["g_code"].astype(np.uint32) << 16))
    ref = np.stack([oracle.scan_scores_lut(qr[i], 0.0, enc["codes"], sh, gh, C, C8, lead)
                    for i in range(Q)])
    xt = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], C, Rm, None, C8, lead)
    xn = np.linalg.norm(xt, axis=1)
    recs_t = _t(recs)
    qr_t = _t(qr.astype(np.float32))
    # contiguous: every record of the pool
    got = R.rslm_score(plan, recs_t, qr_t).cpu().numpy()
    for i in range(Q):
        tol = H.score_tol(ref[i], np.linalg.norm(q[i]), xn)
        assert np.all(np.abs(got[i] - ref[i]) <= tol), np.abs(got[i] - ref[i]).max()
    # gathered by ids, some outside the pool
    ids = rng.integers(0, n_pool, n).astype(np.int64)
    ids[:3] = [-1, n_pool, n_pool + 5]
    got = R.rslm_score(plan, recs_t, qr_t, ids=_t(ids)).cpu().numpy()
    assert np.all(np.isneginf(got[:, :3]))
    for i in range(Q):
        sel = ids[3:]
        tol = H.score_tol(ref[i][sel], np.linalg.norm(q[i]), xn[sel])
        assert np.all(np.abs(got[i, 3:] - ref[i][sel]) <= tol)


def test_lite_plan_is_rejected_by_the_rslm_rescoring_codec(R):
    """A Lite plan as the rescoring codec is not supported (status, no launch)."""
    from paper_2608_30384_amd import _lib as L
    plan = R.Plan(256, 4, passes=0, scale_mode="global", lite=True)
    codes2 = torch.zeros((4, plan.canon_bytes), dtype=torch.uint8, device=DEV)
    scales2 = torch.zeros(4, dtype=torch.int32, device=DEV)
    q = torch.zeros((1, 256), dtype=torch.float32, device=DEV)
    with pytest.raises(L.RslmError):
        R.rslm_rescore_rslm(plan, codes2, scales2, q, torch.zeros((1, 2), device=DEV),
                            torch.zeros((1, 2), dtype=torch.int32, device=DEV), 1)


DECODE_CASES = [(768, 4, 2, "global", False), (96, 4, 2, "local", False), (101, 3, 2, "global", False),
                (100, 1, 2, "global", False), (98, 2, 1, "local", False), (256, 4, 1, "global", True),
                (2049, 4, 2, "local", False), (64, 2, 0, "global", False)]


@pytest.mark.parametrize("D,bits,passes,mode,lite", DECODE_CASES)
def test_decode_parity(R, D, bits, passes, mode, lite):
    """rslm_decode (Decompress) against the oracle's reconstruction of the same
    codes and scales: x~ = g^ (c + R^T s^ C[code])."""
    n, nlist = 150, 5
    x = synth.aniso(n, D, seed=D + bits)
    cen = x[np.random.default_rng(D).choice(n, nlist, replace=False)] * 0.9
    assign, _ = oracle.assign_l2(x, cen)
    Rm = H.rot(D, passes)
    C = synth.codebook(bits)
    C8 = synth.codebook(3) if lite else None
    lead = oracle.lite_lead(mode) if lite else 0
    enc = oracle.encode(x, Rm, C, bits, centroids=cen[assign], scale_mode=mode, C_lead=C8)
    ref = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], C, Rm, cen[assign], C8,
                             lead)
    plan = R.Plan(D, bits, passes=passes, scale_mode=mode, lite=lite)
    codes = enc["codes"].copy()
    if lite:   # the scan layout carries the embedded scale bits as well
        for j in range(lead):
            w = enc["s_code"] if j < 16 else enc["g_code"]
            codes[:, j] |= ((w.astype(np.int64) >> (j % 16)) & 1) << 3
    tiles = R.rslm_pack_codes(plan, _t(oracle.pack_canonical(codes, bits)), n)
    sc = (enc["s_code"].astype(np.uint32) | (enc["g_code"].astype(np.uint32) << 16)).view(np.int32)
    got = R.rslm_decode(plan, tiles, _t(sc), n, rec_list=_t(assign, torch.int32),
                        centroids=_t(cen.astype(np.float32))).cpu().numpy()
    scale = np.maximum(np.linalg.norm(ref, axis=1), np.linalg.norm(cen[assign], axis=1))
    err = np.abs(got - ref).max(1)
    assert np.all(err <= 5e-6 * scale), (err / scale).max()


@pytest.mark.parametrize("D,passes,mode,k", [(768, 2, "global", 100), (256, 1, "local", 10),
                                             (128, 1, "global", 25), (1024, 2, "global", 10),
                                             # above D = 1,024: scored in passes, the scales
                                             # read again from chunk 0 in the last one
                                             (1536, 2, "global", 10), (1152, 2, "local", 17)])
def test_lite_ivf_scan_parity(R, D, passes, mode, k):
    """The IVF scan over Rslm4Lite records (scales read from the codes; no
    scales array) against the oracle's IVF search with the K = 8 leading
    codebook."""
    n, nlist, Q, nprobe = 2500, 9, 20, 3
    x = synth.aniso(n, D, seed=D + 11)
    cen = oracle.kmeans(x[:600], nlist, iters=4, seed=1)
    assign, _ = oracle.assign_l2(x, cen)
    Rm = H.rot(D, passes)
    C16, C8 = synth.codebook(4), synth.codebook(3)
    lead = oracle.lite_lead(mode)
    enc = oracle.encode(x, Rm, C16, 4, centroids=cen[assign], scale_mode=mode, C_lead=C8)
    # records of the lists, padded to whole tiles, codes with the embedded scales
    recs = oracle.pack_records(enc["codes"], enc["s_code"], enc["g_code"], 4, mode, lite=True)
    counts = np.bincount(assign, minlength=nlist)
    padded = (counts + 15) // 16 * 16
    offsets = np.concatenate([[0], np.cumsum(padded)[:-1]]).astype(np.int64)
    total = int(padded.sum())
    canon = np.zeros((total, recs.shape[1]), dtype=np.uint8)
    ids = np.full(total, -1, dtype=np.int32)
    fill = offsets.copy()
    for row in range(n):
        L = assign[row]
        canon[fill[L]] = recs[row]
        ids[fill[L]] = row
        fill[L] += 1
    plan = R.Plan(D, 4, passes=passes, scale_mode=mode, lite=True)
    tiles = R.rslm_pack_codes(plan, _t(canon), total)
    index = R.Index(_t(offsets), _t(counts.astype(np.int32)), _t(ids), tiles,
                    torch.zeros(1, dtype=torch.int32, device=DEV))
    sh, gh = H.dec_scales(enc["s_code"].astype(np.uint32) | (enc["g_code"].astype(np.uint32) << 16))
    lists = {L: {"ids": np.where(assign == L)[0], "codes": enc["codes"][assign == L],
                 "s_hat": sh[assign == L], "g_hat": gh[assign == L]} for L in range(nlist)}
    q = synth.queries_like("aniso", Q, D, data_seed=D + 11, query_seed=3)
    qr = q.astype(np.float64) @ Rm.T
    ref_s, ref_i, pid = oracle.ivf_search(q, qr, cen, lists, C16, nprobe, k, C8, lead)
    _, cands = oracle.ivf_candidates(q, qr, cen, lists, C16, nprobe, C8, lead)
    pdot = (q.astype(np.float64) @ cen.T)[np.arange(Q)[:, None], pid]
    gs, gi = R.rslm_scan_topk(plan, index, _t(qr.astype(np.float32)), _t(pid, torch.int32),
                              _t(pdot.astype(np.float32)), k)
    gs, gi = gs.cpu().numpy(), gi.cpu().numpy()
    xt = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], C16, Rm, cen[assign], C8,
                            lead)
    xn = np.linalg.norm(xt, axis=1).max()
    diffs = 0
    for i in range(Q):
        qn = np.linalg.norm(q[i])
        diffs += H.check_topk(gs[i], gi[i], ref_s[i], ref_i[i],
                              lambda s, qn=qn: H.score_tol(s, qn, xn), *cands[i])
    assert diffs <= max(1, Q // 10)


def test_scan_rejects_oversized_score_regions(R):
    """nprobe * max_list_size must not exceed 2^30 - 4 (a query's score region
    is read with 32-bit byte ranges of whole 16-byte groups): above it the
    call returns INVALID_ARG, at it the call gets as far as the workspace
    check; neither launches anything."""
    import ctypes as C
    from paper_2608_30384_amd import _lib as L
    plan = R.Plan(64, 4, passes=0, scale_mode="global")
    nlist, nprobe, Q, k = 64, 64, 1, 10
    buf = torch.zeros(4096, dtype=torch.int64, device=DEV)
    p = buf.data_ptr()
    q = torch.zeros((Q, 64), dtype=torch.float32, device=DEV)
    pid = torch.zeros((Q, nprobe), dtype=torch.int32, device=DEV)
    out = torch.zeros((Q, k), dtype=torch.float32, device=DEV)
    for np_, max_list, want in ((nprobe, (1 << 30) // nprobe, 1),
                                (nprobe, (1 << 30) // nprobe - 1, 4),
                                (1, (1 << 30) - 3, 1), (1, (1 << 30) - 4, 4)):
        idx = L.Index(nlist, max_list, p, p, p, p, p)
        st = L.lib().rslm_scan_topk(plan.handle, C.byref(idx), q.data_ptr(), Q, pid.data_ptr(),
                                    out.data_ptr(), np_, k, out.data_ptr(), pid.data_ptr(),
                                    p, 0, None)
        assert st == want, (np_, max_list, st)
    torch.cuda.synchronize()


def test_scan_rejects_misaligned_arrays(R):
    """Codes must be 16-byte aligned, list offsets 8-byte, the other arrays
    4-byte aligned: a misaligned pointer returns INVALID_ARG before any
    launch (pointers are only inspected, never dereferenced)."""
    import ctypes as C
    from paper_2608_30384_amd import _lib as L
    plan = R.Plan(64, 4, passes=0, scale_mode="global")
    nlist, nprobe, Q, k = 4, 2, 1, 10
    buf = torch.zeros(4096, dtype=torch.int64, device=DEV)
    p = buf.data_ptr()
    q = torch.zeros((Q, 64), dtype=torch.float32, device=DEV)
    pid = torch.zeros((Q, nprobe), dtype=torch.int32, device=DEV)
    out = torch.zeros((Q, k), dtype=torch.float32, device=DEV)
    for codes, scales, offs in ((p + 4, p, p), (p, p + 2, p), (p, p, p + 4)):
        idx = L.Index(nlist, 16, offs, p, p, codes, scales)
        st = L.lib().rslm_scan_topk(plan.handle, C.byref(idx), q.data_ptr(), Q, pid.data_ptr(),
                                    out.data_ptr(), nprobe, k, out.data_ptr(), pid.data_ptr(),
                                    p, 0, None)   # (a missed check stops at the workspace: 4)
        assert st == 1, (codes - p, scales - p, offs - p, st)
    torch.cuda.synchronize()


def test_unified_workspace_size_matches_the_scan_call(R):
    """rslm_workspace_size(RSLM_WS_SCAN_TOPK, ...) answers as
    rslm_scan_topk_workspace for a real plan and index."""
    import ctypes as C
    from paper_2608_30384_amd import _lib as L
    plan = R.Plan(768, 4, passes=2, scale_mode="global")
    buf = torch.zeros(64, dtype=torch.int64, device=DEV)
    p = buf.data_ptr()
    for nlist, max_list, Q, nprobe, k in ((4096, 3431, 256, 64, 100), (16, 40, 3, 2, 10)):
        idx = L.Index(nlist, max_list, p, p, p, p, p)
        want = L.lib().rslm_scan_topk_workspace(plan.handle, C.byref(idx), Q, nprobe, k)
        got = L.lib().rslm_workspace_size(0, plan.handle, C.byref(idx), Q, 0, 0, nprobe, k)
        assert want > 0 and got == want, (got, want)

