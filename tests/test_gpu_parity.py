"""Parity of the HIP path (through the C ABI) with the float64 oracle.

Inputs are seeded and synthetic; every expected value comes from ``oracle``.
Sizes span several tiles with ragged tails; the tolerance rules are the ones
stated for this path: rotation |dy| <= 2e-6 ||x||; codes bit-exact except
sub-vectors within 1e-5 of a decision threshold (at most 1e-4 of them);
scale codes exact except within 1e-5 of a rounding boundary; scores within
1e-4 relative (floor 1e-3 ||q|| ||x~||); top-k id sets identical except at
near-ties.
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


# ------------------------------------------------------------------ rotation
@pytest.mark.parametrize("D", [1, 4, 8, 64, 96, 98, 100, 101, 128, 256, 300, 768, 1024, 1536,
                               2048, 2049])
@pytest.mark.parametrize("passes", [0, 1, 2])
def test_fwht_forward_inverse(R, D, passes):
    plan = R.Plan(D, 4, passes=passes)
    assert plan.passes == passes
    x = np.random.default_rng(D * 3 + passes).standard_normal((37, D)).astype(np.float32)
    Rm = H.rot(D, passes)
    y = R.rslm_fwht(plan, _t(x)).cpu().numpy()
    ref = x.astype(np.float64) @ Rm.T
    bound = 2e-6 * np.linalg.norm(x, axis=1, keepdims=True)
    assert np.all(np.abs(y - ref) <= bound)
    xi = R.rslm_fwht(plan, _t(x), inverse=True).cpu().numpy()
    refi = x.astype(np.float64) @ Rm
    assert np.all(np.abs(xi - refi) <= bound)


def test_fwht_in_place_and_empty(R):
    plan = R.Plan(96, 4, passes=2)
    x = _t(np.random.default_rng(0).standard_normal((5, 96)).astype(np.float32))
    ref = R.rslm_fwht(plan, x.clone())
    R.rslm_fwht(plan, x, x)
    assert torch.equal(x, ref)
    R.rslm_fwht(plan, x[:0].contiguous())


def test_plan_info(R):
    plan = R.Plan(96, 4)
    assert plan.passes == 1          # the paper's rule: 4-bit, D <= 256
    assert plan.info.block == 64 and plan.info.n_full_blocks == 1
    assert abs(plan.emax - oracle.e_max(96)) < 1e-9
    for D in (1, 2, 768, 2049):
        assert abs(R.Plan(D, 2).emax - oracle.e_max(D)) < 1e-9
    assert R.Plan(1024, 1).canon_bytes == oracle.canonical_code_bytes(1024, 1)


# ------------------------------------------------------------------ packing
@pytest.mark.parametrize("bits,D", [(4, 96), (4, 768), (3, 101), (3, 1024), (2, 100), (2, 128),
                                    (1, 98), (1, 1024)])
def test_pack_unpack_roundtrip(R, bits, D):
    plan = R.Plan(D, bits, passes=2)
    n = 45
    rng = np.random.default_rng(bits * 100 + D)
    K, g = oracle.codec_shape(bits)
    codes = rng.integers(0, K, (n, -(-D // g)))
    canon = oracle.pack_canonical(codes, bits)
    assert canon.shape[1] == plan.canon_bytes
    tiles = R.rslm_pack_codes(plan, _t(canon), n)
    back = R.rslm_unpack_codes(plan, tiles, n).cpu().numpy()
    assert np.array_equal(back, canon)


# ------------------------------------------------------------------ encode
ENC_CASES = [
    # (D, bits, passes, mode)
    (128, 2, 1, "global"),     # the tiny configuration's codec
    (96, 4, 2, "global"),      # non-power-of-two, overlapping blocks
    (768, 4, 2, "global"),     # text-embedding shape
    (768, 4, 2, "local"),
    (101, 3, 2, "global"),
    (98, 1, 2, "local"),       # padded 4-D sub-vectors
    (1024, 1, 2, "global"),
    (1024, 3, 2, "global"),
    (256, 2, 2, "global"),
    (64, 4, 0, "global"),      # no rotation
    # above the register path: the paper's odd-D Compress shape (block-wise
    # cascade with the overlap block) and the 1,536-d text-embedding width
    (2049, 4, 2, "local"),
    (2049, 3, 2, "global"),
    (1536, 1, 2, "global"),
    (1536, 4, 2, "global"),    # register path, 12 blocks of 128
    (1536, 3, 2, "local"),
    (2048, 4, 2, "local"),     # register path, 16 blocks of 128
]


def _encode_inputs(D, n, nlist, seed):
    x = synth.aniso(n, D, seed=seed, normalize=False)
    cen = x[np.random.default_rng(seed).choice(n, nlist, replace=False)] * 0.9
    assign, _ = oracle.assign_l2(x, cen)
    return x, cen, assign


@pytest.mark.parametrize("D,bits,passes,mode", ENC_CASES)
def test_encode_parity(R, D, bits, passes, mode):
    n, nlist = 300, 7
    x, cen, assign = _encode_inputs(D, n, nlist, seed=D + bits)
    Rm = H.rot(D, passes)
    C = synth.codebook(bits)
    ref = oracle.encode(x, Rm, C, bits, centroids=cen[assign], scale_mode=mode)
    plan = R.Plan(D, bits, passes=passes, scale_mode=mode)
    xt, ct = _t(x), _t(cen.astype(np.float32))
    crot = R.rslm_fwht(plan, ct)
    codes = torch.zeros(plan.code_bytes(n), dtype=torch.uint8, device=DEV)
    scales = torch.zeros(n, dtype=torch.int32, device=DEV)
    resid = torch.zeros((n, D), dtype=torch.float32, device=DEV)
    R.rslm_encode(plan, xt, codes, scales, rec_list=_t(assign, torch.int32), centroids=ct,
                  centroids_rot=crot, resid_rot=resid)
    canon = R.rslm_unpack_codes(plan, codes, n).cpu().numpy()
    K, g = C.shape
    n_sub = -(-D // g)
    gcodes = oracle.unpack_canonical(canon, bits, n_sub)
    mism = gcodes != ref["codes"]
    near = H.near_threshold(ref["u"], C)
    assert not np.any(mism & ~near), np.argwhere(mism & ~near)[:5]
    assert mism.sum() <= max(2, 1e-4 * mism.size)
    rows_ok = ~mism.any(1)
    sc = scales.cpu().numpy().astype(np.uint32)
    su, gu = sc & 0xFFFF, sc >> 16
    s_near = H.near_rounding(ref["s"], oracle.dec_ue7m9, oracle.enc_ue7m9)
    bad = (su != ref["s_code"]) & rows_ok & ~s_near
    assert not bad.any(), (np.where(bad), su[bad], ref["s_code"][bad])
    assert np.all(np.abs(su.astype(int) - ref["s_code"].astype(int)) <= 1)
    if mode == "global":
        g_near = H.near_rounding(ref["g"], oracle.dec_ue4m12, oracle.enc_ue4m12)
        okg = rows_ok & ~g_near & (su == ref["s_code"])
        assert np.all(gu[okg] == ref["g_code"][okg])
        assert np.all(np.abs(gu.astype(int) - ref["g_code"].astype(int)) <= 1)
    else:
        assert np.all(gu == 0x7000)
    # rotated second residual R x - g^ (R c + s^ C[code]) on rows that agree
    sh, gh = H.dec_scales(sc)
    chat = C.astype(np.float64)[ref["codes"]].reshape(n, -1)[:, :D]
    rc = cen[assign] @ Rm.T
    r2 = x @ Rm.T - gh[:, None] * (rc + sh[:, None] * chat)
    ok = rows_ok & (su == ref["s_code"]) & (gu == ref["g_code"])
    err = np.abs(resid.cpu().numpy() - r2)[ok]
    assert np.all(err <= 5e-6 * np.linalg.norm(x[ok], axis=1, keepdims=True) + 1e-7)


def test_encode_zero_residual_and_padding_records(R):
    D = 96
    plan = R.Plan(D, 4, passes=2)
    x = synth.gmix(20, D, 4, seed=5)
    cen = x[:3].copy()
    rec_list = np.array([0, 1, 2] + [0] * 17, dtype=np.int32)
    src = np.arange(20, dtype=np.int64)
    src[5] = -1                                    # padding record
    xt, ct = _t(x), _t(cen)
    crot = R.rslm_fwht(plan, ct)
    codes = torch.full((plan.code_bytes(20),), 0xAB, dtype=torch.uint8, device=DEV)
    scales = torch.full((20,), 12345, dtype=torch.int32, device=DEV)
    R.rslm_encode(plan, xt, codes, scales, n_records=20, src_row=_t(src), rec_list=_t(rec_list),
                  centroids=ct, centroids_rot=crot)
    sc = scales.cpu().numpy().astype(np.uint32)
    canon = R.rslm_unpack_codes(plan, codes, 20).cpu().numpy()
    assert np.all(canon[:3] == 0) and np.all(sc[:3] & 0xFFFF == 0)   # x == c: R9
    assert np.all(sc[:3] >> 16 == 0x7000)                             # ||x|| / ||c|| = 1
    assert sc[5] == 12345                                             # padding untouched


# ------------------------------------------------------------------ routing
def _unaligned(a):
    """A device copy of a float32 matrix whose base is 4 bytes past a
    16-byte boundary (selects the kernel without 16-byte operand loads)."""
    flat = torch.empty(a.size + 1, dtype=torch.float32, device=DEV)
    flat[1:] = torch.from_numpy(np.ascontiguousarray(a).reshape(-1)).to(DEV)
    return flat[1:].view(a.shape)


# D % 4 == 0 with aligned rows runs the matrix-core kernel (128-row blocks,
# centre tiles of 128, k slabs of 32); other shapes the vector-ALU one
@pytest.mark.parametrize("D,nlist,n", [(96, 100, 700), (768, 257, 300), (128, 16, 1000),
                                       (36, 300, 1000), (4, 129, 131), (33, 70, 200),
                                       (100, 250, 700)])
@pytest.mark.parametrize("aligned", [True, False])
def test_assign_parity(R, D, nlist, n, aligned):
    rng = np.random.default_rng(D)
    x = synth.gmix(n, D, 32, seed=D)
    cen = x[rng.choice(n, nlist, replace=False)] + 0.01 * rng.standard_normal((nlist, D)).astype(np.float32)
    xt = _t(x) if aligned else _unaligned(x)
    ids, dist = R.ivf_assign_probe(xt, _t(cen.astype(np.float32)), 1, R.IVF_ASSIGN_L2)
    ids = ids.cpu().numpy()
    dist = dist.cpu().numpy()
    ref, best = oracle.assign_l2(x, cen.astype(np.float32))
    d_gpu_choice = ((x.astype(np.float64) - cen.astype(np.float32)[ids]) ** 2).sum(1)
    assert np.all((ids == ref) | (d_gpu_choice - best <= 1e-5 * (1 + best)))
    assert np.mean(ids == ref) > 0.99
    assert np.all(np.abs(dist - best) <= 1e-4 * (1 + np.abs(best)) + 1e-4 * (x * x).sum(1))


@pytest.mark.parametrize("D", [64, 33])
def test_assign_ties_take_the_lowest_id(R, D):
    """Exact duplicates of every centre (placed in other centre tiles and in
    the other half of a tile) give bit-identical distances: the lower id
    must win, as in the oracle's argmin."""
    rng = np.random.default_rng(5)
    base = rng.standard_normal((100, D)).astype(np.float32)
    perm = rng.permutation(300)
    cen = np.concatenate([base, base, base])[perm]
    x = synth.gmix(777, D, 16, seed=3)
    ids, _ = R.ivf_assign_probe(_t(x), _t(cen), 1, R.IVF_ASSIGN_L2)
    ids = ids.cpu().numpy()
    ref, best = oracle.assign_l2(x, cen)
    # the chosen centre's base row, and no duplicate of it with a lower id
    src = perm % 100
    for i, c in enumerate(ids):
        same = np.flatnonzero(src == src[c])
        assert c == same.min()
    d_gpu_choice = ((x.astype(np.float64) - cen[ids]) ** 2).sum(1)
    assert np.all((ids == ref) | (d_gpu_choice - best <= 1e-5 * (1 + best)))


@pytest.mark.parametrize("D,nlist,nprobe,Q", [(96, 300, 32, 50), (768, 4096, 64, 20), (128, 16, 4, 100),
                                              (64, 5000, 1, 7), (32, 100, 100, 3),
                                              # D not a multiple of 16; nlist above the
                                              # register-resident selection (16,384)
                                              (100, 700, 50, 9), (33, 40, 7, 5),
                                              (128, 20000, 128, 3),
                                              # >= 1,024 tiles of 128 x 128: the large-batch
                                              # kernel, ragged rows, centres and k slab
                                              (36, 16500, 40, 1000)])
def test_probe_parity(R, D, nlist, nprobe, Q):
    rng = np.random.default_rng(nlist)
    cen = rng.standard_normal((nlist, D)).astype(np.float32)
    q = rng.standard_normal((Q, D)).astype(np.float32)
    ids, dots = R.ivf_assign_probe(_t(q), _t(cen), nprobe, R.IVF_PROBE_IP)
    ids, dots = ids.cpu().numpy(), dots.cpu().numpy()
    rid, rdot, alldots = oracle.probe_ip(q, cen, nprobe)
    for i in range(Q):
        tol = 1e-5 * np.linalg.norm(q[i]) * np.abs(cen).max() * np.sqrt(D)
        assert len(set(ids[i])) == nprobe
        assert np.all(np.abs(dots[i] - alldots[i, ids[i]]) <= tol)
        if set(ids[i]) != set(rid[i]):
            srt = np.sort(alldots[i])[::-1]
            assert srt[nprobe - 1] - srt[nprobe] <= 2 * tol
        # ordered by (dot desc, id asc) in the returned dots
        for a, b in zip(range(nprobe - 1), range(1, nprobe)):
            assert dots[i, a] > dots[i, b] or (dots[i, a] == dots[i, b] and ids[i, a] < ids[i, b])


@pytest.mark.parametrize("n_equal", [3000, 40])
def test_probe_ties(R, n_equal):
    """Equal dots are ordered by list id: n_equal identical centres (more than
    the selection buffer when 3000) among distinct ones."""
    D, nlist, nprobe, Q = 64, 4000, 64, 4
    rng = np.random.default_rng(n_equal)
    cen = rng.standard_normal((nlist, D)).astype(np.float32) * 0.01
    dup = rng.choice(nlist, n_equal, replace=False)
    cen[dup] = 1.0
    q = np.ones((Q, D), np.float32)
    ids, dots = R.ivf_assign_probe(_t(q), _t(cen), nprobe, R.IVF_PROBE_IP)
    ids = ids.cpu().numpy()
    want = np.sort(dup)[:nprobe] if n_equal >= nprobe else None
    for i in range(Q):
        if want is not None:
            assert np.array_equal(ids[i], want)
        else:
            assert np.array_equal(ids[i, :n_equal], np.sort(dup))


# ------------------------------------------------------------------ scan
def _oracle_index(D, bits, passes, mode, n, nlist, seed, list_skew=False):
    """Oracle-encoded collection grouped into lists (all on the host)."""
    x = synth.gmix(n, D, 24, seed=seed)
    rng = np.random.default_rng(seed)
    cen = x[rng.choice(n, nlist, replace=False)].astype(np.float64)
    if list_skew:
        assign = np.minimum((rng.random(n) ** 3 * nlist).astype(np.int64), nlist - 1)
    else:
        assign, _ = oracle.assign_l2(x, cen)
    Rm = H.rot(D, passes)
    C = synth.codebook(bits)
    enc = oracle.encode(x, Rm, C, bits, centroids=cen[assign], scale_mode=mode)
    return x, cen, assign, Rm, C, enc


def _device_index(R, plan, enc, assign, nlist, bits):
    """Canonical oracle codes -> librslm tile layout (rslm_pack_codes)."""
    n = len(assign)
    order = np.argsort(assign, kind="stable")
    counts = np.bincount(assign, minlength=nlist)
    padded = (counts + 15) // 16 * 16
    offsets = np.concatenate([[0], np.cumsum(padded)[:-1]]).astype(np.int64)
    total = int(padded.sum())
    canon = oracle.pack_canonical(enc["codes"], bits)
    canon_rec = np.zeros((total, canon.shape[1]), dtype=np.uint8)
    scales = np.zeros(total, dtype=np.uint32)
    ids = np.full(total, -1, dtype=np.int32)
    starts = np.concatenate([[0], np.cumsum(counts)[:-1]])
    for j, row in enumerate(order):
        L = assign[row]
        r = offsets[L] + (j - starts[L])
        canon_rec[r] = canon[row]
        scales[r] = int(enc["s_code"][row]) | (int(enc["g_code"][row]) << 16)
        ids[r] = row
    tiles = R.rslm_pack_codes(plan, _t(canon_rec), total)
    return R.Index(_t(offsets), _t(counts.astype(np.int32)), _t(ids), tiles,
                   _t(scales.view(np.int32)))


def _oracle_lists(enc, assign, nlist):
    sh, gh = H.dec_scales(enc["s_code"].astype(np.uint32) | (enc["g_code"].astype(np.uint32) << 16))
    out = {}
    for L in range(nlist):
        sel = np.where(assign == L)[0]
        out[L] = {"ids": sel, "codes": enc["codes"][sel], "s_hat": sh[sel], "g_hat": gh[sel]}
    return out


SCAN_CASES = [
    # D, bits, passes, mode, n, nlist, Q, nprobe, k, skew
    (128, 2, 1, "global", 3000, 16, 40, 4, 10, False),     # tiny-config shape
    (96, 4, 2, "global", 4000, 12, 30, 6, 100, True),      # big skewed lists: several chunks
    (768, 4, 2, "global", 2500, 9, 20, 3, 100, False),
    (768, 4, 2, "local", 1200, 5, 9, 5, 17, False),
    (100, 1, 2, "global", 2000, 10, 25, 4, 10, False),
    (101, 3, 2, "global", 2000, 10, 25, 4, 10, False),
    (1024, 4, 2, "global", 900, 6, 12, 3, 10, False),     # 32 chunks at 4 bits: 256 VGPRs
    (1024, 3, 2, "global", 900, 6, 12, 2, 10, False),
    (1024, 1, 2, "global", 900, 6, 12, 6, 1, False),
    (256, 2, 2, "local", 1500, 30, 50, 30, 1000, False),   # k larger than most candidate sets
    (64, 4, 1, "global", 30000, 20000, 8, 50, 10, True),   # > 16,384 lists: planned in two
                                                           # passes, many lists empty
    # D > 1,024: the chunks are scored in passes (48 chunks: 2 x 24; 2049 -> 72: 3 x 24;
    # 3-bit 1100 -> 48: 3 x 16; 2-bit 2048: 4 x 16; 1-bit 3072: 6 x 16)
    (1536, 4, 2, "global", 900, 6, 12, 3, 10, False),
    (2049, 4, 2, "local", 700, 5, 10, 2, 17, False),
    (1100, 3, 2, "global", 700, 5, 10, 2, 10, False),
    (2048, 2, 2, "global", 600, 5, 10, 3, 10, False),
    (3072, 1, 2, "global", 500, 4, 8, 2, 10, False),
    (1536, 4, 2, "global", 9000, 3, 8, 2, 100, True),      # lists of several chunks, in passes
    # 1- and 2-bit codes decoded by whole bytes (24 chunks and more, passes of 24)
    (1024, 2, 2, "global", 900, 6, 12, 3, 10, False),
    (768, 1, 2, "local", 900, 6, 12, 4, 10, False),
    (1536, 2, 2, "global", 600, 5, 10, 3, 10, False),
]


@pytest.mark.parametrize("D,bits,passes,mode,n,nlist,Q,nprobe,k,skew", SCAN_CASES)
def test_scan_topk_parity(R, D, bits, passes, mode, n, nlist, Q, nprobe, k, skew):
    x, cen, assign, Rm, C, enc = _oracle_index(D, bits, passes, mode, n, nlist, seed=D * 7 + bits,
                                               list_skew=skew)
    plan = R.Plan(D, bits, passes=passes, scale_mode=mode)
    index = _device_index(R, plan, enc, assign, nlist, bits)
    q = synth.queries_like("gmix", Q, D, data_seed=D * 7 + bits, n_comp=24)
    qr = q.astype(np.float64) @ Rm.T
    lists = _oracle_lists(enc, assign, nlist)
    ref_s, ref_i, pid = oracle.ivf_search(q, qr, cen, lists, C, nprobe, k)
    _, cands = oracle.ivf_candidates(q, qr, cen, lists, C, nprobe)
    pdot = (q.astype(np.float64) @ cen.T)[np.arange(Q)[:, None], pid]
    gs, gi = R.rslm_scan_topk(plan, index, _t(qr.astype(np.float32)), _t(pid, torch.int32),
                              _t(pdot.astype(np.float32)), k)
    gs, gi = gs.cpu().numpy(), gi.cpu().numpy()
    xt = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], C, Rm, cen[assign])
    xn = np.linalg.norm(xt, axis=1).max()
    diffs = 0
    for i in range(Q):
        qn = np.linalg.norm(q[i])
        diffs += H.check_topk(gs[i], gi[i], ref_s[i], ref_i[i],
                              lambda s, qn=qn: H.score_tol(s, qn, xn), *cands[i])
    assert diffs <= max(1, Q // 10)


# ------------------------------------------------------------------ SQ8 + rescore
def test_sq8_parity(R):
    rng = np.random.default_rng(3)
    v = (rng.standard_normal((3001, 97)) * rng.uniform(0.01, 2, 97)).astype(np.float32)
    v[:, 5] = 0.5
    lo, hi = R.rslm_sq8_fit(_t(v))
    rlo, rhi = oracle.sq8_fit(v)
    assert np.array_equal(lo.cpu().numpy(), rlo.astype(np.float32))
    assert np.array_equal(hi.cpu().numpy(), rhi.astype(np.float32))
    codes = R.rslm_sq8_encode(_t(v), lo, hi).cpu().numpy()
    ref = oracle.sq8_encode(v, rlo, rhi)
    step = (rhi - rlo) / 255
    frac = np.where(step > 0, (v - rlo) / np.where(step > 0, step, 1), 0)
    near = np.abs(frac - np.floor(frac) - 0.5) < 1e-4
    assert np.all((codes == ref) | near)
    assert np.all(np.abs(codes.astype(int) - ref.astype(int)) <= 1)
    # accumulate folds a second batch in
    lo2, hi2 = R.rslm_sq8_fit(_t(v[:10] * 3), lo.clone(), hi.clone(), accumulate=True)
    assert np.array_equal(lo2.cpu().numpy(), np.minimum(rlo, (v[:10] * 3).min(0)).astype(np.float32))


@pytest.mark.parametrize("D,k_in,k_out", [(96, 100, 10), (768, 100, 10), (33, 7, 7), (768, 1024, 1)])
def test_rescore_parity(R, D, k_in, k_out):
    rng = np.random.default_rng(D + k_in)
    N, Q = 2000, 13
    r2 = (rng.standard_normal((N, D)) * 0.05).astype(np.float32)
    lo, hi = oracle.sq8_fit(r2)
    codes2 = oracle.sq8_encode(r2, lo, hi)
    qr = rng.standard_normal((Q, D)).astype(np.float32)
    cand = np.stack([rng.choice(N, k_in, replace=False) for _ in range(Q)]).astype(np.int32)
    cand[0, 3:] = -1                              # a short shortlist
    s1 = rng.standard_normal((Q, k_in)).astype(np.float32)
    ref_s, ref_i = oracle.rescore_sq8(qr.astype(np.float64), s1, cand, codes2, lo, hi, k_out)
    cands = oracle.rescore_sq8_scores(qr.astype(np.float64), s1, cand, codes2, lo, hi)
    gs, gi = R.rslm_rescore(_t(codes2), _t(lo.astype(np.float32)), _t(hi.astype(np.float32)),
                            _t(qr), _t(s1), _t(cand), k_out)
    gs, gi = gs.cpu().numpy(), gi.cpu().numpy()
    for i in range(Q):
        t = 1e-5 * (np.abs(ref_s[i][np.isfinite(ref_s[i])]).max() + np.linalg.norm(qr[i]))
        H.check_topk(gs[i], gi[i], ref_s[i], ref_i[i], lambda s, t=t: np.full(np.shape(s), t),
                     *cands[i])


# ------------------------------------------------------------------ end to end, tiny config
def test_end_to_end_tiny_config(R):
    """10,000 x 128 Gaussian mixture, 16 lists (k-means 10 it, seed 0), 2-bit
    Lloyd-Max with one rotation pass, 100 queries, nprobe 4, top-10."""
    N, D, nlist, Q, nprobe, k = 10000, 128, 16, 100, 4, 10
    x = synth.gmix(N, D, 16, seed=100)
    q = synth.queries_like("gmix", Q, D, data_seed=100, n_comp=16)
    cen = oracle.kmeans(x, nlist, iters=10, seed=0)
    assign, _ = oracle.assign_l2(x, cen)
    Rm = H.rot(D, 1)
    C = synth.codebook(2)
    enc = oracle.encode(x, Rm, C, 2, centroids=cen[assign], scale_mode="global")
    lists = _oracle_lists(enc, assign, nlist)
    ref_s, ref_i, ref_p = oracle.ivf_search(q, q.astype(np.float64) @ Rm.T, cen, lists, C, nprobe, k)

    plan = R.Plan(D, 2, passes=1, scale_mode="global")
    xt, ct, qt = _t(x), _t(cen.astype(np.float32)), _t(q)
    from paper_2608_30384_amd import ivf
    index, crot, gassign = ivf.build_index(plan, xt, ct)
    assert np.mean(gassign.cpu().numpy() == assign) > 0.999
    qrot = R.rslm_fwht(plan, qt)
    pid, pdot = R.ivf_assign_probe(qt, ct, nprobe, R.IVF_PROBE_IP)
    assert np.mean(np.sort(pid.cpu().numpy(), 1) == np.sort(ref_p, 1)) > 0.99
    gs, gi = R.rslm_scan_topk(plan, index, qrot, pid, pdot, k)
    gs, gi = gs.cpu().numpy(), gi.cpu().numpy()
    # encode agreement on the whole collection
    canon_gpu = R.rslm_unpack_codes(plan, index.codes, index.ids.numel()).cpu().numpy()
    ids_rec = index.ids.cpu().numpy()
    ok = ids_rec >= 0
    gcodes = oracle.unpack_canonical(canon_gpu[ok], 2, D // 2)
    assert np.mean(gcodes == enc["codes"][ids_rec[ok]]) > 1 - 1e-4
    xt_o = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], C, Rm, cen[assign])
    recall = np.mean([len(set(gi[i]) & set(ref_i[i])) / k for i in range(Q)])
    assert recall >= 0.99
    # scores of the returned ids against the oracle's reconstruction; a
    # tolerated code flip near a threshold may move a score beyond 1e-4
    viol = 0
    for i in range(Q):
        exact = xt_o[gi[i]] @ q[i].astype(np.float64)
        tol = H.score_tol(exact, np.linalg.norm(q[i]), np.linalg.norm(xt_o[gi[i]], axis=1))
        viol += int(np.sum(np.abs(gs[i] - exact) > tol))
    assert viol <= 0.01 * Q * k


# ------------------------------------------------------------------ large / tied top-k
def _scan_vs_oracle(R, D, bits, passes, x, cen, assign, q, nprobe, k, max_list=None):
    Rm = H.rot(D, passes)
    C = synth.codebook(bits)
    enc = oracle.encode(x, Rm, C, bits, centroids=cen[assign], scale_mode="global")
    nlist = len(cen)
    plan = R.Plan(D, bits, passes=passes, scale_mode="global")
    index = _device_index(R, plan, enc, assign, nlist, bits)
    if max_list is not None:   # a looser bound: wider score regions, same results
        index.max_list_size = max(index.max_list_size, max_list)
    qr = q.astype(np.float64) @ Rm.T
    lists = _oracle_lists(enc, assign, nlist)
    ref_s, ref_i, pid = oracle.ivf_search(q, qr, cen, lists, C, nprobe, k)
    _, cands = oracle.ivf_candidates(q, qr, cen, lists, C, nprobe)
    pdot = (q.astype(np.float64) @ cen.T)[np.arange(len(q))[:, None], pid]
    gs, gi = R.rslm_scan_topk(plan, index, _t(qr.astype(np.float32)), _t(pid, torch.int32),
                              _t(pdot.astype(np.float32)), k)
    return gs.cpu().numpy(), gi.cpu().numpy(), ref_s, ref_i, enc, Rm, C, cands


# max_list: a looser bound on the list sizes (wider per-query score regions,
# the same results)
@pytest.mark.parametrize("max_list", [None, 100_000])
def test_scan_topk_large_candidate_sets(R, max_list):
    """~70,000 candidates per query: the streaming threshold selection."""
    D, bits, n, nlist, Q, nprobe, k = 64, 4, 90000, 9, 6, 7, 100
    x = synth.gmix(n, D, 12, seed=77)
    rng = np.random.default_rng(77)
    cen = x[rng.choice(n, nlist, replace=False)].astype(np.float64)
    assign, _ = oracle.assign_l2(x, cen)
    q = synth.queries_like("gmix", Q, D, data_seed=77, n_comp=12)
    gs, gi, ref_s, ref_i, enc, Rm, C, cands = _scan_vs_oracle(R, D, bits, 2, x, cen, assign, q,
                                                              nprobe, k, max_list)
    xt = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], C, Rm, cen[assign])
    xn = np.linalg.norm(xt, axis=1).max()
    diffs = 0
    for i in range(Q):
        qn = np.linalg.norm(q[i])
        diffs += H.check_topk(gs[i], gi[i], ref_s[i], ref_i[i],
                              lambda s, qn=qn: H.score_tol(s, qn, xn), *cands[i])
    assert diffs <= 1


@pytest.mark.parametrize("max_list", [None, 150_000])
def test_scan_topk_exact_ties(R, max_list):
    """60,000 identical top candidates: the k lowest ids must win.  Every
    top-k slice then holds more tied scores than its sort buffer, so the
    radix selection with the id tie-break runs."""
    D, bits, nlist, Q, nprobe, k = 64, 4, 4, 3, 4, 100
    N = 70000
    base = synth.gmix(N, D, 6, seed=91)
    q = synth.queries_like("gmix", Q, D, data_seed=91, n_comp=6)
    star = q[0] / np.linalg.norm(q[0]) * 3.0          # far above every other candidate for q0
    x = base.copy()
    dup = np.random.default_rng(91).choice(N, 60000, replace=False)
    x[dup] = star.astype(np.float32)
    rng = np.random.default_rng(91)
    cen = np.vstack([x[rng.choice(N, nlist - 1, replace=False)], star[None]]).astype(np.float64)
    assign, _ = oracle.assign_l2(x, cen)
    gs, gi, ref_s, ref_i, enc, Rm, C, cands = _scan_vs_oracle(R, D, bits, 2, x, cen, assign, q,
                                                              nprobe, k, max_list)
    assert np.array_equal(gi[0], np.sort(dup)[:k])
    assert np.array_equal(ref_i[0], gi[0])
    assert np.all(gs[0] == gs[0][0])
    xt = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], C, Rm, cen[assign])
    xn = np.linalg.norm(xt, axis=1).max()
    for i in range(Q):
        qn = np.linalg.norm(q[i])
        H.check_topk(gs[i], gi[i], ref_s[i], ref_i[i], lambda s, qn=qn: H.score_tol(s, qn, xn),
                     *cands[i])
