"""Parity of the RSLM rescoring codec on the GPU (two-stage relative coding,
Section "Relative Quantization") with the float64 oracle.

* ``rslm_encode_two_stage``: first-stage codes and scales as in
  ``rslm_encode``; second-stage codes and scale codes of the second residual
  compared with ``oracle.encode_rescore`` on every vector whose first stage
  agrees exactly (the second stage's input is then the same), with the
  near-tie and rounding-boundary allowances of the first stage.
* ``rslm_rescore`` with ``RSLM_RESCORE_RSLM``: records written by the oracle
  (packed canonically), shortlists with empty slots, every bit width and a
  ragged canonical record size; scores within 1e-4 relative and top-k ids
  identical except at near-ties.
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


TWO_CASES = [
    # D, bits1, passes, bits2, mode2, n
    (768, 4, 2, 2, "global", 700),    # text-embedding shape: register path
    (256, 4, 1, 2, "global", 333),    # register path, one pass
    (96, 4, 2, 2, "global", 517),     # overlap block: general path
    (128, 2, 1, 4, "global", 300),    # 2-D first stage, 1-D second stage
    (101, 3, 2, 1, "local", 300),     # ragged 4-D second stage, local scale
    (768, 4, 2, 3, "global", 200),    # 3-bit second stage: general path
    (2049, 4, 2, 2, "global", 150),   # odd D above 1,024: general path, overlap block
    (1536, 4, 2, 2, "local", 160),    # register path, 12 blocks
    (2048, 4, 2, 2, "global", 120),   # register path, 16 blocks
]


@pytest.mark.parametrize("D,bits1,passes,bits2,mode2,n", TWO_CASES)
def test_encode_two_stage_parity(R, D, bits1, passes, bits2, mode2, n):
    nlist = 6
    x = synth.aniso(n, D, seed=D + 31 * bits2)
    cen = x[np.random.default_rng(D).choice(n, nlist, replace=False)] * 0.9
    assign, _ = oracle.assign_l2(x, cen)
    Rm = H.rot(D, passes)
    C1, C2 = synth.codebook(bits1), synth.codebook(bits2)
    ref1 = oracle.encode(x, Rm, C1, bits1, centroids=cen[assign], scale_mode="global")
    ref2 = oracle.encode_rescore(x, Rm, ref1, C1, C2, bits2, centroids=cen[assign],
                                 scale_mode=mode2)
    plan = R.Plan(D, bits1, passes=passes, scale_mode="global")
    plan2 = R.Plan(D, bits2, passes=0, scale_mode=mode2)
    xt, ct = _t(x), _t(cen.astype(np.float32))
    crot = R.rslm_fwht(plan, ct)
    codes = torch.zeros(plan.code_bytes(n), dtype=torch.uint8, device=DEV)
    scales = torch.zeros(n, dtype=torch.int32, device=DEV)
    codes2 = torch.full((n, plan2.canon_bytes), 0xCD, dtype=torch.uint8, device=DEV)
    scales2 = torch.zeros(n, dtype=torch.int32, device=DEV)
    R.rslm_encode_two_stage(plan, plan2, xt, codes, scales, codes2, scales2,
                            rec_list=_t(assign, torch.int32), centroids=ct, centroids_rot=crot)
    # first stage
    g1 = oracle.unpack_canonical(R.rslm_unpack_codes(plan, codes, n).cpu().numpy(), bits1,
                                 ref1["codes"].shape[1])
    mism1 = g1 != ref1["codes"]
    assert not np.any(mism1 & ~H.near_threshold(ref1["u"], C1))
    sc = scales.cpu().numpy().astype(np.uint32)
    same1 = (~mism1.any(1)) & ((sc & 0xFFFF) == ref1["s_code"]) & ((sc >> 16) == ref1["g_code"])
    assert same1.mean() > 0.98, same1.mean()
    # second stage, on vectors whose first stage agrees
    g2 = oracle.unpack_canonical(codes2.cpu().numpy(), bits2, ref2["codes"].shape[1])
    mism2 = (g2 != ref2["codes"]) & same1[:, None]
    near2 = H.near_threshold(ref2["u"], C2)
    assert not np.any(mism2 & ~near2), np.argwhere(mism2 & ~near2)[:5]
    assert mism2.sum() <= max(2, 1e-4 * mism2.size)
    ok = same1 & ~mism2.any(1)
    sc2 = scales2.cpu().numpy().astype(np.uint32)
    su2, gu2 = sc2 & 0xFFFF, sc2 >> 16
    s_near = H.near_rounding(ref2["s"], oracle.dec_ue7m9, oracle.enc_ue7m9)
    bad = ok & ~s_near & (su2 != ref2["s_code"])
    assert not bad.any(), (np.where(bad), su2[bad], ref2["s_code"][bad])
    assert np.all(np.abs(su2[ok].astype(int) - ref2["s_code"][ok].astype(int)) <= 1)
    if mode2 == "global":
        g_near = H.near_rounding(ref2["g"], oracle.dec_ue4m12, oracle.enc_ue4m12)
        okg = ok & ~g_near & (su2 == ref2["s_code"])
        assert np.all(gu2[okg] == ref2["g_code"][okg]), np.where(gu2[okg] != ref2["g_code"][okg])
        assert np.all(np.abs(gu2[ok].astype(int) - ref2["g_code"][ok].astype(int)) <= 1)
    else:
        assert np.all(gu2 == 0x7000)


def test_encode_two_stage_padding_rows_and_zero_residual(R):
    """Padding records write nothing; a vector equal to its centre has a zero
    first residual, so R a = g^ R c and r2 = (1 - g^) R c (g^ = 1 here: r2 = 0,
    codes2 0 and s2^ 0)."""
    D = 768
    plan = R.Plan(D, 4, passes=2)
    plan2 = R.Plan(D, 2, passes=0)
    x = synth.aniso(24, D, seed=3)
    cen = x[:2].copy()
    rec_list = np.array([0, 1] + [0] * 22, dtype=np.int32)
    src = np.arange(24, dtype=np.int64)
    src[7] = -1
    xt, ct = _t(x), _t(cen)
    crot = R.rslm_fwht(plan, ct)
    codes = torch.zeros(plan.code_bytes(24), dtype=torch.uint8, device=DEV)
    scales = torch.zeros(24, dtype=torch.int32, device=DEV)
    codes2 = torch.full((24, plan2.canon_bytes), 0xAB, dtype=torch.uint8, device=DEV)
    scales2 = torch.full((24,), 777, dtype=torch.int32, device=DEV)
    R.rslm_encode_two_stage(plan, plan2, xt, codes, scales, codes2, scales2, n_records=24,
                            src_row=_t(src), rec_list=_t(rec_list), centroids=ct,
                            centroids_rot=crot)
    c2 = codes2.cpu().numpy()
    s2 = scales2.cpu().numpy().astype(np.uint32)
    assert s2[7] == 777 and np.all(c2[7] == 0xAB)            # padding row untouched
    assert np.all(c2[:2] == 0) and np.all(s2[:2] & 0xFFFF == 0)
    assert np.all(s2[:2] >> 16 == 0x7000)


def test_encode_two_stage_rejects_bad_plans(R):
    from paper_2608_30384_amd import _lib as L
    plan = R.Plan(96, 4, passes=2)
    x = _t(synth.aniso(16, 96, seed=1))
    codes = torch.zeros(plan.code_bytes(16), dtype=torch.uint8, device=DEV)
    scales = torch.zeros(16, dtype=torch.int32, device=DEV)
    for bad in (R.Plan(96, 2, passes=1), R.Plan(64, 2, passes=0)):
        codes2 = torch.zeros((16, bad.canon_bytes), dtype=torch.uint8, device=DEV)
        scales2 = torch.zeros(16, dtype=torch.int32, device=DEV)
        with pytest.raises(L.RslmError):
            R.rslm_encode_two_stage(plan, bad, x, codes, scales, codes2, scales2)


@pytest.mark.parametrize("D,bits2,k_in,k_out", [(768, 2, 100, 10), (96, 4, 100, 10),
                                                (101, 3, 37, 5), (98, 1, 1024, 1000),
                                                (100, 4, 7, 7)])
def test_rescore_rslm_parity(R, D, bits2, k_in, k_out):
    rng = np.random.default_rng(D + bits2)
    N, Q = 1500, 11
    # second-stage records from the oracle: random residual-like vectors
    # encoded against random bases in the rotated space (no rotation)
    x = synth.aniso(N, D, seed=D)
    base = x + 0.2 * rng.standard_normal((N, D)) / np.sqrt(D)
    C2 = synth.codebook(bits2)
    enc2 = oracle.encode(x, np.eye(D), C2, bits2, centroids=base, scale_mode="global")
    canon = oracle.pack_canonical(enc2["codes"], bits2)
    sc2 = (enc2["s_code"].astype(np.uint32) | (enc2["g_code"].astype(np.uint32) << 16))
    qr = rng.standard_normal((Q, D)).astype(np.float32)
    cand = np.stack([rng.choice(N, k_in, replace=False) for _ in range(Q)]).astype(np.int32)
    cand[0, 2:] = -1                                # a short shortlist
    cand[1, :] = -1                                 # an empty one
    s1 = (base[np.maximum(cand, 0)] * qr[:, None, :].astype(np.float64)).sum(-1)   # <q, a>
    s1 = s1.astype(np.float32)
    ref_s, ref_i = oracle.rescore_rslm(qr.astype(np.float64), s1, cand, enc2["codes"],
                                       enc2["s_code"], enc2["g_code"], C2, k_out)
    cands = oracle.rescore_rslm_scores(qr.astype(np.float64), s1, cand, enc2["codes"],
                                       enc2["s_code"], enc2["g_code"], C2)
    plan2 = R.Plan(D, bits2, passes=0, scale_mode="global")
    assert plan2.canon_bytes == canon.shape[1]
    gs, gi = R.rslm_rescore_rslm(plan2, _t(canon), _t(sc2.view(np.int32)), _t(qr), _t(s1),
                                 _t(cand), k_out)
    gs, gi = gs.cpu().numpy(), gi.cpu().numpy()
    assert np.all(gi[1] == -1) and np.all(np.isneginf(gs[1]))
    xt2 = oracle.reconstruct(enc2["codes"], enc2["s_code"], enc2["g_code"], C2, np.eye(D), base)
    xn = np.linalg.norm(xt2, axis=1).max()
    for i in range(Q):
        qn = np.linalg.norm(qr[i])
        H.check_topk(gs[i], gi[i], ref_s[i], ref_i[i], lambda s, qn=qn: H.score_tol(s, qn, xn),
                     *cands[i])


# 503 rows: the last wavefront holds three rows (its SQ8 ranges are prepared
# by the lanes that remain)
@pytest.mark.parametrize("D,passes,n,lite", [(768, 2, 500, False), (768, 2, 503, False),
                                             (256, 1, 300, False),
                                             (96, 2, 333, False), (768, 2, 400, True),
                                             (1536, 2, 200, False), (2048, 2, 150, True)])
def test_encode_sq8_parity(R, D, passes, n, lite):
    """rslm_encode_sq8: SQ8 codes of the rotated second residual written in the
    encoding pass, against the oracle's residual R x - R a quantised with the
    same float32 ranges; rows whose first stage agrees must match except at
    rounding midpoints (+-1 there)."""
    nlist = 5
    x = synth.aniso(n, D, seed=D + 7)
    cen = x[np.random.default_rng(D + 1).choice(n, nlist, replace=False)] * 0.9
    assign, _ = oracle.assign_l2(x, cen)
    Rm = H.rot(D, passes)
    C = synth.codebook(4)
    C8 = synth.codebook(3) if lite else None
    lead = oracle.lite_lead("global") if lite else 0
    ref = oracle.encode(x, Rm, C, 4, centroids=cen[assign], scale_mode="global", C_lead=C8)
    ra = oracle.first_stage_rotated(ref["codes"], ref["s_code"], ref["g_code"], C, Rm, cen[assign],
                                    C8, lead)
    r2 = x.astype(np.float64) @ Rm.T - ra
    lo, hi = oracle.sq8_fit(r2)
    lo32, hi32 = lo.astype(np.float32), hi.astype(np.float32)
    ref2 = oracle.sq8_encode(r2, lo32.astype(np.float64), hi32.astype(np.float64))
    plan = R.Plan(D, 4, passes=passes, scale_mode="global", lite=lite)
    xt, ct = _t(x), _t(cen.astype(np.float32))
    crot = R.rslm_fwht(plan, ct)
    codes = torch.zeros(plan.code_bytes(n), dtype=torch.uint8, device=DEV)
    scales = torch.zeros(n, dtype=torch.int32, device=DEV)
    codes2 = torch.full((n, D), 0xEE, dtype=torch.uint8, device=DEV)
    R.rslm_encode_sq8(plan, xt, codes, scales, _t(lo32), _t(hi32), codes2,
                      rec_list=_t(assign, torch.int32), centroids=ct, centroids_rot=crot)
    g1 = oracle.unpack_canonical(R.rslm_unpack_codes(plan, codes, n).cpu().numpy(), 4, D)
    if lite:
        g1[:, :lead] &= 7   # drop the embedded scale bits
    sc = scales.cpu().numpy().astype(np.uint32)
    same = ((g1 == ref["codes"]).all(1) & ((sc & 0xFFFF) == ref["s_code"]) &
            ((sc >> 16) == ref["g_code"]))
    assert same.mean() > 0.98
    got = codes2.cpu().numpy()
    step = (hi32.astype(np.float64) - lo32) / 255.0
    frac = (r2 - lo32) / np.where(step > 0, step, 1.0)
    near = np.abs(frac - np.floor(frac) - 0.5) < 1e-3
    d = np.abs(got.astype(int) - ref2.astype(int))[same]
    assert np.all(d <= 1)
    assert np.all((d == 0) | near[same])
    # the same codes as the two-call route (float residual, then SQ8)
    resid = torch.zeros((n, D), dtype=torch.float32, device=DEV)
    R.rslm_encode(plan, xt, codes, scales, rec_list=_t(assign, torch.int32), centroids=ct,
                  centroids_rot=crot, resid_rot=resid)
    two_call = R.rslm_sq8_encode(resid, _t(lo32), _t(hi32)).cpu().numpy()
    assert np.array_equal(got, two_call)
