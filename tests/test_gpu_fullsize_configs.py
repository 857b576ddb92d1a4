"""Parity at the full sizes of the mid-size and bit-width-sweep workloads,
through the entry points the benchmark uses.

* Mid-size, non-power-of-two dimension: 1,000,000 x 96 unit-norm Gaussian
  mixture rows (1,024 components), 1,024 lists, 4-bit RSLM with global
  scaling and both rotation passes (the workload exercises the block-wise
  cascade: overlapping blocks, permutation and strided transpose), SQ8
  rescoring codes; a batch of 256 queries, nprobe = 32, top-100 from the
  scan, top-10 after rescoring.
* Bit-width sweep: 10,000,000 x 1,024 unit-norm anisotropic rows, 4,096
  lists, codes at 1, 2, 3 and 4 bits of the same data (global scaling, two
  passes); a batch of 256 queries, nprobe = 64, top-10.

The oracle checks sampled outputs it can compute one by one: the rotated
queries and probe lists of the batch, assignment, codes and scale codes of
sampled vectors, and for two queries the returned top-k against the oracle's
scores of every member of the probed lists (each returned id's score, and
completeness: every member scored above the returned k-th must be returned;
the sweep checks all 64 probed lists of its first query and the best 8 of
its second), and the rescored shortlist: SQ8 records against the oracle's
second residual, the rescoring against the decode of the stored records.
Oracle inputs are the seeded data (the mixture generated on the host, the
sweep's rows on the device by torch's generator and copied back) and seeded
centres; nothing the oracle consumes is produced by the library.
"""

import numpy as np
import pytest

import oracle
import synth
from tests import fullsize_common as F
from tests import helpers as H

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


# ------------------------------------------------------------------ mid-size
MN, MD, MNLIST, MQ, MNPROBE, MK, MK_OUT = 1_000_000, 96, 1024, 256, 32, 100, 10


@pytest.fixture(scope="module")
def mid():
    import paper_2608_30384_amd as R
    from paper_2608_30384_amd import ivf

    dev = torch.device("cuda", 0)
    xh = synth.gmix(MN, MD, 1024, seed=21)
    x = torch.from_numpy(xh).to(dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(5)
    cen = x[torch.randperm(MN, generator=gen, device=dev)[:MNLIST]].clone()
    plan = R.Plan(MD, 4, passes=2, scale_mode="global")
    resid = torch.empty_like(x)
    index, _, assign = ivf.build_index(plan, x, cen, resid_rot=resid)
    codes2, lo, hi = ivf.build_sq8(resid)
    del resid
    q = synth.queries_like("gmix", MQ, MD, data_seed=21, query_seed=22, n_comp=1024)
    qt = torch.from_numpy(q).to(dev)
    qrot = R.rslm_fwht(plan, qt)
    pid, pdot = R.ivf_assign_probe(qt, cen, MNPROBE, R.IVF_PROBE_IP)
    s1, i1 = R.rslm_scan_topk(plan, index, qrot, pid, pdot, MK)
    s2, i2 = R.rslm_rescore(codes2, lo, hi, qrot, s1, i1, MK_OUT)
    torch.cuda.synchronize()
    out = dict(R=R, plan=plan, xh=xh, cen=cen.cpu().numpy().astype(np.float64), q=q, cen_t=cen,
               crot=R.rslm_fwht(plan, cen), codes2=codes2, lo=lo.cpu().numpy(), hi=hi.cpu().numpy(),
               index=index, assign=assign.cpu().numpy(), pos=F.record_positions(torch, index, MN),
               qrot=qrot.cpu().numpy(), pid=pid.cpu().numpy(), pdot=pdot.cpu().numpy(),
               s1=s1.cpu().numpy(), i1=i1.cpu().numpy(), s2=s2.cpu().numpy(),
               i2=i2.cpu().numpy(), Rm=H.rot(MD, 2), C=synth.codebook(4))
    yield out
    del out
    torch.cuda.empty_cache()


def test_mid_rotation_and_probe(mid):
    f = mid
    qr = f["q"].astype(np.float64) @ f["Rm"].T
    assert np.all(np.abs(f["qrot"] - qr) <= 2e-6 * np.linalg.norm(f["q"], axis=1, keepdims=True))
    rid, _, dots = oracle.probe_ip(f["q"], f["cen"], MNPROBE)
    cmax = np.abs(f["cen"]).max()
    for i in range(MQ):
        tol = 1e-5 * np.linalg.norm(f["q"][i]) * cmax * np.sqrt(MD)
        assert np.all(np.abs(f["pdot"][i] - dots[i, f["pid"][i]]) <= tol)
        if set(f["pid"][i]) != set(rid[i]):
            srt = np.sort(dots[i])[::-1]
            assert srt[MNPROBE - 1] - srt[MNPROBE] <= 2 * tol


def test_mid_assign_and_encode_sampled(mid):
    f = mid
    ids = synth.random_rows(MN, 2000, seed=12)
    xs = f["xh"][ids].astype(np.float64)
    a, keep = F.check_assign(f["assign"][ids], xs, f["cen"])
    enc = oracle.encode(xs[keep], f["Rm"], f["C"], 4, centroids=f["cen"][a[keep]],
                        scale_mode="global")
    codes, sc = F.gpu_records(torch, f["R"], f["plan"], f["index"], f["pos"], ids[keep], 4, MD)
    ok = F.check_codes(codes, sc, enc, f["C"])
    assert ok.mean() > 0.98


@pytest.mark.parametrize("i", [3, 200])
def test_mid_scan_topk_sampled(mid, i):
    f = mid
    gi, gs = f["i1"][i], f["s1"][i]
    F.check_topk_order(gs, gi, MK)
    qn = np.linalg.norm(f["q"][i])
    members, lst = F.members_of(torch, f["index"], f["pid"][i])
    xs = f["xh"][members].astype(np.float64)
    best = lst == f["pid"][i][0]
    a, _ = oracle.assign_l2_expanded(xs[best], f["cen"])
    assert (a == f["pid"][i][0]).mean() >= 0.99
    sm, xnm, near, _ = F.oracle_member_scores(xs, lst, f["cen"], f["q"][i], f["Rm"], f["C"], 4)
    F.check_probed(gs, gi, members, sm, H.score_tol(sm, qn, xnm), near)


@pytest.mark.parametrize("i", [3, 200])
def test_mid_rescore_sampled(mid, i):
    f = mid
    ri, rs = f["i2"][i], f["s2"][i]
    cand, s1 = f["i1"][i], f["s1"][i].astype(np.float64)
    assert set(ri.tolist()) <= set(cand.tolist())
    F.check_topk_order(rs, ri, MK_OUT)
    qr = f["q"][i].astype(np.float64) @ f["Rm"].T
    lo, hi = f["lo"].astype(np.float64), f["hi"].astype(np.float64)
    step = (hi - lo) / 255.0
    t = torch.from_numpy(cand.astype(np.int64)).to(f["codes2"].device)
    c2 = f["codes2"][t].cpu().numpy()
    xs = f["xh"][cand].astype(np.float64)
    a, _ = oracle.assign_l2_expanded(xs, f["cen"])
    enc1 = oracle.encode(xs, f["Rm"], f["C"], 4, centroids=f["cen"][a], scale_mode="global")
    err, r2, same, _ = F.r2_error(f["R"], torch, f["plan"], xs, a, f["cen_t"], f["crot"], f["Rm"],
                               enc1, f["C"], f["cen"])
    same &= f["assign"][cand] == a
    assert same.mean() >= 0.95
    bound = F.r2_bound(xs, f["cen"][a])
    assert np.all(err[same] <= bound[same]), (err / bound).max()
    assert np.all(r2[same] >= lo - err[same, None]) and np.all(r2[same] <= hi + err[same, None])
    dec = lo + c2 * step
    slack = 0.5 * step * (1 + 1e-4) + err[:, None]
    assert np.all(np.abs(dec - r2)[same] <= slack[same])
    s2 = s1 + dec @ qr
    ref_s, ref_i = oracle.topk(s2, cand, MK_OUT)
    tol = 1e-5 * (np.abs(s2).max() + np.linalg.norm(qr))
    H.check_topk(rs, ri, ref_s, ref_i, lambda v: np.full(np.shape(v), tol), s2, cand)
    exact = xs @ f["q"][i].astype(np.float64)
    sel = np.array([np.nonzero(cand == v)[0][0] for v in ri])
    err1 = np.abs(f["s1"][i][sel] - exact[sel])
    err2 = np.abs(rs - exact[sel])
    assert np.median(err2) < 0.25 * np.median(err1)


# ------------------------------------------------------------------ bit-width sweep
SN, SD, SNLIST, SQ, SNPROBE, SK = 10_000_000, 1024, 4096, 256, 64, 10


@pytest.fixture(scope="module")
def sweep():
    import paper_2608_30384_amd as R
    from paper_2608_30384_amd import ivf

    dev = torch.device("cuda", 0)
    x = synth.aniso_torch(SN, SD, alpha=1.0, seed=100, normalize=True, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(9)
    cen = x[torch.randperm(SN, generator=gen, device=dev)[:SNLIST]].clone()
    assign, _ = R.ivf_assign_probe(x, cen, 1, R.IVF_ASSIGN_L2)
    q = synth.queries_like("aniso", SQ, SD, data_seed=100, query_seed=200, normalize=True)
    qt = torch.from_numpy(q).to(dev)
    pid, pdot = R.ivf_assign_probe(qt, cen, SNPROBE, R.IVF_PROBE_IP)
    torch.cuda.synchronize()
    out = dict(R=R, ivf=ivf, x=x, cent=cen, cen=cen.cpu().numpy().astype(np.float64), q=q, qt=qt,
               assign_t=assign, assign=assign.cpu().numpy(), pid_t=pid, pdot_t=pdot,
               pid=pid.cpu().numpy(), Rm=H.rot(SD, 2))
    yield out
    del out
    torch.cuda.empty_cache()


def _rows(f, ids):
    t = torch.from_numpy(np.asarray(ids, dtype=np.int64)).to(f["x"].device)
    return f["x"][t].cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_sweep_bits_sampled(sweep, bits):
    f = sweep
    R = f["R"]
    plan = R.Plan(SD, bits, passes=-1, scale_mode="global")
    assert plan.passes == 2
    index, _, _ = f["ivf"].build_index(plan, f["x"], f["cent"], assign=f["assign_t"])
    qrot = R.rslm_fwht(plan, f["qt"])
    s1, i1 = R.rslm_scan_topk(plan, index, qrot, f["pid_t"], f["pdot_t"], SK)
    s1, i1 = s1.cpu().numpy(), i1.cpu().numpy()
    pos = F.record_positions(torch, index, SN)
    C = synth.codebook(bits)
    K, g = C.shape
    n_sub = -(-SD // g)
    # codes and scales of sampled vectors
    ids = synth.random_rows(SN, 600, seed=13 + bits)
    xs = _rows(f, ids)
    a, keep = F.check_assign(f["assign"][ids], xs, f["cen"])
    enc = oracle.encode(xs[keep], f["Rm"], C, bits, centroids=f["cen"][a[keep]],
                        scale_mode="global")
    codes, sc = F.gpu_records(torch, R, plan, index, pos, ids[keep], bits, n_sub)
    assert F.check_codes(codes, sc, enc, C).mean() > 0.98

    # two queries: the returned top-10 against the oracle's scores of the
    # members of all probed lists (query 0) or of the best 8 (query 211)
    for i, n_lists in ((0, SNPROBE), (211, 8)):
        gi, gs = i1[i], s1[i]
        F.check_topk_order(gs, gi, SK)
        qn = np.linalg.norm(f["q"][i])
        members, lst = F.members_of(torch, index, f["pid"][i][:n_lists])
        xs = _rows(f, members)
        best = lst == f["pid"][i][0]
        ao, _ = oracle.assign_l2_expanded(xs[best], f["cen"])
        assert (ao == f["pid"][i][0]).mean() >= 0.99
        sm, xnm, near, _ = F.oracle_member_scores(xs, lst, f["cen"], f["q"][i], f["Rm"], C, bits)
        tolm = H.score_tol(sm, qn, xnm)
        if n_lists == SNPROBE:
            F.check_probed(gs, gi, members, sm, tolm, near)
        else:
            # only part of the candidates: the returned ids from these lists
            # pair with their scores, and none of these lists' members above
            # the returned k-th is missing
            inl = np.isin(gi, members)
            pos = {int(v): j for j, v in enumerate(members)}
            j = np.array([pos[int(v)] for v in gi[inl]], dtype=np.int64)
            assert not np.any((np.abs(gs[inl] - sm[j]) > tolm[j]) & ~near[j])
            above = np.nonzero(sm > gs[-1] + tolm)[0]
            missed = above[~np.isin(members[above], gi)]
            assert not np.any(~near[missed]) and len(missed) <= 3
    del index, pos
    torch.cuda.empty_cache()
