"""Parity at the text-embedding workload's full size, in the launch
configuration the benchmark times.

10,000,000 x 768 anisotropic Gaussian rows, 4,096 lists, 4-bit RSLM with
global scaling (two rotation passes), SQ8 rescoring codes, one batch of 256
queries, nprobe = 64, top-100 from the scan, top-10 after rescoring.  The
index is built and searched through the same entry points as ``bench.py``.

The oracle cannot redo the whole collection, so it checks sampled outputs it
can compute one by one:

* the rotated queries and the probe lists of the whole batch;
* assignment, codes and scale codes of 1,500 sampled vectors;
* for two queries, over every member of the query's 64 probed lists (about
  135,000 rows each, encoded by the oracle against their lists' centres):
  each returned id's score against the oracle's score of that id, and
  completeness (every member the oracle scores above the returned k-th
  score must have been returned); only rows in an encoding near-tie window
  may differ;
* rescoring: the SQ8 records of the shortlist against the oracle's second
  residual of those rows (within half a quantisation step plus the measured
  float32 error of the residual), the rescored scores against the SQ8
  decode of the stored records (score1 + <q_rot, lo + code * step>), with
  the (score desc, id asc) order and ids of that definition, and the
  rescored scores closer to the exact inner products than the scan's.

Oracle inputs are the seeded data (generated on the device by torch's
generator and copied to the host) and centres chosen as a seeded sample of
the rows; nothing the oracle consumes is produced by the library.
"""

import numpy as np
import pytest

import oracle
import synth
from tests import fullsize_common as F
from tests import helpers as H

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

N, D, NLIST, Q, NPROBE, K, K_OUT, BITS = 10_000_000, 768, 4096, 256, 64, 100, 10, 4


@pytest.fixture(scope="module")
def full():
    import paper_2608_30384_amd as R
    from paper_2608_30384_amd import ivf

    dev = torch.device("cuda", 0)
    x = synth.aniso_torch(N, D, alpha=1.0, seed=100, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(7)
    cen = x[torch.randperm(N, generator=gen, device=dev)[:NLIST]].clone()
    plan = R.Plan(D, BITS, passes=-1, scale_mode="global")
    assert plan.passes == 2
    resid = torch.empty_like(x)
    index, _, assign = ivf.build_index(plan, x, cen, resid_rot=resid)
    codes2, lo, hi = ivf.build_sq8(resid)
    del resid
    q = synth.queries_like("aniso", Q, D, data_seed=100, query_seed=200)
    qt = torch.from_numpy(q).to(dev)
    qrot = R.rslm_fwht(plan, qt)
    pid, pdot = R.ivf_assign_probe(qt, cen, NPROBE, R.IVF_PROBE_IP)
    s1, i1 = R.rslm_scan_topk(plan, index, qrot, pid, pdot, K)
    s2, i2 = R.rslm_rescore(codes2, lo, hi, qrot, s1, i1, K_OUT)
    torch.cuda.synchronize()
    # record position of every vector id
    ids_rec = index.ids.long()
    valid = ids_rec >= 0
    pos = torch.full((N,), -1, dtype=torch.int64, device=dev)
    pos[ids_rec[valid]] = torch.arange(ids_rec.numel(), device=dev)[valid]
    canon = R.rslm_unpack_codes(plan, index.codes, ids_rec.numel())
    out = dict(R=R, plan=plan, x=x, cen=cen.cpu().numpy().astype(np.float64), q=q, index=index,
               cen_t=cen, crot=R.rslm_fwht(plan, cen), codes2=codes2, lo=lo.cpu().numpy(),
               hi=hi.cpu().numpy(), assign=assign, pos=pos, canon=canon, qrot=qrot.cpu().numpy(),
               pid=pid.cpu().numpy(), pdot=pdot.cpu().numpy(), s1=s1.cpu().numpy(),
               i1=i1.cpu().numpy(), s2=s2.cpu().numpy(), i2=i2.cpu().numpy(),
               Rm=H.rot(D, 2), C=synth.codebook(BITS))
    yield out
    del out
    torch.cuda.empty_cache()


def _rows(f, ids):
    t = torch.from_numpy(np.asarray(ids, dtype=np.int64)).to(f["x"].device)
    return f["x"][t].cpu().numpy().astype(np.float64)


def _gpu_records(f, ids):
    """Codes (n, D) and decoded scales of the records holding vector ids."""
    t = torch.from_numpy(np.asarray(ids, dtype=np.int64)).to(f["x"].device)
    p = f["pos"][t]
    assert bool((p >= 0).all())
    canon = f["canon"][p].cpu().numpy()
    sc = f["index"].scales[p].cpu().numpy()
    codes = oracle.unpack_canonical(canon, BITS, D)
    sh, gh = H.dec_scales(sc)
    return codes, sc.astype(np.uint32), sh, gh


def test_rotation_and_probe_full_batch(full):
    f = full
    qr = f["q"].astype(np.float64) @ f["Rm"].T
    bound = 2e-6 * np.linalg.norm(f["q"], axis=1, keepdims=True)
    assert np.all(np.abs(f["qrot"] - qr) <= bound)
    rid, _, dots = oracle.probe_ip(f["q"], f["cen"], NPROBE)
    cmax = np.abs(f["cen"]).max()
    for i in range(Q):
        tol = 1e-5 * np.linalg.norm(f["q"][i]) * cmax * np.sqrt(D)
        assert np.all(np.abs(f["pdot"][i] - dots[i, f["pid"][i]]) <= tol)
        if set(f["pid"][i]) != set(rid[i]):
            srt = np.sort(dots[i])[::-1]
            assert srt[NPROBE - 1] - srt[NPROBE] <= 2 * tol


def test_assign_and_encode_sampled(full):
    f = full
    ids = synth.random_rows(N, 1500, seed=11)
    xs = _rows(f, ids)
    a, best = oracle.assign_l2_expanded(xs, f["cen"])
    ga = f["assign"][torch.from_numpy(ids).to(f["x"].device)].cpu().numpy()
    differ = np.nonzero(ga != a)[0]
    assert len(differ) <= 2
    for r in differ:   # only near-equidistant centres may disagree
        dg = ((xs[r] - f["cen"][ga[r]]) ** 2).sum()
        assert dg - best[r] <= 1e-4 * (1.0 + best[r])
    keep = ga == a
    enc = oracle.encode(xs[keep], f["Rm"], f["C"], BITS, centroids=f["cen"][a[keep]],
                        scale_mode="global")
    codes, sc, _, _ = _gpu_records(f, ids[keep])
    near = H.near_threshold(enc["u"], f["C"])
    flips = codes != enc["codes"]
    assert not np.any(flips & ~near)
    assert flips.sum() <= max(2, 1e-4 * flips.size)
    s_ok = (sc & 0xFFFF) == enc["s_code"]
    g_ok = (sc >> 16) == enc["g_code"]
    rows_flip = flips.any(1)
    s_near = H.near_rounding(enc["s"], oracle.dec_ue7m9, oracle.enc_ue7m9)
    g_near = H.near_rounding(enc["g"], oracle.dec_ue4m12, oracle.enc_ue4m12)
    assert np.all(s_ok | s_near | rows_flip)
    assert np.all(g_ok | g_near | rows_flip)
    assert np.all(np.abs((sc & 0xFFFF).astype(np.int64) - enc["s_code"].astype(np.int64)) <= 1)


@pytest.mark.parametrize("i", [0, 137])
def test_scan_topk_sampled(full, i):
    f = full
    gi, gs = f["i1"][i], f["s1"][i]
    F.check_topk_order(gs, gi, K)
    qn = np.linalg.norm(f["q"][i])
    members, lst = F.members_of(torch, f["index"], f["pid"][i])
    xs = _rows(f, members)
    # the oracle's own assignment agrees on the best probed list's members
    best = lst == f["pid"][i][0]
    a, _ = oracle.assign_l2_expanded(xs[best], f["cen"])
    assert (a == f["pid"][i][0]).mean() >= 0.99
    sm, xnm, near, _ = F.oracle_member_scores(xs, lst, f["cen"], f["q"][i], f["Rm"], f["C"], BITS)
    F.check_probed(gs, gi, members, sm, H.score_tol(sm, qn, xnm), near)


@pytest.mark.parametrize("i", [0, 137])
def test_rescore_sampled(full, i):
    f = full
    ri, rs = f["i2"][i], f["s2"][i]
    cand, s1 = f["i1"][i], f["s1"][i].astype(np.float64)
    assert set(ri.tolist()) <= set(cand.tolist())
    F.check_topk_order(rs, ri, K_OUT)
    qr = f["q"][i].astype(np.float64) @ f["Rm"].T
    lo, hi = f["lo"].astype(np.float64), f["hi"].astype(np.float64)
    step = (hi - lo) / 255.0
    t = torch.from_numpy(cand.astype(np.int64)).to(f["codes2"].device)
    c2 = f["codes2"][t].cpu().numpy()
    # the stored SQ8 records against the oracle's second residual of the rows
    xs = _rows(f, cand)
    a, _ = oracle.assign_l2_expanded(xs, f["cen"])
    enc1 = oracle.encode(xs, f["Rm"], f["C"], BITS, centroids=f["cen"][a], scale_mode="global")
    err, r2, same, _ = F.r2_error(f["R"], torch, f["plan"], xs, a, f["cen_t"], f["crot"], f["Rm"],
                               enc1, f["C"], f["cen"])
    same &= f["assign"][t].cpu().numpy() == a      # the stored records used the same list
    assert same.mean() >= 0.95
    bound = F.r2_bound(xs, f["cen"][a])
    assert np.all(err[same] <= bound[same]), (err / bound).max()
    assert np.all(r2[same] >= lo - err[same, None]) and np.all(r2[same] <= hi + err[same, None])
    dec = lo + c2 * step
    slack = 0.5 * step * (1 + 1e-4) + err[:, None]
    assert np.all(np.abs(dec - r2)[same] <= slack[same])
    # the rescoring kernel against the SQ8 decode of the stored records
    s2 = s1 + dec @ qr
    ref_s, ref_i = oracle.topk(s2, cand, K_OUT)
    tol = 1e-5 * (np.abs(s2).max() + np.linalg.norm(qr))
    H.check_topk(rs, ri, ref_s, ref_i, lambda v: np.full(np.shape(v), tol), s2, cand)
    # and it brings the scores closer to the exact inner products
    exact = xs @ f["q"][i].astype(np.float64)
    err1 = np.abs(s1 - exact)
    sel = np.array([np.nonzero(cand == v)[0][0] for v in ri])
    err2 = np.abs(rs - exact[sel])
    assert np.median(err2) < 0.25 * np.median(err1[sel])
