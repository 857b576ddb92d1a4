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
sampled vectors, every returned score of two queries against the oracle's
encoding of those vectors, completeness over each query's best probed list,
and the rescored shortlist.  Oracle inputs are the seeded data (the mixture
generated on the host, the sweep's rows on the device by torch's generator and
copied back) and seeded centres; nothing the oracle consumes is produced by
the library.
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
    out = dict(R=R, plan=plan, xh=xh, cen=cen.cpu().numpy().astype(np.float64), q=q,
               index=index, assign=assign.cpu().numpy(), pos=F.record_positions(torch, index, MN),
               qrot=qrot.cpu().numpy(), pid=pid.cpu().numpy(), pdot=pdot.cpu().numpy(),
               s1=s1.cpu().numpy(), i1=i1.cpu().numpy(), s2=s2.cpu().numpy(),
               i2=i2.cpu().numpy(), Rm=H.rot(MD, 2), C=synth.codebook(4))
    yield out
    del out
    torch.cuda.empty_cache()


def _mid_oracle(f, i, ids):
    xs = f["xh"][ids].astype(np.float64)
    a, _ = oracle.assign_l2_expanded(xs, f["cen"])
    enc = oracle.encode(xs, f["Rm"], f["C"], 4, centroids=f["cen"][a], scale_mode="global")
    xt = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], f["C"], f["Rm"],
                            f["cen"][a])
    return a, xt @ f["q"][i].astype(np.float64), np.linalg.norm(xt, axis=1), xs


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
    a, exact, xn, _ = _mid_oracle(f, i, gi)
    assert np.mean([L in set(f["pid"][i].tolist()) for L in a]) >= 0.99
    F.check_scores(gs, exact, qn, xn)
    L = int(f["pid"][i][0])
    o = int(f["index"].list_offsets[L].item())
    n_l = int(f["index"].list_sizes[L].item())
    members = f["index"].ids[o:o + n_l].cpu().numpy().astype(np.int64)
    am, sm, xnm, _ = _mid_oracle(f, i, members)
    assert (am == L).mean() >= 0.99
    F.check_complete(members, am == L, sm, H.score_tol(sm, qn, xnm), gs[-1], set(gi.tolist()))


@pytest.mark.parametrize("i", [3, 200])
def test_mid_rescore_sampled(mid, i):
    f = mid
    ri, rs = f["i2"][i], f["s2"][i]
    assert set(ri.tolist()) <= set(f["i1"][i].tolist())
    F.check_topk_order(rs, ri, MK_OUT)
    cand = f["i1"][i]
    exact = f["xh"][cand].astype(np.float64) @ f["q"][i].astype(np.float64)
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

    def oracle_scores(i, ids_):
        xr = _rows(f, ids_)
        ao, _ = oracle.assign_l2_expanded(xr, f["cen"])
        e = oracle.encode(xr, f["Rm"], C, bits, centroids=f["cen"][ao], scale_mode="global")
        xt = oracle.reconstruct(e["codes"], e["s_code"], e["g_code"], C, f["Rm"], f["cen"][ao])
        return ao, xt @ f["q"][i].astype(np.float64), np.linalg.norm(xt, axis=1)

    # two queries: returned scores and completeness over the best probed list
    for i in (0, 211):
        gi, gs = i1[i], s1[i]
        F.check_topk_order(gs, gi, SK)
        qn = np.linalg.norm(f["q"][i])
        ao, exact, xn = oracle_scores(i, gi)
        F.check_scores(gs, exact, qn, xn, max_viol=1)
        L = int(f["pid"][i][0])
        o = int(index.list_offsets[L].item())
        n_l = int(index.list_sizes[L].item())
        members = index.ids[o:o + n_l].cpu().numpy().astype(np.int64)
        am, sm, xnm = oracle_scores(i, members)
        assert (am == L).mean() >= 0.99
        F.check_complete(members, am == L, sm, H.score_tol(sm, qn, xnm), gs[-1],
                         set(gi.tolist()))
    del index, pos
    torch.cuda.empty_cache()
