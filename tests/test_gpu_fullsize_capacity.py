"""Parity at the capacity workload's full size, built and searched the way the
benchmark does.

100,000,000 x 768 anisotropic rows (never resident as float32: generated in
blocks of 2^22 rows from a per-block seeded device generator), 16,384 lists
(k-means on the first 4,194,304 rows), 4-bit RSLM scan records and 2-bit RSLM
rescoring records written by the blocked two-stage encode; one batch of 1,024
queries, nprobe = 128, top-100 from the scan, RSLM rescoring to top-10.

The oracle checks sampled outputs it can compute one by one: assignment, both
stages' codes and scale codes of sampled rows (the second stage's near-tie
windows derived from the measured float32 error of its input, checked against
its bound), for two queries every returned score against the oracle's
encoding of that vector and completeness over the members of the query's 16
best probed lists, and the rescored top-10 against the oracle's RSLM
rescoring of the same shortlist.  Sampled rows are copied from the regenerated
blocks; nothing the oracle consumes is produced by the library.
"""

import numpy as np
import pytest

import oracle
import synth
from tests import fullsize_common as F
from tests import helpers as H

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

N, D, NLIST, Q, NPROBE, K, K_OUT = 100_000_000, 768, 16384, 1024, 128, 100, 10
BLK = synth.TORCH_BLOCK


@pytest.fixture(scope="module")
def cap():
    import paper_2608_30384_amd as R
    from paper_2608_30384_amd import ivf

    dev = torch.device("cuda", 0)
    plan = R.Plan(D, 4, passes=-1, scale_mode="global")
    plan2 = R.Plan(D, 2, passes=0, scale_mode="global")
    xb = torch.empty((BLK, D), dtype=torch.float32, device=dev)

    def block(b):
        synth.aniso_torch_block(b, D, seed=100, out=xb)
        return xb[:min(BLK, N - b * BLK)]

    cen = ivf.kmeans(block(0)[:256 * NLIST].contiguous(), NLIST, iters=10, seed=0)
    sample = synth.random_rows(N, 500, seed=17)
    rows = {}

    def keep_rows(b, xs):
        sel = sample[(sample >= b * BLK) & (sample < b * BLK + len(xs))]
        if len(sel):
            t = torch.from_numpy(sel - b * BLK).to(dev)
            for r, v in zip(sel, xs[t].cpu().numpy()):
                rows[int(r)] = v.astype(np.float64)
    index, codes2, scales2, _ = ivf.build_two_stage_blocked(plan, plan2, block, N, BLK, cen,
                                                            on_block=keep_rows)
    q = synth.queries_like("aniso", Q, D, data_seed=100, query_seed=200)
    qt = torch.from_numpy(q).to(dev)
    qrot = R.rslm_fwht(plan, qt)
    pid, pdot = R.ivf_assign_probe(qt, cen, NPROBE, R.IVF_PROBE_IP)
    s1, i1 = R.rslm_scan_topk(plan, index, qrot, pid, pdot, K)
    s2, i2 = R.rslm_rescore_rslm(plan2, codes2, scales2, qrot, s1, i1, K_OUT)
    torch.cuda.synchronize()
    out = dict(R=R, plan=plan, plan2=plan2, block=block, cen=cen.cpu().numpy().astype(np.float64),
               cen_t=cen, crot=R.rslm_fwht(plan, cen),
               q=q, index=index, codes2=codes2, scales2=scales2, sample=sample,
               rows=np.stack([rows[int(r)] for r in sample]),
               pos=F.record_positions(torch, index, N), qrot=qrot.cpu().numpy(),
               pid=pid.cpu().numpy(), s1=s1.cpu().numpy(), i1=i1.cpu().numpy(),
               s2=s2.cpu().numpy(), i2=i2.cpu().numpy(), Rm=H.rot(D, 2),
               C1=synth.codebook(4), C2=synth.codebook(2))
    yield out
    del out
    torch.cuda.empty_cache()


def _rows(f, ids):
    """Rows of vector ids, from their regenerated blocks."""
    ids = np.asarray(ids, dtype=np.int64)
    out = np.empty((len(ids), D))
    for b in np.unique(ids // BLK):
        m = ids // BLK == b
        xs = f["block"](int(b))
        t = torch.from_numpy(ids[m] - b * BLK).to(xs.device)
        out[m] = xs[t].cpu().numpy()
    return out


def _assign_of(f, ids):
    """The list each vector id was filed under (from the record positions)."""
    t = torch.from_numpy(np.asarray(ids, dtype=np.int64)).to(f["pos"].device)
    p = f["pos"][t].cpu().numpy()
    offs = f["index"].list_offsets.cpu().numpy()
    return np.searchsorted(offs, p, side="right") - 1


def test_capacity_two_stage_encode_sampled(cap):
    f = cap
    ids, xs = f["sample"], f["rows"]
    a, keep = F.check_assign(_assign_of(f, ids), xs, f["cen"])
    enc1 = oracle.encode(xs[keep], f["Rm"], f["C1"], 4, centroids=f["cen"][a[keep]],
                         scale_mode="global")
    codes, sc = F.gpu_records(torch, f["R"], f["plan"], f["index"], f["pos"], ids[keep], 4, D)
    ok1 = F.check_codes(codes, sc, enc1, f["C1"])
    assert ok1.mean() > 0.98
    # second stage on the rows whose first stage agrees exactly
    enc2 = oracle.encode_rescore(xs[keep], f["Rm"], enc1, f["C1"], f["C2"], 2,
                                 centroids=f["cen"][a[keep]], scale_mode="global")
    t = torch.from_numpy(ids[keep]).to(f["codes2"].device)
    g2 = oracle.unpack_canonical(f["codes2"][t].cpu().numpy(), 2, D // 2)
    sc2 = f["scales2"][t].cpu().numpy().astype(np.uint32)
    # The second stage codes r2 = R x - R a, a difference of nearly equal
    # vectors: measure the float32 error of the library's r2 on these rows
    # (the same expression, through rslm_encode's resid_rot), check it
    # against its bound, and take the near-tie windows from it: a coordinate
    # of u2 = r2 E_max / max|r2| moves by at most 2 err E_max / max|r2|, a
    # 2-D distance difference by 2 sqrt(2) times that; the scale
    # ||r2|| / ||c2^|| by the measured relative change of ||r2||.
    xk = xs[keep]
    err, r2, same, got = F.r2_error(f["R"], torch, f["plan"], xk, a[keep], f["cen_t"], f["crot"],
                                    f["Rm"], enc1, f["C1"], f["cen"])
    use = same & ok1
    assert use.mean() > 0.97
    bound = F.r2_bound(xk, f["cen"][a[keep]])
    assert np.all(err[use] <= bound[use]), (err / bound).max()
    m2 = np.abs(r2).max(1)
    n2 = np.linalg.norm(r2, axis=1)
    eps_code = 4.0 * err * oracle.e_max(D) / m2
    eps_scale = 2.0 * np.abs(np.linalg.norm(got, axis=1) - n2) / n2 + 2.0 ** -22
    sub = {k: (v[use] if isinstance(v, np.ndarray) and len(v) == len(use) else v)
           for k, v in enc2.items()}
    assert F.check_codes(g2[use], sc2[use], sub, f["C2"], eps_code=eps_code[use],
                         eps_scale=eps_scale[use]).mean() > 0.98


@pytest.mark.parametrize("i", [0, 777])
def test_capacity_scan_and_rescore_sampled(cap, i):
    f = cap
    gi, gs = f["i1"][i], f["s1"][i]
    F.check_topk_order(gs, gi, K)
    qn = np.linalg.norm(f["q"][i])

    def oracle_scores(ids_):
        xr = _rows(f, ids_)
        ao, _ = oracle.assign_l2_expanded(xr, f["cen"])
        e = oracle.encode(xr, f["Rm"], f["C1"], 4, centroids=f["cen"][ao], scale_mode="global")
        xt = oracle.reconstruct(e["codes"], e["s_code"], e["g_code"], f["C1"], f["Rm"],
                                f["cen"][ao])
        return ao, e, xt @ f["q"][i].astype(np.float64), np.linalg.norm(xt, axis=1), xr

    ao, e1, exact, xn, xr = oracle_scores(gi)
    assert np.mean([L in set(f["pid"][i].tolist()) for L in ao]) >= 0.99
    # pairing of every returned id and completeness over the members of the
    # 16 best probed lists, each row encoded against its list's centre
    members, lst = F.members_of(torch, f["index"], f["pid"][i][:16])
    gl = _assign_of(f, gi)
    extra = ~np.isin(gi, members)
    members = np.concatenate([members, gi[extra]])
    lst = np.concatenate([lst, gl[extra]])
    xm = _rows(f, members)
    best = lst == f["pid"][i][0]
    am, _ = oracle.assign_l2_expanded(xm[best], f["cen"])
    assert (am == f["pid"][i][0]).mean() >= 0.99
    sm, xnm, near, _ = F.oracle_member_scores(xm, lst, f["cen"], f["q"][i], f["Rm"], f["C1"], 4)
    F.check_probed(gs, gi, members, sm, H.score_tol(sm, qn, xnm), near)
    # rescoring: the oracle's RSLM rescoring of the same shortlist (second
    # stage encoded by the oracle from the shortlist's rows, first-stage
    # scores its own); every rescored id must be one of the oracle's top-10
    # within the tolerance, at its score (a vector whose first-stage code sits
    # on a decision threshold gets another second stage: at most one)
    ri, rs = f["i2"][i], f["s2"][i]
    assert set(ri.tolist()) <= set(gi.tolist())
    F.check_topk_order(rs, ri, K_OUT)
    e2 = oracle.encode_rescore(xr, f["Rm"], e1, f["C1"], f["C2"], 2, centroids=f["cen"][ao],
                               scale_mode="global")
    qr = f["q"][i].astype(np.float64) @ f["Rm"].T
    ref_s, ref_i = oracle.rescore_rslm(qr[None], exact[None], np.arange(K)[None, :], e2["codes"],
                                       e2["s_code"], e2["g_code"], f["C2"], K)
    ref = np.empty(K)
    ref[ref_i[0]] = ref_s[0]                      # oracle rescored score per shortlist slot
    slot = np.array([np.nonzero(gi == v)[0][0] for v in ri])
    tol = 1.1 * (H.score_tol(ref[slot], qn, xn.max()) + np.abs(gs - exact).max())
    kth = ref_s[0][K_OUT - 1]
    assert np.sum(np.abs(rs - ref[slot]) > tol) <= 1
    assert np.sum(ref[slot] < kth - 2 * tol) <= 1
