"""Checks shared by the full-size parity tests: sampled outputs of an index
built and searched through the library's entry points, compared with what the
oracle computes for the same rows one by one.  Imported by tests only."""

import numpy as np

import oracle
from tests import helpers as H


def record_positions(torch, index, n):
    """Record position of every vector id of an index (-1: not indexed)."""
    ids_rec = index.ids.long()
    valid = ids_rec >= 0
    pos = torch.full((n,), -1, dtype=torch.int64, device=ids_rec.device)
    pos[ids_rec[valid]] = torch.arange(ids_rec.numel(), device=ids_rec.device)[valid]
    return pos


def gpu_records(torch, R, plan, index, pos, ids, bits, n_sub):
    """Codes (n, n_sub) and scale words of the records holding vector ids."""
    t = torch.from_numpy(np.asarray(ids, dtype=np.int64)).to(pos.device)
    p = pos[t]
    assert bool((p >= 0).all())
    # only the tiles (16 records each) that hold them are unpacked
    tb = plan.code_bytes(16)
    tiles = (p // 16).cpu().numpy()
    uniq, inv = np.unique(tiles, return_inverse=True)
    sel = index.codes.view(-1, tb)[torch.from_numpy(uniq).to(pos.device)].contiguous()
    canon = R.rslm_unpack_codes(plan, sel.view(-1), len(uniq) * 16)
    rows = torch.from_numpy(inv * 16).to(pos.device) + (p % 16)
    canon = canon[rows].cpu().numpy()
    sc = index.scales[p].cpu().numpy().astype(np.uint32)
    return oracle.unpack_canonical(canon, bits, n_sub), sc


def check_assign(ga, xs, cen, max_differ=2):
    """GPU assignment against the oracle's; returns the oracle's ids and the
    rows where both agree (only near-equidistant centres may disagree)."""
    a, best = oracle.assign_l2_expanded(xs, cen)
    differ = np.nonzero(ga != a)[0]
    assert len(differ) <= max_differ, len(differ)
    for r in differ:
        dg = ((xs[r] - cen[ga[r]]) ** 2).sum()
        assert dg - best[r] <= 1e-4 * (1.0 + best[r])
    return a, ga == a


def check_codes(codes, sc, enc, C, global_scale=True, eps_code=None, eps_scale=None):
    """Codes bit-exact except near-ties (at most max(2, 1e-4) of them); s^
    codes exact except near a rounding midpoint or on rows with a flipped
    code, never more than 1 ulp off; g^ codes likewise on rows whose codes and
    s^ agree.  Returns the rows whose codes and scale codes all agree.

    The near-tie windows are 1e-5 in the normalised coordinate (codes) and
    relative to the scale (scale codes), unless per-row windows ``eps_code`` /
    ``eps_scale`` are given (never below 1e-5): the second stage's input is
    a difference of nearly equal vectors, and its windows come from the
    float32 error of that difference as measured by the caller."""
    n = len(codes)
    eps = np.full(n, 1e-5) if eps_code is None else np.maximum(1e-5, eps_code)
    epss = np.full(n, 1e-5) if eps_scale is None else np.maximum(1e-5, eps_scale)
    near = np.concatenate([H.near_threshold(enc["u"][i:i + 1], C, eps=eps[i]) for i in range(n)])
    flips = codes != enc["codes"]
    assert not np.any(flips & ~near), np.argwhere(flips & ~near)[:5]
    assert flips.sum() <= max(2, 1e-4 * flips.size)
    su, gu = sc & 0xFFFF, sc >> 16
    rows_flip = flips.any(1)

    def near_round(v, dec, enc_fn):
        return np.array([H.near_rounding(v[i:i + 1], dec, enc_fn, rel=epss[i])[0]
                         for i in range(n)], dtype=bool)
    s_near = near_round(enc["s"], oracle.dec_ue7m9, oracle.enc_ue7m9)
    assert np.all((su == enc["s_code"]) | s_near | rows_flip)
    assert np.all(np.abs(su.astype(np.int64) - enc["s_code"].astype(np.int64)) <= 1)
    ok = ~rows_flip & (su == enc["s_code"])
    if global_scale:
        g_near = near_round(enc["g"], oracle.dec_ue4m12, oracle.enc_ue4m12)
        # (a row whose codes or s^ differ has another denominator for g^)
        assert np.all((gu == enc["g_code"]) | g_near | ~ok)
        assert np.all(np.abs(gu[ok].astype(np.int64) - enc["g_code"][ok].astype(np.int64)) <= 1)
        ok &= gu == enc["g_code"]
    return ok


def check_topk_order(gs, gi, k):
    """k distinct valid ids, sorted by (score desc, id asc)."""
    assert np.all(gi >= 0) and len(set(gi.tolist())) == k
    assert all(gs[j] > gs[j + 1] or (gs[j] == gs[j + 1] and gi[j] < gi[j + 1])
               for j in range(k - 1))


def members_of(torch, index, lists):
    """Vector ids and list ids of every member of the given lists (host)."""
    offs = index.list_offsets.cpu().numpy()
    sizes = index.list_sizes.cpu().numpy()
    lists = np.asarray(lists, dtype=np.int64)
    rec = np.concatenate([np.arange(offs[L], offs[L] + sizes[L]) for L in lists])
    lst = np.concatenate([np.full(sizes[L], L, dtype=np.int64) for L in lists])
    ids = index.ids[torch.from_numpy(rec).to(index.ids.device)].cpu().numpy().astype(np.int64)
    return ids, lst


def oracle_member_scores(xs, lst, cen, q, Rm, C, bits, scale_mode="global"):
    """The oracle's encoding of rows ``xs`` against the centres of the lists
    they are filed under, and their scan scores for query ``q`` (dense route
    over the reconstruction).  Also marks the rows whose encoding sits in a
    near-tie window (a code within 1e-5 of a decision threshold, a scale
    within 1e-5 of a rounding midpoint): the library may encode those
    differently.  Returns (scores, ||x~||, near, enc)."""
    enc = oracle.encode(xs, Rm, C, bits, centroids=cen[lst], scale_mode=scale_mode)
    xt = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], C, Rm, cen[lst])
    near = H.near_threshold_rows(enc["u"], C)
    near |= H.near_rounding(enc["s"], oracle.dec_ue7m9, oracle.enc_ue7m9)
    if scale_mode == "global":
        near |= H.near_rounding(enc["g"], oracle.dec_ue4m12, oracle.enc_ue4m12)
    return xt @ np.asarray(q, dtype=np.float64), np.linalg.norm(xt, axis=1), near, enc


def check_probed(gs, gi, members, sm, tolm, near, max_near=3):
    """Pairing and completeness of a returned top-k over every member of the
    query's probed lists, against the oracle's scores of those members:
      * every returned id is a member, and its returned score is within
        tolerance of the oracle's score of that id;
      * every member the oracle scores above the returned k-th score (beyond
        tolerance) was returned.
    Only rows in an encoding near-tie window (``near``) may break either
    rule, at most ``max_near`` of them."""
    pos = {int(v): j for j, v in enumerate(members)}
    assert all(int(v) in pos for v in gi), "a returned id outside the probed lists"
    j = np.array([pos[int(v)] for v in gi])
    bad = np.abs(gs - sm[j]) > tolm[j]
    assert not np.any(bad & ~near[j]), (gi[bad], gs[bad], sm[j][bad])
    kth = gs[-1]
    above = np.nonzero(sm > kth + tolm)[0]
    missed = above[~np.isin(members[above], gi)]
    assert not np.any(~near[missed]), (members[missed], sm[missed], kth)
    assert bad.sum() + len(missed) <= max_near, (bad.sum(), len(missed))


def r2_error(R, torch, plan, xs, lst, cen_t, crot, Rm, enc1, C1, cen):
    """Measured float32 error of the library's rotated second residual
    R x - g^ (R c + s^ C[code]) on rows xs (filed under lists lst), against
    the oracle's float64 value: the library's resid_rot output of
    rslm_encode, which evaluates the same expression as the two-stage
    encoder.  Returns (per-row max |error|, oracle r2, rows whose first
    stage agrees, the library's r2)."""
    dev = cen_t.device
    n, D = xs.shape
    xt = torch.from_numpy(np.ascontiguousarray(xs, dtype=np.float32)).to(dev)
    codes = torch.zeros(plan.code_bytes(n), dtype=torch.uint8, device=dev)
    scales = torch.zeros(n, dtype=torch.int32, device=dev)
    resid = torch.zeros((n, D), dtype=torch.float32, device=dev)
    R.rslm_encode(plan, xt, codes, scales, rec_list=torch.from_numpy(lst.astype(np.int32)).to(dev),
                  centroids=cen_t, centroids_rot=crot, resid_rot=resid)
    g1 = oracle.unpack_canonical(R.rslm_unpack_codes(plan, codes, n).cpu().numpy(), plan.bits,
                                 enc1["codes"].shape[1])
    sc = scales.cpu().numpy().astype(np.uint32)
    same = ((g1 == enc1["codes"]).all(1) & ((sc & 0xFFFF) == enc1["s_code"]) &
            ((sc >> 16) == enc1["g_code"]))
    ra = oracle.first_stage_rotated(enc1["codes"], enc1["s_code"], enc1["g_code"], C1, Rm,
                                    cen[lst])
    r2 = np.asarray(xs, dtype=np.float64) @ Rm.T - ra
    got = resid.cpu().numpy().astype(np.float64)
    err = np.abs(got - r2).max(1)
    return err, r2, same, got


def r2_bound(xs, cen_rows):
    """Float32 error bound of the rotated second residual: R (x - c) through
    at most 14 butterfly stages of an orthonormal transform, each adding at
    most one rounding per element at the scale of the operand's norm, then
    four more operations at the scale of ||x|| + ||c||: 2^-19 (||x|| + ||c||)
    (32 units of float32 roundoff)."""
    return 2.0 ** -19 * (np.linalg.norm(xs, axis=1) + np.linalg.norm(cen_rows, axis=1))
