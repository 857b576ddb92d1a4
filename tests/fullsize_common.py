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


def check_codes(codes, sc, enc, C, global_scale=True, amp=None):
    """Codes bit-exact except near-ties (at most max(2, 1e-4) of them); s^
    codes exact except near a rounding midpoint or on rows with a flipped
    code, never more than 1 ulp off; g^ codes likewise on rows whose codes and
    s^ agree.  Returns the rows whose codes and scale codes all agree.

    The near-tie windows are 1e-5 (relative to the normalised coordinate or
    to the scale) times ``amp`` per row, default 1: a second-stage input
    x - a is a difference of nearly equal vectors, so the float32 path's
    error relative to it grows by ||x|| / ||x - a||."""
    n = len(codes)
    amp = np.ones(n) if amp is None else np.maximum(1.0, np.asarray(amp, dtype=np.float64))
    eps = 1e-5 * amp
    near = np.concatenate([H.near_threshold(enc["u"][i:i + 1], C, eps=eps[i]) for i in range(n)])
    flips = codes != enc["codes"]
    assert not np.any(flips & ~near), np.argwhere(flips & ~near)[:5]
    assert flips.sum() <= max(2, 1e-4 * flips.size)
    su, gu = sc & 0xFFFF, sc >> 16
    rows_flip = flips.any(1)

    def near_round(v, dec, enc_fn):
        return np.array([H.near_rounding(v[i:i + 1], dec, enc_fn, rel=eps[i])[0]
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


def check_scores(gs, exact, qn, xn, max_viol=2):
    """Returned scores against the oracle's scores of the same vectors."""
    tol = H.score_tol(exact, qn, xn)
    viol = np.abs(gs - exact) > tol
    assert viol.sum() <= max_viol, (gs[viol], exact[viol])


def check_complete(members, ok, sm, tolm, kth, returned, max_missed=1):
    """Every member the oracle scores above the k-th returned score (beyond
    tolerance) must have been returned."""
    missed = [v for v, s, t, o in zip(members, sm, tolm, ok)
              if o and s > kth + t and int(v) not in returned]
    assert len(missed) <= max_missed, missed
