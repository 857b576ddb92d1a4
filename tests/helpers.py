"""Test-side helpers: cached oracle rotations, tolerance rules, and host-side
index assembly from oracle outputs.  Imported by tests only."""

import functools

import numpy as np

import oracle
import synth

S1 = synth.sign_table()
P = synth.permutation_table()


@functools.lru_cache(maxsize=64)
def rot(D, passes):
    return oracle.rotation_matrix(D, passes, S1, P)


def near_threshold(u, C, eps=1e-5):
    """Mask (n, n_sub) of sub-vectors whose assignment is within eps of a tie.

    g = 1: |u_j - t_k| < eps for a decision threshold t_k (midpoints);
    g > 1: ||u_j - C_2nd|| - ||u_j - C_1st|| < eps (codebook units).
    """
    C = np.asarray(C, dtype=np.float64)
    K, g = C.shape
    n = u.shape[0]
    sub = u.reshape(n, -1, g)
    if g == 1:
        t = 0.5 * (C[1:, 0] + C[:-1, 0])
        return (np.abs(sub[:, :, 0, None] - t[None, None, :]) < eps).any(-1)
    d = np.sqrt(((sub[:, :, None, :] - C[None, None]) ** 2).sum(-1))
    d.sort(-1)
    return (d[:, :, 1] - d[:, :, 0]) < eps


def near_threshold_rows(u, C, eps=1e-5, chunk=2048):
    """Per row: does any sub-vector lie within eps of a tie (``near_threshold``
    evaluated in chunks of rows, for large row counts)."""
    out = np.zeros(len(u), dtype=bool)
    for lo in range(0, len(u), chunk):
        out[lo:lo + chunk] = near_threshold(u[lo:lo + chunk], C, eps).any(1)
    return out


def near_rounding(s, dec, enc, rel=1e-5):
    """True where s lies within rel of the midpoint between two scale codes."""
    out = np.zeros(len(s), dtype=bool)
    for i, v in enumerate(s):
        if v <= 0:
            continue
        u = enc(v)
        lo, hi = dec(max(u - 1, 0)), dec(u + 1)
        c = dec(u)
        m1, m2 = 0.5 * (lo + c), 0.5 * (c + hi)
        out[i] = abs(v - m1) < rel * v or abs(v - m2) < rel * v
    return out


def score_tol(s_ref, qn, xn, rel=1e-4):
    """Tolerance of the scores: rel * max(|s|, 1e-3 ||q|| ||x~||)."""
    return rel * np.maximum(np.abs(s_ref), 1e-3 * qn * xn)


def dec_scales(scales_u32):
    s = np.asarray(scales_u32).astype(np.uint32)
    sh = np.array([oracle.dec_ue7m9(int(v) & 0xFFFF) for v in s])
    gh = np.array([oracle.dec_ue4m12(int(v) >> 16) for v in s])
    return sh, gh


def check_topk(gpu_s, gpu_i, ref_s, ref_i, tol_fn, cand_s, cand_i):
    """A returned top-k against the oracle's, for one query.

    ``cand_s`` / ``cand_i``: the oracle's scores of every candidate the query
    sees (all members of its probed lists, or its whole shortlist);
    ``tol_fn(scores)`` gives the absolute score tolerance at those scores.
    Asserts:
      * the valid slots (id >= 0) are the same as the oracle's, ids distinct;
      * the returned order is (score desc, id asc);
      * pairing: every returned score is within tolerance of the oracle's
        score of the id returned beside it;
      * position-wise, the returned scores match the oracle's k best;
      * the id sets are equal except at the boundary: an id only one side
        returned must score within tolerance of the oracle's k-th score.
    Returns 1 if the id sets differ (a tolerated near-tie), else 0.
    """
    k = len(ref_i)
    valid = ref_i >= 0
    assert np.array_equal(gpu_i >= 0, valid), (gpu_i, ref_i)
    gi = gpu_i[valid].astype(np.int64)
    gs = gpu_s[valid].astype(np.float64)
    assert len(set(gi.tolist())) == len(gi), "duplicate ids"
    assert all(gs[j] > gs[j + 1] or (gs[j] == gs[j + 1] and gi[j] < gi[j + 1])
               for j in range(len(gi) - 1)), (gs, gi)
    lookup = dict(zip(np.asarray(cand_i, dtype=np.int64).tolist(),
                      np.asarray(cand_s, dtype=np.float64).tolist()))
    assert all(int(v) in lookup for v in gi), "an id outside the query's candidates"
    own = np.array([lookup[int(v)] for v in gi])
    assert np.all(np.abs(gs - own) <= tol_fn(own) + 1e-30), (gs, own, gi)
    rs = ref_s[valid]
    assert np.all(np.abs(gs - rs) <= tol_fn(rs) + 1e-30), (gs, rs)
    diff = 0
    if len(rs) and set(gi.tolist()) != set(ref_i[valid].tolist()):
        kth = rs[-1]
        t = float(tol_fn(np.array([kth]))[0])
        odd = set(gi.tolist()) ^ set(ref_i[valid].tolist())
        for v in odd:
            assert abs(lookup[int(v)] - kth) <= 2 * t + 1e-30, (v, lookup[int(v)], kth, t)
        diff = 1
    return diff
