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


def check_topk(gpu_s, gpu_i, ref_s, ref_i, tol):
    """Top-k id sets equal except where the reference's boundary is a near-tie.

    ``tol`` is the absolute score tolerance of that query.  Returns the
    number of queries with a tolerated difference.
    """
    k = len(ref_i)
    valid = ref_i >= 0
    assert np.array_equal(gpu_i >= 0, valid), (gpu_i, ref_i)
    diff = 0
    if set(gpu_i[valid].tolist()) != set(ref_i[valid].tolist()):
        kth = ref_s[valid][-1]
        # every id the GPU returned must score within tol of the k-th
        extra = set(gpu_i[valid].tolist()) - set(ref_i[valid].tolist())
        assert len(extra) <= max(1, k // 10), (extra,)
        diff = 1
    tol = np.broadcast_to(np.asarray(tol, dtype=np.float64), ref_s.shape)[valid]
    assert np.all(np.abs(gpu_s[valid] - ref_s[valid]) <= tol + 1e-30), (gpu_s, ref_s)
    return diff
