"""Oracle: IVF routing, second-stage scan, top-k and rescoring (float64).

Follows the paper's ANN pipeline:
  * Section "End-to-End Comparison with Faiss and ScaNN", Setup: partition the
    collection with Euclidean k-means, quantise each vector's residual against
    its assigned partition centre, route a query to the n_probe partitions with
    the largest dot product with their centres, scan the quantised residuals of
    those partitions and keep the top-k.
  * Section "Relative Quantization": a candidate's score is
    <q, a + r~> = <q, a> + <q, r~> (local) or s (<q, a> + <q, r~>) (global),
    reusing <q, a>; with a = the partition centre in the first stage.
  * Section "Performance Impact and Memory Savings": the query is rotated once
    and dot products are taken in the rotated space; a candidate's residual
    term is a sum of per-sub-vector lookups <q_rot[j g:(j+1) g], C_k>.
  * Section "Background and Related Work": two-stage retrieval -- a low-bit
    scan produces a shortlist which a higher-fidelity representation rescores.
    The 8-bit rescoring codec is SQ8 (a per-dimension min/max range with 256
    levels) applied to the second residual r2 = x - x~1, relative with local
    scaling ("RelApprox-SQ8", tables tab:recall_eval_relative).

Readings where the paper is not explicit:
  * ties: (score desc, id asc) for top-k; (dot desc, list id asc) for
    probing; the lowest centre id for assignment;
  * k-means: init with nlist distinct random sample points, fixed iteration
    count, an empty cluster keeps its centre;
  * SQ8: lo_d / hi_d are the min / max of coordinate d over the collection,
    step = (hi - lo) / 255 (0 gives code 0), code = clamp(round-half-even(
    (v - lo) / step), 0, 255); it is applied in the rotated space (the rotation
    is a fixed table of the codec), scored against the rotated query;
  * top-k lists shorter than k are padded with (-inf, -1).
"""

import numpy as np

from .codec import dec_ue4m12, dec_ue7m9


def assign_l2(x, centroids, chunk=2048):
    """argmin_p ||x - c_p||^2 per row (lowest p on ties); also the minimum."""
    x = np.asarray(x, dtype=np.float64)
    c = np.asarray(centroids, dtype=np.float64)
    ids = np.empty(len(x), dtype=np.int64)
    best = np.empty(len(x))
    for lo in range(0, len(x), chunk):
        d = ((x[lo:lo + chunk, None, :] - c[None, :, :]) ** 2).sum(-1)
        ids[lo:lo + chunk] = d.argmin(1)
        best[lo:lo + chunk] = d.min(1)
    return ids, best


def assign_l2_expanded(x, centroids, chunk=4096):
    """The same argmin as ``assign_l2`` through the identity
    ||x - c||^2 = ||x||^2 - 2 <x, c> + ||c||^2 (float64, library matmul), for
    large centre sets where the direct difference tensor does not fit.
    Rounding can move a distance by a few ulps of ||x||^2, so a row whose two
    best centres are that close may pick the other one."""
    x = np.asarray(x, dtype=np.float64)
    c = np.asarray(centroids, dtype=np.float64)
    cn = (c * c).sum(1)
    ids = np.empty(len(x), dtype=np.int64)
    best = np.empty(len(x))
    for lo in range(0, len(x), chunk):
        xb = x[lo:lo + chunk]
        d = (xb * xb).sum(1)[:, None] - 2.0 * (xb @ c.T) + cn[None, :]
        ids[lo:lo + chunk] = d.argmin(1)
        best[lo:lo + chunk] = d.min(1)
    return ids, best


def probe_ip(q, centroids, nprobe):
    """The nprobe centres with the largest <q, c> per query (ties: lower id)."""
    q = np.asarray(q, dtype=np.float64)
    c = np.asarray(centroids, dtype=np.float64)
    dots = q @ c.T
    nl = c.shape[0]
    ids = np.empty((len(q), nprobe), dtype=np.int64)
    vals = np.empty((len(q), nprobe))
    for i in range(len(q)):
        order = np.lexsort((np.arange(nl), -dots[i]))[:nprobe]
        ids[i] = order
        vals[i] = dots[i, order]
    return ids, vals, dots


def kmeans(x, nlist, iters=10, seed=0, init=None):
    """Euclidean k-means (Lloyd): random distinct-point init (or the given
    initial centres), fixed iterations; each iteration assigns every point to
    its nearest centre (lowest id on ties) and moves each centre to the mean
    of its points, an empty cluster keeping its centre."""
    x = np.asarray(x, dtype=np.float64)
    if init is None:
        rng = np.random.default_rng(seed)
        c = x[rng.choice(len(x), nlist, replace=False)].copy()
    else:
        c = np.array(init, dtype=np.float64)
        assert c.shape == (nlist, x.shape[1])
    for _ in range(iters):
        a, _ = assign_l2(x, c)
        for p in range(nlist):
            sel = a == p
            if sel.any():
                c[p] = x[sel].mean(0)
    return c


def scan_scores_lut(q_rot, qc_dot, codes, s_hat, g_hat, C, C_lead=None, lead=0):
    """LUT route: g^ (<q, c> + s^ sum_j LUT[j, code_j]) for one query.

    q_rot: rotated query (length D, zero-padded here to n_sub * g);
    codes: (n, n_sub); s_hat / g_hat: decoded scales (n,); qc_dot: <q, c_p>.
    The first ``lead`` sub-vectors look up C_lead (Rslm4Lite).
    """
    C = np.asarray(C, dtype=np.float64)
    K, g = C.shape
    n, n_sub = codes.shape
    qp = np.zeros(n_sub * g)
    qp[:len(q_rot)] = q_rot
    lut = qp.reshape(n_sub, g) @ C.T                  # LUT[j, k]
    if lead:
        Cl = np.asarray(C_lead, dtype=np.float64)
        lut[:lead] = 0.0
        lut[:lead, :Cl.shape[0]] = qp[:lead, None] * Cl[None, :, 0]
    resid = lut[np.arange(n_sub)[None, :], codes].sum(1)
    return g_hat * (qc_dot + s_hat * resid)


def scan_scores_dense(q, xtilde):
    """Dense route: <q, x~> with x~ reconstructed in the original space."""
    return np.asarray(xtilde, dtype=np.float64) @ np.asarray(q, dtype=np.float64)


def topk(scores, ids, k):
    """Top-k by (score desc, id asc), padded with (-inf, -1)."""
    scores = np.asarray(scores, dtype=np.float64)
    ids = np.asarray(ids, dtype=np.int64)
    order = np.lexsort((ids, -scores))[:k]
    out_s = np.full(k, -np.inf)
    out_i = np.full(k, -1, dtype=np.int64)
    out_s[:len(order)] = scores[order]
    out_i[:len(order)] = ids[order]
    return out_s, out_i


def ivf_candidates(q, q_rot, centroids, lists, C, nprobe, C_lead=None, lead=0):
    """Route and scan (LUT route): every candidate of every probed list.

    ``lists[p]`` = dict(ids, codes (n_p, n_sub), s_hat (n_p,), g_hat (n_p,)).
    Rslm4Lite: the first ``lead`` codes look up C_lead.
    Returns (probe ids (Q, nprobe), per query a pair (scores, ids) over the
    members of its probed lists, in probe order).
    """
    pid, pdot, _ = probe_ip(q, centroids, nprobe)
    out = []
    for i in range(len(q)):
        all_s, all_i = [np.zeros(0)], [np.zeros(0, dtype=np.int64)]
        for j in range(nprobe):
            L = lists[int(pid[i, j])]
            if len(L["ids"]) == 0:
                continue
            all_s.append(scan_scores_lut(q_rot[i], pdot[i, j], L["codes"],
                                         L["s_hat"], L["g_hat"], C, C_lead, lead))
            all_i.append(np.asarray(L["ids"], dtype=np.int64))
        out.append((np.concatenate(all_s), np.concatenate(all_i)))
    return pid, out


def ivf_search(q, q_rot, centroids, lists, C, nprobe, k, C_lead=None, lead=0):
    """Route, scan (LUT route) and select for a batch of queries.

    Returns (scores (Q, k), ids (Q, k), probe ids (Q, nprobe)).
    """
    pid, cands = ivf_candidates(q, q_rot, centroids, lists, C, nprobe, C_lead, lead)
    Q = len(q)
    out_s = np.full((Q, k), -np.inf)
    out_i = np.full((Q, k), -1, dtype=np.int64)
    for i, (s, ids) in enumerate(cands):
        out_s[i], out_i[i] = topk(s, ids, k)
    return out_s, out_i, pid


def sq8_fit(v):
    v = np.asarray(v, dtype=np.float64)
    return v.min(0), v.max(0)


def sq8_encode(v, lo, hi):
    v = np.asarray(v, dtype=np.float64)
    step = (hi - lo) / 255.0
    safe = np.where(step > 0, step, 1.0)
    code = np.rint((v - lo) / safe)
    code = np.where(step > 0, code, 0.0)
    return np.clip(code, 0, 255).astype(np.uint8)


def sq8_decode(codes, lo, hi):
    step = (hi - lo) / 255.0
    return lo + codes.astype(np.float64) * step


def rescore_sq8_scores(q_rot, cand_scores, cand_ids, codes2, lo, hi):
    """score2 = score1 + <q_rot, r~2> of every shortlisted candidate.

    q_rot: (Q, D); cand_*: (Q, k_in), ids < 0 are empty slots; codes2 (N, D)
    uint8 indexed by id.  Returns per query a pair (score2, ids).
    """
    out = []
    for i in range(cand_ids.shape[0]):
        ok = cand_ids[i] >= 0
        ids = np.asarray(cand_ids[i][ok], dtype=np.int64)
        r2 = sq8_decode(codes2[ids], lo, hi)
        s2 = np.asarray(cand_scores[i][ok], dtype=np.float64) + r2 @ q_rot[i]
        out.append((s2, ids))
    return out


def rescore_sq8(q_rot, cand_scores, cand_ids, codes2, lo, hi, k_out):
    """score2 = score1 + <q_rot, r~2> over the shortlist, then top-k_out."""
    Q, _ = cand_ids.shape
    out_s = np.full((Q, k_out), -np.inf)
    out_i = np.full((Q, k_out), -1, dtype=np.int64)
    for i, (s2, ids) in enumerate(rescore_sq8_scores(q_rot, cand_scores, cand_ids, codes2,
                                                     lo, hi)):
        out_s[i], out_i[i] = topk(s2, ids, k_out)
    return out_s, out_i


def rescore_rslm(q_rot, cand_scores, cand_ids, codes2, s2_code, g2_code, C2, k_out):
    """RSLM rescoring codec (global relative scaling, Section "Relative
    Quantization"): score2 = g2^ (score1 + s2^ sum_j LUT[j, code2_j]) with
    LUT[j, k] = <q_rot[j g:(j+1) g], C2_k> and score1 = <q, a> the
    shortlist's first-stage score; then the top-k_out.

    codes2 (N, n_sub), s2_code / g2_code (N,) are indexed by vector id;
    cand_* are (Q, k_in) with ids < 0 for empty slots.
    """
    Q, _ = cand_ids.shape
    out_s = np.full((Q, k_out), -np.inf)
    out_i = np.full((Q, k_out), -1, dtype=np.int64)
    for i, (s2, ids) in enumerate(rescore_rslm_scores(q_rot, cand_scores, cand_ids, codes2,
                                                      s2_code, g2_code, C2)):
        out_s[i], out_i[i] = topk(s2, ids, k_out)
    return out_s, out_i


def rescore_rslm_scores(q_rot, cand_scores, cand_ids, codes2, s2_code, g2_code, C2):
    """score2 of every shortlisted candidate under the RSLM rescoring codec
    (see ``rescore_rslm``); per query a pair (score2, ids)."""
    sh = np.array([dec_ue7m9(u) for u in s2_code])
    gh = np.array([dec_ue4m12(u) for u in g2_code])
    out = []
    for i in range(cand_ids.shape[0]):
        ok = cand_ids[i] >= 0
        ids = np.asarray(cand_ids[i][ok], dtype=np.int64)
        s1 = np.asarray(cand_scores[i][ok], dtype=np.float64)
        s2 = scan_scores_lut(q_rot[i], s1, codes2[ids], sh[ids], gh[ids], C2) if len(ids) \
            else np.zeros(0)
        out.append((s2, ids))
    return out


def brute_force_mips(q, x, k):
    """Exact maximum inner product search over raw vectors (float64)."""
    q = np.asarray(q, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    s = q @ x.T
    out_s = np.empty((len(q), k))
    out_i = np.empty((len(q), k), dtype=np.int64)
    ids = np.arange(x.shape[0])
    for i in range(len(q)):
        out_s[i], out_i[i] = topk(s[i], ids, k)
    return out_s, out_i
