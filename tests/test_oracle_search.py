"""Pins for the oracle's routing, scan, top-k and rescoring.

Sources of truth: the scoring identity of Section "Relative Quantization"
checked through an independent dense reconstruction route, brute force on tiny
inputs (exhaustive probing equals exhaustive scoring), explicit min/max for
SQ8, and hand-made tie cases for the ordering rules.
"""

import os

import numpy as np
import pytest

import oracle
import synth

S1 = synth.sign_table()
P = synth.permutation_table()


def _small_index(D=64, bits=4, n=300, nlist=6, seed=0, mode="global"):
    x = synth.gmix(n, D, 8, seed=seed + 100)
    cent = oracle.kmeans(x, nlist, iters=5, seed=seed)
    assign, _ = oracle.assign_l2(x, cent)
    R = oracle.rotation_matrix(D, oracle.resolve_passes(bits, D, 2), S1, P)
    C = synth.codebook(bits)
    enc = oracle.encode(x, R, C, bits, centroids=cent[assign], scale_mode=mode)
    return x, cent, assign, R, C, enc


def test_lut_route_equals_dense_route():
    for bits in (1, 2, 3, 4):
        x, cent, assign, R, C, enc = _small_index(bits=bits, seed=bits)
        q = synth.queries_like("gmix", 3, x.shape[1], data_seed=100 + bits, n_comp=8)
        xt = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], C, R, cent[assign])
        sh = np.array([oracle.dec_ue7m9(u) for u in enc["s_code"]])
        gh = np.array([oracle.dec_ue4m12(u) for u in enc["g_code"]])
        for qq in q:
            lut = oracle.scan_scores_lut(R @ qq, cent[assign] @ qq, enc["codes"], sh, gh, C)
            dense = oracle.scan_scores_dense(qq, xt)
            assert np.abs(lut - dense).max() < 1e-12 * max(1.0, np.abs(dense).max())


def test_probe_is_sorted_dots():
    rng = np.random.default_rng(0)
    c = rng.standard_normal((50, 16))
    q = rng.standard_normal((5, 16))
    ids, vals, dots = oracle.probe_ip(q, c, 7)
    for i in range(5):
        ref = sorted(range(50), key=lambda p: (-dots[i, p], p))[:7]
        assert ids[i].tolist() == ref
    # ties go to the lower list id: small integers make every dot product
    # exact, so duplicated centres tie bit for bit
    ci = rng.integers(-3, 4, (3, 16)).astype(np.float64)
    c2 = np.vstack([ci, ci, ci])
    ids2, vals2, _ = oracle.probe_ip(ci[:1], c2, 4)
    assert vals2[0, 0] == vals2[0, 1] == vals2[0, 2]
    order = sorted(range(9), key=lambda p: (-float(ci[0] @ c2[p]), p))
    assert ids2[0].tolist() == order[:4]
    assert ids2[0].tolist()[:3] == [0, 3, 6]


def test_assign_lowest_on_tie():
    c = np.array([[1.0, 0.0], [-1.0, 0.0], [1.0, 0.0]])
    ids, d = oracle.assign_l2(np.array([[0.0, 1.0], [2.0, 0.0]]), c)
    assert ids.tolist() == [0, 0]


def test_assign_expanded_matches_direct():
    """The expanded-distance route picks the direct route's centre, and its
    minimum is the squared distance to that centre (brute force)."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((300, 24)) * 3.0 + 1.0
    c = rng.standard_normal((40, 24)) * 3.0
    ids, d = oracle.assign_l2(x, c)
    ide, de = oracle.assign_l2_expanded(x, c, chunk=64)
    assert np.array_equal(ids, ide)
    brute = np.array([((x[i] - c[ide[i]]) ** 2).sum() for i in range(len(x))])
    assert np.allclose(de, brute, rtol=1e-12, atol=1e-9)
    assert np.allclose(d, de, rtol=1e-12, atol=1e-9)
    # exact ties still go to the lower centre id
    c2 = np.array([[1.0, 0.0], [-1.0, 0.0], [1.0, 0.0]])
    ide2, _ = oracle.assign_l2_expanded(np.array([[0.0, 1.0], [2.0, 0.0]]), c2)
    assert ide2.tolist() == [0, 0]


def test_topk_ties_and_padding():
    s, i = oracle.topk([1.0, 3.0, 3.0, 2.0], [9, 7, 4, 1], 3)
    assert i.tolist() == [4, 7, 1]
    s, i = oracle.topk([1.0], [5], 3)
    assert i.tolist() == [5, -1, -1] and np.isneginf(s[1:]).all()


def test_exhaustive_ivf_equals_brute_force_on_decoded():
    x, cent, assign, R, C, enc = _small_index(D=64, bits=4, n=240, nlist=5, seed=9)
    sh = np.array([oracle.dec_ue7m9(u) for u in enc["s_code"]])
    gh = np.array([oracle.dec_ue4m12(u) for u in enc["g_code"]])
    lists = {}
    for p in range(5):
        sel = np.where(assign == p)[0]
        lists[p] = {"ids": sel, "codes": enc["codes"][sel], "s_hat": sh[sel], "g_hat": gh[sel]}
    q = synth.queries_like("gmix", 4, 64, data_seed=109, n_comp=8)
    qr = q @ R.T
    s, i, _ = oracle.ivf_search(q, qr, cent, lists, C, nprobe=5, k=10)
    xt = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], C, R, cent[assign])
    bs, bi = oracle.brute_force_mips(q, xt, 10)
    assert np.array_equal(i, bi)
    assert np.abs(s - bs).max() < 1e-10


def test_brute_force_small():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((30, 8))
    q = rng.standard_normal((2, 8))
    s, i = oracle.brute_force_mips(q, x, 4)
    for r in range(2):
        best = max(range(30), key=lambda j: float(x[j] @ q[r]))
        assert i[r, 0] == best


def test_sq8():
    rng = np.random.default_rng(4)
    v = rng.standard_normal((200, 12))
    v[:, 3] = 0.25                                            # constant column
    lo, hi = oracle.sq8_fit(v)
    assert np.array_equal(lo, v.min(0)) and np.array_equal(hi, v.max(0))
    codes = oracle.sq8_encode(v, lo, hi)
    assert codes[:, 3].max() == 0
    assert codes.min() == 0 and codes.max() == 255
    dec = oracle.sq8_decode(codes, lo, hi)
    step = (hi - lo) / 255
    assert np.all(np.abs(dec - v) <= step / 2 + 1e-12)


def test_rescore_identity():
    # score2 = <q, a> + <q_rot, r~2> equals <q, a + R^T r~2> computed densely.
    x, cent, assign, R, C, enc = _small_index(D=64, bits=2, n=200, nlist=4, seed=3)
    xt1 = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], C, R, cent[assign])
    r2 = (x - xt1) @ R.T
    lo, hi = oracle.sq8_fit(r2)
    codes2 = oracle.sq8_encode(r2, lo, hi)
    q = synth.queries_like("gmix", 2, 64, data_seed=103, n_comp=8)
    qr = q @ R.T
    cand = np.array([[5, 17, 3, 44, -1], [0, 1, 2, 3, 4]])
    s1 = np.stack([xt1[np.maximum(cand[i], 0)] @ q[i] for i in range(2)])
    s, i = oracle.rescore_sq8(qr, s1, cand, codes2, lo, hi, 3)
    r2dec = oracle.sq8_decode(codes2, lo, hi)
    for r in range(2):
        ok = cand[r] >= 0
        dense = (xt1[cand[r][ok]] + r2dec[cand[r][ok]] @ R) @ q[r]
        ref_s, ref_i = oracle.topk(dense, cand[r][ok], 3)
        assert np.array_equal(i[r], ref_i)
        assert np.abs(s[r] - ref_s).max() < 1e-10
    # the rescored scores approach exact MIPS: error shrinks versus the scan
    e1 = np.abs(s1[1] - x[cand[1]] @ q[1]).mean()
    e2 = np.abs(xt1[cand[1]] @ q[1] + r2dec[cand[1]] @ qr[1] - x[cand[1]] @ q[1]).mean()
    assert e2 < e1


def test_kmeans_objective_decreases():
    x = synth.gmix(500, 16, 4, seed=11)
    prev = np.inf
    for it in (1, 3, 8):
        c = oracle.kmeans(x, 4, iters=it, seed=0)
        _, d = oracle.assign_l2(x, c)
        assert d.mean() <= prev + 1e-12
        prev = d.mean()


def _read_kmeans_golden():
    path = os.path.join(os.path.dirname(__file__), "golden", "kmeans_hand.txt")
    cases = []
    for line in open(path):
        line = line.split("#")[0].strip()
        if not line:
            continue
        pts, init, it, want = [f.strip() for f in line.split("|")]
        cases.append(([float(v) for v in pts.split()], [float(v) for v in init.split()], int(it),
                      [eval(v, {}) for v in want.split()]))
    return cases


@pytest.mark.parametrize("pts,init,iters,want", _read_kmeans_golden())
def test_kmeans_hand_computed(pts, init, iters, want):
    """Lloyd iterations worked by hand (tests/golden/kmeans_hand.txt): the
    lowest-id tie rule of the assignment, the mean update and the empty
    cluster keeping its centre."""
    x = np.array(pts)[:, None]
    c = oracle.kmeans(x, len(init), iters=iters, init=np.array(init)[:, None])
    assert np.allclose(c[:, 0], want, rtol=0, atol=1e-12)
