"""The top-k comparison used by every GPU scan and rescore parity test
(``helpers.check_topk``) must reject the mistakes it exists to catch.  Run on
the CPU with the oracle's own outputs standing in for a device result: the
oracle's answer passes, and each planted mistake (permuted ids, a score
paired with the wrong id, a wrong order, a dropped or foreign id) fails."""

import numpy as np
import pytest

import oracle
import synth
from tests import helpers as H


@pytest.fixture(scope="module")
def case():
    D, bits, n, nlist, Q, nprobe, k = 64, 4, 3000, 8, 6, 3, 20
    x = synth.gmix(n, D, 8, seed=5)
    rng = np.random.default_rng(5)
    cen = x[rng.choice(n, nlist, replace=False)].astype(np.float64)
    assign, _ = oracle.assign_l2(x, cen)
    Rm = H.rot(D, 2)
    C = synth.codebook(bits)
    enc = oracle.encode(x, Rm, C, bits, centroids=cen[assign], scale_mode="global")
    sh, gh = H.dec_scales(enc["s_code"].astype(np.uint32) | (enc["g_code"].astype(np.uint32) << 16))
    lists = {L: {"ids": np.where(assign == L)[0], "codes": enc["codes"][assign == L],
                 "s_hat": sh[assign == L], "g_hat": gh[assign == L]} for L in range(nlist)}
    q = synth.queries_like("gmix", Q, D, data_seed=5, n_comp=8)
    qr = q.astype(np.float64) @ Rm.T
    ref_s, ref_i, _ = oracle.ivf_search(q, qr, cen, lists, C, nprobe, k)
    _, cands = oracle.ivf_candidates(q, qr, cen, lists, C, nprobe)
    xn = np.linalg.norm(x, axis=1).max() * 2
    tols = [lambda s, qn=np.linalg.norm(q[i]): H.score_tol(s, qn, xn) for i in range(Q)]
    return ref_s, ref_i, cands, tols


def _run(case, mutate):
    ref_s, ref_i, cands, tols = case
    gs, gi = ref_s[0].astype(np.float32).copy(), ref_i[0].copy()
    gs, gi = mutate(gs, gi, cands[0])
    return H.check_topk(gs, gi, ref_s[0], ref_i[0], tols[0], *cands[0])


def test_oracle_answer_passes(case):
    ref_s, ref_i, cands, tols = case
    for i in range(len(ref_i)):
        assert H.check_topk(ref_s[i].astype(np.float32), ref_i[i], ref_s[i], ref_i[i], tols[i],
                            *cands[i]) == 0


def _swap_ids(gs, gi, c):
    gi[[0, 5]] = gi[[5, 0]]
    return gs, gi


def _rotate_ids(gs, gi, c):
    return gs, np.roll(gi, 1)


def _reverse_order(gs, gi, c):
    return gs[::-1].copy(), gi[::-1].copy()


def _foreign_id(gs, gi, c):
    gi[3] = 10 ** 6
    return gs, gi


def _duplicate(gs, gi, c):
    gi[4] = gi[3]
    return gs, gi


def _deep_candidate(gs, gi, c):
    # replace the last id by a low-scoring candidate, keeping its own score
    s, ids = c
    j = int(np.argmin(s))
    gi[-1], gs[-1] = ids[j], s[j]
    return gs, gi


@pytest.mark.parametrize("mutate", [_swap_ids, _rotate_ids, _reverse_order, _foreign_id,
                                    _duplicate, _deep_candidate])
def test_planted_mistakes_fail(case, mutate):
    with pytest.raises(AssertionError):
        _run(case, mutate)
