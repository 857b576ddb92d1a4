"""Pins for the oracle's RSLM rescoring codec (two-stage relative coding).

Section "Relative Quantization": a second RSLM stage encodes the error of the
first, r2 = x - a with a = x~1 the first-stage approximation, so that
<q, a + r~2> = <q, a> + <q, r~2> reuses the first-stage score; the global
mode restores the norm of the whole vector with g2 = ||x|| / ||a + r~2||.

Sources of truth: an independent dense reconstruction route in the original
space (x~2 = g2^ (a + R^T s2^ c2^), scored with a plain dot product), the
norm-restoration property of the global scale (to the UE4M12 rounding), the
exactly-zero second residual of a constructed-exact first stage, and the
error reduction the second stage must deliver.
"""

import numpy as np
import pytest

import oracle
import synth
from tests import helpers as H


def _two_stage(D, bits1, bits2, n, seed, mode2="global", passes=2):
    x = synth.aniso(n, D, seed=seed)
    rng = np.random.default_rng(seed)
    cen = x[rng.choice(n, 4, replace=False)]
    a_id, _ = oracle.assign_l2(x, cen)
    R = H.rot(D, passes)
    C1, C2 = synth.codebook(bits1), synth.codebook(bits2)
    enc1 = oracle.encode(x, R, C1, bits1, centroids=cen[a_id], scale_mode="global")
    enc2 = oracle.encode_rescore(x, R, enc1, C1, C2, bits2, centroids=cen[a_id],
                                 scale_mode=mode2)
    return x, cen[a_id], R, C1, C2, enc1, enc2


@pytest.mark.parametrize("bits1,bits2", [(4, 2), (4, 1), (2, 4), (3, 3)])
def test_rescore_lut_route_equals_dense_route(bits1, bits2):
    D = 96
    x, c, R, C1, C2, enc1, enc2 = _two_stage(D, bits1, bits2, 200, 10 + bits2)
    a = oracle.reconstruct(enc1["codes"], enc1["s_code"], enc1["g_code"], C1, R, c)
    x2 = oracle.reconstruct_rescore(enc1, enc2, C1, C2, R, c)
    q = synth.queries_like("aniso", 4, D, data_seed=10 + bits2, query_seed=7)
    n = len(x)
    for qq in q:
        s1 = a @ qq                                     # first-stage score <q, a>
        cand = np.arange(n)[None, :]
        s2, i2 = oracle.rescore_rslm((R @ qq)[None, :], s1[None, :], cand, enc2["codes"],
                                     enc2["s_code"], enc2["g_code"], C2, n)
        dense = x2 @ qq
        assert np.abs(s2[0] - dense[i2[0]]).max() < 1e-12 * np.abs(dense).max()
        # ranking: (score desc, id asc)
        order = np.lexsort((np.arange(n), -dense))
        assert np.array_equal(i2[0], order) or np.allclose(dense[i2[0]], dense[order])


@pytest.mark.parametrize("bits2", [1, 2, 3, 4])
def test_rescore_global_scale_restores_the_norm(bits2):
    x, c, R, C1, C2, enc1, enc2 = _two_stage(128, 4, bits2, 150, 3 + bits2)
    x2 = oracle.reconstruct_rescore(enc1, enc2, C1, C2, R, c)
    rel = np.abs(np.linalg.norm(x2, axis=1) / np.linalg.norm(x, axis=1) - 1.0)
    assert rel.max() <= 2.0 ** -13 * 1.0001


def test_rescore_stage_reduces_the_error():
    """The second stage quantises the first stage's error, so the distortion
    drops roughly by the codebook's relative MSE (2-D K=16: ~0.107 per
    dimension); a dropped or sign-flipped term would raise it instead."""
    x, c, R, C1, C2, enc1, enc2 = _two_stage(256, 4, 2, 300, 21)
    a = oracle.reconstruct(enc1["codes"], enc1["s_code"], enc1["g_code"], C1, R, c)
    x2 = oracle.reconstruct_rescore(enc1, enc2, C1, C2, R, c)
    e1 = ((x - a) ** 2).sum(1)
    e2 = ((x - x2) ** 2).sum(1)
    ratio = e2.sum() / e1.sum()
    assert 0.03 < ratio < 0.2, ratio


def test_rescore_local_mode():
    """Local mode: the second scale is 1.0 (code 0x7000) and the score is
    <q, a> + <q_rot, s2^ c2^>."""
    D = 64
    x, c, R, C1, C2, enc1, enc2 = _two_stage(D, 4, 2, 80, 5, mode2="local")
    assert (enc2["g_code"] == 0x7000).all()
    a = oracle.reconstruct(enc1["codes"], enc1["s_code"], enc1["g_code"], C1, R, c)
    rr2 = oracle.decode_rotated(enc2["codes"], enc2["s_code"], C2, D)
    q = synth.queries_like("aniso", 1, D, data_seed=5, query_seed=9)[0]
    s2, i2 = oracle.rescore_rslm((R @ q)[None], (a @ q)[None], np.arange(len(x))[None],
                                 enc2["codes"], enc2["s_code"], enc2["g_code"], C2, len(x))
    ref = (a + rr2 @ R) @ q
    assert np.abs(s2[0] - ref[i2[0]]).max() < 1e-12 * np.abs(ref).max()


def test_rescore_of_an_exact_first_stage_is_zero():
    """x = c + R^T (s C1[codes]) is reproduced exactly by the first stage
    (g1^ = 1), so the second residual is exactly zero: codes2 = 0, s2^ = 0
    and g2^ = ||x|| / ||a|| = 1."""
    D, bits1 = 128, 4
    rng = np.random.default_rng(4)
    C1 = synth.codebook(bits1).astype(np.float64)
    R = H.rot(D, 2)
    n = 32
    codes = rng.integers(0, 16, (n, D))
    codes[:, 3] = 15
    s = np.array([oracle.dec_ue7m9(oracle.enc_ue7m9(v)) for v in rng.uniform(0.1, 2.0, n)])
    c = rng.standard_normal((n, D)) * 0.3
    x = c + (s[:, None] * C1[codes].reshape(n, D)) @ R
    enc1 = oracle.encode(x, R, C1, bits1, centroids=c, scale_mode="global")
    assert np.array_equal(enc1["codes"], codes)
    assert (enc1["g_code"] == 0x7000).all()
    C2 = synth.codebook(2)
    enc2 = oracle.encode_rescore(x, R, enc1, C1, C2, 2, centroids=c)
    ra = oracle.first_stage_rotated(enc1["codes"], enc1["s_code"], enc1["g_code"], C1, R, c)
    resid = np.abs(x @ R.T - ra).max()
    if resid == 0.0:
        assert (enc2["codes"] == 0).all() and (enc2["s_code"] == 0).all()
        assert (enc2["g_code"] == 0x7000).all()
    else:
        # float64 rounding leaves a residual at the 1e-16 level: its scale
        # must be negligible and the global scale still 1.0
        assert resid < 1e-12
        sh = np.array([oracle.dec_ue7m9(u) for u in enc2["s_code"]])
        assert sh.max() < 1e-12
        assert (enc2["g_code"] == 0x7000).all()


def test_first_stage_rotated_is_the_rotated_reconstruction():
    x, c, R, C1, C2, enc1, enc2 = _two_stage(100, 3, 2, 60, 8)
    a = oracle.reconstruct(enc1["codes"], enc1["s_code"], enc1["g_code"], C1, R, c)
    ra = oracle.first_stage_rotated(enc1["codes"], enc1["s_code"], enc1["g_code"], C1, R, c)
    assert np.abs(ra - a @ R.T).max() < 1e-12
