"""Pins for the oracle's packed records and the Rslm4Lite codec.

Sources of truth: the record sizes the paper prints (Rslm1 at D = 100 and
D = 1536 with one and two scale suffixes; Rslm4 at D = 256 against
Rslm4Lite's ceil(D / 2)), hand-placed bits of the embedded scales, round
trips, and for Rslm4Lite (16 or 32 leading coordinates on the K = 8
codebook): a constructed-exact encoding whose codes and scales are known in
advance, norm restoration, the LUT route against a dense reconstruction, and
the per-coordinate distortion of the two codebooks.
"""

import numpy as np
import pytest

import oracle
import synth
from tests import helpers as H


def test_record_sizes_from_paper():
    # glove (D = 100), Rslm1: 13 B of codes + 2 B scale = 15 B; two scales 17 B
    assert oracle.record_bytes(100, 1, "local") == 15
    assert oracle.record_bytes(100, 1, "global") == 17
    assert abs(17 / 13 - 1.31) < 0.005
    # openai (D = 1536), Rslm1: 192 + 2 = 194 B; two scales 196 B (+2 %)
    assert oracle.record_bytes(1536, 1, "local") == 194
    assert oracle.record_bytes(1536, 1, "global") == 196
    assert abs(196 / 192 - 1.02) < 0.005
    # D = 256: Rslm4 needs 130 B (three 64-B cache lines), Rslm4Lite 128 B (two)
    assert oracle.record_bytes(256, 4, "local") == 130
    assert oracle.record_bytes(256, 4, "local", lite=True) == 128
    assert oracle.record_bytes(101, 4, "global", lite=True) == 51


def test_lite_embedded_bit_positions():
    codes = np.zeros((1, 64), dtype=np.int64)
    rec = oracle.pack_records(codes, [0x0001], [0x7000], 4, "local", lite=True)
    assert rec.shape == (1, 32) and rec[0, 0] == 0x08 and rec[0, 1:].sum() == 0
    rec = oracle.pack_records(codes, [0x8000], [0x7000], 4, "local", lite=True)
    assert rec[0, 7] == 0x80 and rec[0, :7].sum() == 0
    rec = oracle.pack_records(codes, [0], [0x0001], 4, "global", lite=True)
    assert rec[0, 8] == 0x08 and rec[0, :8].sum() == 0 and rec[0, 9:].sum() == 0
    codes[0, 1] = 5
    rec = oracle.pack_records(codes, [0x0002], [0x7000], 4, "local", lite=True)
    assert rec[0, 0] == 0xD0    # nibble 1 = 5 | 8


def test_suffix_byte_order():
    codes = np.zeros((1, 8), dtype=np.int64)
    rec = oracle.pack_records(codes, [0x1234], [0xABCD], 4, "global")
    assert rec[0, 4:].tolist() == [0x34, 0x12, 0xCD, 0xAB]


@pytest.mark.parametrize("bits,D,mode,lite", [(1, 100, "local", False), (2, 98, "global", False),
                                              (3, 101, "global", False), (4, 256, "local", False),
                                              (4, 256, "local", True), (4, 96, "global", True),
                                              (4, 65, "global", True)])
def test_records_round_trip(bits, D, mode, lite):
    rng = np.random.default_rng(D + bits)
    K, g = oracle.codec_shape(bits)
    n_sub = -(-D // g)
    codes = rng.integers(0, K, (20, n_sub))
    if lite:
        codes[:, :oracle.lite_lead(mode)] = rng.integers(0, 8, (20, oracle.lite_lead(mode)))
    s = rng.integers(0, 1 << 16, 20).astype(np.uint16)
    gg = rng.integers(0, 1 << 16, 20).astype(np.uint16) if mode == "global" else \
        np.full(20, 0x7000, np.uint16)
    rec = oracle.pack_records(codes, s, gg, bits, mode, lite)
    assert rec.shape == (20, oracle.record_bytes(D, bits, mode, lite))
    c2, s2, g2 = oracle.unpack_records(rec, bits, D, mode, lite)
    assert np.array_equal(c2, codes) and np.array_equal(s2, s) and np.array_equal(g2, gg)


@pytest.mark.parametrize("D,mode,passes", [(128, "local", 1), (256, "global", 2), (96, "global", 2)])
def test_lite_constructed_exact(D, mode, passes):
    """x = c + R^T (s c^) with c^ from the K = 8 codebook on the leading
    coordinates and K = 16 elsewhere (an outermost K = 16 level present) is
    encoded back to the same codes with s^ = s and g^ = 1."""
    rng = np.random.default_rng(D)
    C16, C8 = synth.codebook(4).astype(np.float64), synth.codebook(3).astype(np.float64)
    R = H.rot(D, passes)
    n, lead = 32, oracle.lite_lead(mode)
    codes = rng.integers(0, 16, (n, D))
    codes[:, lead:lead + 1] = 15
    codes[:, :lead] = rng.integers(0, 8, (n, lead))
    chat = C16[codes, 0]
    chat[:, :lead] = C8[codes[:, :lead], 0]
    s = np.array([oracle.dec_ue7m9(oracle.enc_ue7m9(v)) for v in rng.uniform(0.05, 2.0, n)])
    c = rng.standard_normal((n, D)) * 0.3
    x = c + (s[:, None] * chat) @ R
    enc = oracle.encode(x, R, C16, 4, centroids=c, scale_mode=mode, C_lead=C8)
    assert np.array_equal(enc["codes"], codes)
    assert np.array_equal([oracle.dec_ue7m9(u) for u in enc["s_code"]], s)
    if mode == "global":
        assert (enc["g_code"] == 0x7000).all()


@pytest.mark.parametrize("mode", ["local", "global"])
def test_lite_norm_restoration_and_routes(mode):
    D = 192
    x = synth.aniso(150, D, seed=4).astype(np.float64)
    c = x[:3].mean(0, keepdims=True).repeat(150, 0) * 0.5
    R = H.rot(D, 2)
    C16, C8 = synth.codebook(4), synth.codebook(3)
    lead = oracle.lite_lead(mode)
    enc = oracle.encode(x, R, C16, 4, centroids=c, scale_mode=mode, C_lead=C8)
    assert enc["codes"][:, :lead].max() < 8
    xt = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], C16, R, c, C8, lead)
    if mode == "global":
        rel = np.abs(np.linalg.norm(xt, axis=1) / np.linalg.norm(x, axis=1) - 1)
        assert rel.max() <= 2.0 ** -13 * 1.0001
    else:
        rr = oracle.decode_rotated(enc["codes"], enc["s_code"], C16, D, C8, lead)
        rel = np.abs(np.linalg.norm(rr, axis=1) / np.linalg.norm(x - c, axis=1) - 1)
        assert rel.max() <= 2.0 ** -10
    q = synth.queries_like("aniso", 3, D, data_seed=4, query_seed=5).astype(np.float64)
    sh, gh = H.dec_scales(enc["s_code"].astype(np.uint32) | (enc["g_code"].astype(np.uint32) << 16))
    for qq in q:
        lut = oracle.scan_scores_lut(R @ qq, c @ qq, enc["codes"], sh, gh, C16, C8, lead)
        dense = xt @ qq
        assert np.abs(lut - dense).max() < 1e-12 * np.abs(dense).max()


def test_lite_distortion_per_codebook():
    """Per-coordinate error of the normalised coordinates: the leading (K = 8)
    coordinates are quantised more coarsely than the rest (K = 16), by about
    the ratio of the two Lloyd-Max distortions (0.0345 / 0.0095)."""
    D = 512
    x = synth.aniso(400, D, seed=9, normalize=True)
    R = H.rot(D, 2)
    C16, C8 = synth.codebook(4).astype(np.float64), synth.codebook(3).astype(np.float64)
    enc = oracle.encode(x, R, C16, 4, scale_mode="local", C_lead=C8)
    u = enc["u"][:, :D]
    chat = C16[enc["codes"], 0]
    chat[:, :16] = C8[enc["codes"][:, :16], 0]
    e_lead = ((u[:, :16] - chat[:, :16]) ** 2).mean()
    e_rest = ((u[:, 16:] - chat[:, 16:]) ** 2).mean()
    assert 2.0 < e_lead / e_rest < 6.0, (e_lead, e_rest)
