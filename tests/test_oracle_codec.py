"""Pins for the oracle's encoder, tables and scale formats.

Sources of truth: closed forms of E_max, the published 1-D Lloyd-Max levels
and distortions for N(0,1) (J. Max, 1960), the Lloyd optimality conditions,
the paper's printed packed sizes (Section "End-to-End Comparison": 13/15 B at
D=100 and 192/194 B at D=1536 for 1 bit; tab:rslm_codecs), exhaustive
round trips of the 16-bit scale formats, and a constructed-exact encoding
whose answer is known in advance.
"""

import math
import os

import numpy as np
import pytest
from scipy.stats import norm

import oracle
import synth

S1 = synth.sign_table()
P = synth.permutation_table()


# --- E_max -----------------------------------------------------------------

def test_emax_closed_forms():
    assert abs(oracle.e_max(1) - math.sqrt(2 / math.pi)) < 1e-12
    assert abs(oracle.e_max(2) - 2 / math.sqrt(math.pi)) < 1e-12


@pytest.mark.parametrize("D", [16, 64, 96])
def test_emax_monte_carlo(D):
    rng = np.random.default_rng(D)
    z = np.abs(rng.standard_normal((1 << 17, D))).max(1)
    se = z.std() / math.sqrt(len(z))
    assert abs(oracle.e_max(D) - z.mean()) < 5 * se


def test_emax_monotone():
    v = [oracle.e_max(d) for d in (64, 96, 128, 256, 768, 1024, 2049)]
    assert all(a < b for a, b in zip(v[:-1], v[1:]))


# --- scale formats -----------------------------------------------------------

@pytest.mark.parametrize("enc,dec,mb,bias,emaxc,fbias", [
    (oracle.enc_ue7m9, oracle.dec_ue7m9, 9, 63, 127, 64),
    (oracle.enc_ue4m12, oracle.dec_ue4m12, 12, 7, 15, 120),
])
def test_scale_format_exhaustive(enc, dec, mb, bias, emaxc, fbias):
    prev = -1.0
    for u in range(1 << 16):
        e = u >> mb
        if e < 1 or e > emaxc:
            continue
        v = dec(u)
        assert v > prev
        prev = v
        assert enc(v) == u
        # float32 bit formula: bits = (u << (23 - mb)) + (fbias << 23)
        bits = np.uint32((u << (23 - mb)) + (fbias << 23))
        assert float(bits.view(np.float32)) == v
    assert dec(0) == 0.0 and enc(0.0) == 0


def test_ue7m9_rounding_and_range():
    one = oracle.enc_ue7m9(1.0)
    assert one == (63 << 9)
    ulp = 2.0 ** -9
    assert oracle.enc_ue7m9(1.0 + ulp / 2) == one            # tie -> even (m=0)
    assert oracle.enc_ue7m9(1.0 + 1.5 * ulp) == one + 2      # tie -> even (m=2)
    assert oracle.enc_ue7m9(1.0 + 0.51 * ulp) == one + 1
    assert oracle.enc_ue7m9(1e30) == (127 << 9) | 511        # saturate
    assert oracle.enc_ue7m9(2.0 ** -63) == 0                 # below 2^-62
    assert oracle.dec_ue7m9(oracle.enc_ue7m9(2.0 ** -62)) == 2.0 ** -62
    assert oracle.enc_ue4m12(1.0) == 0x7000


# --- codebooks ---------------------------------------------------------------

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden_rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


# positive output levels and distortion of the N(0,1) Lloyd-Max quantizers
MAX_1960 = {int(r[0]): ([float(v) for v in r[2:]], float(r[1]))
            for r in _golden_rows("lloyd_max_gaussian.txt")}


def _mse_1d(c):
    t = 0.5 * (c[1:] + c[:-1])
    lo = np.concatenate([[-np.inf], t])
    hi = np.concatenate([t, [np.inf]])
    # E[(Z - c_k)^2 ; cell k] in closed form
    def part(a, b, ck):
        pa = norm.pdf(a) if np.isfinite(a) else 0.0
        pb = norm.pdf(b) if np.isfinite(b) else 0.0
        aa = a * pa if np.isfinite(a) else 0.0
        bb = b * pb if np.isfinite(b) else 0.0
        m0 = norm.cdf(b) - norm.cdf(a)
        m1 = pa - pb
        m2 = m0 + aa - bb
        return m2 - 2 * ck * m1 + ck * ck * m0
    return sum(part(a, b, ck) for a, b, ck in zip(lo, hi, c))


@pytest.mark.parametrize("name,K", [("lm1d_k2", 2), ("lm1d_k4", 4), (3, 8), (4, 16)])
def test_lloyd_max_1d(name, K):
    c = synth.codebook(name)[:, 0].astype(np.float64)
    assert c.shape == (K,)
    assert np.all(np.diff(c) > 0)
    assert np.abs(c + c[::-1]).max() == 0.0                   # symmetric
    levels, mse = MAX_1960[K]
    assert np.abs(c[K // 2:] - np.array(levels)).max() < 1.5e-3
    m = _mse_1d(c)
    assert abs(m - mse) < 2e-4 * max(1.0, mse * 100)
    # optimality: each level is the conditional mean of its cell
    t = 0.5 * (c[1:] + c[:-1])
    lo = np.concatenate([[-np.inf], t])
    hi = np.concatenate([t, [np.inf]])
    mass = norm.cdf(hi) - norm.cdf(lo)
    cm = (norm.pdf(lo) - norm.pdf(hi)) / mass
    assert np.abs(cm - c).max() < 1e-3
    # centroid condition => E||q(Z)||^2 = E||Z||^2 - MSE
    assert abs((mass * c * c).sum() - (1 - m)) < 1e-3
    # every level is exactly representable in float16
    assert np.array_equal(c.astype(np.float16).astype(np.float64), c)


@pytest.mark.parametrize("bits,scalar_mse", [(2, 0.1175), (1, 0.3634)])
def test_multidim_codebook_lloyd_conditions(bits, scalar_mse):
    C = synth.codebook(bits).astype(np.float64)
    K, g = C.shape
    assert (K, g) == oracle.codec_shape(bits)
    rng = np.random.default_rng(12345)
    x = rng.standard_normal((1 << 20, g))
    d = ((x[:, None, :] - C[None]) ** 2).sum(-1)
    a = d.argmin(1)
    mse = d.min(1).mean() / g
    assert mse < scalar_mse - 0.005                          # beats the scalar product code
    for k in range(K):
        cell = x[a == k]
        sem = cell.std(0) / math.sqrt(len(cell))
        assert np.all(np.abs(cell.mean(0) - C[k]) < 5 * sem + 2e-3)
    assert np.array_equal(C.astype(np.float16).astype(np.float64), C)


# --- packing -----------------------------------------------------------------

def test_packed_sizes_from_paper():
    assert oracle.canonical_code_bytes(768, 4) == 384
    assert oracle.canonical_code_bytes(1024, 3) == 384
    rows = _golden_rows("record_sizes.txt")
    assert len(rows) == 6
    for _, D, codec, mode, nbytes, lines in rows:
        bits = int(codec[4])
        got = oracle.record_bytes(int(D), bits, mode, lite=codec.endswith("Lite"))
        assert got == int(nbytes), (D, codec, mode)
        if lines != "-":
            assert -(-got // 64) == int(lines)


def test_codec_table_from_paper():
    rows = _golden_rows("codec_specs.txt")
    assert [r[0] for r in rows] == ["Rslm1", "Rslm2", "Rslm3", "Rslm4", "Rslm4Lite"]
    for codec, bits, g, K, scale in rows:
        bits, g = int(bits), int(g)
        if scale == "embedded":
            k_main, k_lead = (int(v) for v in K.split("/"))
            assert oracle.codec_shape(bits) == (k_main, g)
            assert synth.codebook(3).shape == (k_lead, 1)    # the K = 8 lead codebook
            assert oracle.lite_lead("local") == 16
            for D in (64, 100, 256, 768):
                assert oracle.record_bytes(D, bits, "local", lite=True) == -(-D // 2)
            continue
        assert oracle.codec_shape(bits) == (int(K), g)
        assert synth.codebook(bits).shape == (int(K), g)
        assert scale == "suffix2"
        for D in (64, 100, 768, 1536):
            assert oracle.record_bytes(D, bits, "local") == oracle.canonical_code_bytes(D, bits) + 2


def test_pack_bit_positions():
    assert oracle.pack_canonical(np.array([[1, 2]]), 4).tolist() == [[0x21]]
    assert oracle.pack_canonical(np.array([[1, 2, 3]]), 3).tolist() == [[0xD1, 0x00]]
    rng = np.random.default_rng(1)
    for bits in (1, 2, 3, 4):
        K, g = oracle.codec_shape(bits)
        codes = rng.integers(0, K, (5, 37))
        pk = oracle.pack_canonical(codes, bits)
        assert np.array_equal(oracle.unpack_canonical(pk, bits, 37), codes)


# --- encoder -------------------------------------------------------------------

def _constructed(D, bits, passes, n, seed):
    """x = c + R^T (s C[codes]) with s on the UE7M9 grid and an outer level used."""
    rng = np.random.default_rng(seed)
    C = synth.codebook(bits).astype(np.float64)
    K, g = C.shape
    R = oracle.rotation_matrix(D, passes, S1, P)
    codes = rng.integers(0, K, (n, D // g))
    codes[:, rng.integers(0, D // g)] = K - 1                # an outermost level
    s = np.array([oracle.dec_ue7m9(oracle.enc_ue7m9(v)) for v in rng.uniform(0.05, 3.0, n)])
    c = rng.standard_normal((n, D)) * 0.3
    z = s[:, None] * C[codes].reshape(n, D)
    x = c + z @ R
    return x, c, codes, s, R, C


@pytest.mark.parametrize("D,bits,passes", [(96, 4, 2), (128, 4, 1), (256, 4, 2), (64, 3, 2), (100, 3, 1)])
def test_constructed_exact_round_trip(D, bits, passes):
    x, c, codes, s, R, C = _constructed(D, bits, passes, 64, D + bits)
    enc = oracle.encode(x, R, C, bits, centroids=c, scale_mode="global")
    assert np.array_equal(enc["codes"], codes)
    assert np.array_equal([oracle.dec_ue7m9(u) for u in enc["s_code"]], s)
    assert np.all(enc["g_code"] == 0x7000)
    # the scan then equals exact MIPS on x
    q = np.random.default_rng(7).standard_normal(D)
    qr = R @ q
    sh = np.array([oracle.dec_ue7m9(u) for u in enc["s_code"]])
    sc = oracle.scan_scores_lut(qr, c @ q, enc["codes"], sh, np.ones(len(x)), C)
    assert np.abs(sc - x @ q).max() < 1e-10 * np.abs(x @ q).max()


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
@pytest.mark.parametrize("D", [98, 101, 128])
def test_norm_correction(bits, D):
    rng = np.random.default_rng(bits * 1000 + D)
    x = rng.standard_normal((50, D))
    c = x + 0.3 * rng.standard_normal((50, D))
    R = oracle.rotation_matrix(D, 2, S1, P)
    C = synth.codebook(bits)
    enc = oracle.encode(x, R, C, bits, centroids=c, scale_mode="global")
    rr = oracle.decode_rotated(enc["codes"], enc["s_code"], C, D)
    rn = np.linalg.norm(x - c, axis=1)
    assert np.all(np.abs(np.linalg.norm(rr, axis=1) / rn - 1) <= 2.0 ** -10)
    xt = oracle.reconstruct(enc["codes"], enc["s_code"], enc["g_code"], C, R, c)
    assert np.all(np.abs(np.linalg.norm(xt, axis=1) / np.linalg.norm(x, axis=1) - 1) <= 2.0 ** -13)
    # the scale rounds to nearest: the pre-rounding value is within half a step
    for s, u in zip(enc["s"], enc["s_code"]):
        assert abs(oracle.dec_ue7m9(u) - s) <= 2.0 ** -10 * s * 1.0000001


def test_local_mode_and_zero_residual():
    D = 64
    rng = np.random.default_rng(3)
    x = rng.standard_normal((4, D))
    c = x.copy()
    c[1] += 0.1
    R = oracle.rotation_matrix(D, 2, S1, P)
    C = synth.codebook(4)
    enc = oracle.encode(x, R, C, 4, centroids=c, scale_mode="global")
    assert np.all(enc["codes"][0] == 0) and enc["s_code"][0] == 0
    g0 = oracle.dec_ue4m12(enc["g_code"][0])
    assert abs(g0 - 1.0) <= 2.0 ** -12                       # ||x|| / ||c|| with c = x
    loc = oracle.encode(x, R, C, 4, centroids=c, scale_mode="local")
    assert np.all(loc["g_code"] == 0x7000)
    assert np.array_equal(loc["codes"], enc["codes"])


def test_padding_uses_valid_coordinates_only():
    # D = 98 with 4-D sub-vectors: two padded coordinates never reach norms.
    D = 98
    rng = np.random.default_rng(5)
    x = rng.standard_normal((20, D))
    R = oracle.rotation_matrix(D, 2, S1, P)
    C = synth.codebook(1)
    enc = oracle.encode(x, R, C, 1, scale_mode="local")
    assert enc["codes"].shape == (20, 25)
    assert np.all(enc["u"][:, D:] == 0)
    rr = oracle.decode_rotated(enc["codes"], enc["s_code"], C, D)
    assert rr.shape == (20, D)
