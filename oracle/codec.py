"""Oracle: the RSLM encoder and its scale formats (float64).

Follows Section "Rslm codec family" of the paper:
  * "Quantization Using Lloyd-Max Codebook": the EVT initial scale
    s_initial = max_i |z_i| / E_max(D); normalisation by 1/s_initial; nearest
    centroid per sub-vector of size g (b=1: 4-D K=16, b=2: 2-D K=16, b=3: 1-D
    K=8, b=4: 1-D K=16); zero padding to a multiple of g with only the D valid
    coordinates used for norms and scores.
  * "Norm Correction": the reconstruction s * x^ with s = ||x|| / ||x^||.
  * "Scale Encoding": a 16-bit unsigned float UE7M9 without subnormals.
  * "Relative Quantization": the residual r = x - a is what gets quantised;
    the local mode keeps only the residual's scale, the global mode adds a
    second scale ||x|| / ||a + r~|| stored as UE4M12.
  * "Codecs Description" / tab:rslm_codecs: packed codes followed by scales.

Readings where the paper is not explicit:
  * E_max(D) = E[max_{i<=D} |Z_i|] for i.i.d. standard normal Z_i, i.e. the
    integral over t >= 0 of 1 - (2 Phi(t) - 1)^D, D the true dimension;
  * s is taken in codebook units, s = ||r|| / ||C[codes]|| over the D valid
    coordinates (s_initial cancels from the reconstruction s * C[codes]);
  * UE7M9: u = e << 9 | m encodes 2^(e-63) (1 + m/512) for e in [1, 127],
    u = 0 encodes 0; rounding to nearest-even on 10 significant bits,
    overflow saturates to the largest code, results below 2^-62 flush to 0;
  * UE4M12: u = e << 12 | m encodes 2^(e-7) (1 + m/4096), e in [1, 15];
  * the global scale uses the decoded local scale (what a scorer sees);
  * the local mode stores the UE4M12 code of 1.0 (0x7000) as its second
    scale so that one record format serves both modes;
  * a vector whose residual is exactly zero gets codes 0 and local scale 0;
    a zero denominator gives a zero global scale;
  * canonical packing: a little-endian bit stream, code j at bits
    [w*j, w*j + w) with w = log2(K).
"""

import math

import numpy as np
from scipy import integrate, special


def codec_shape(bits):
    """(K, g): centroid count and sub-vector size for a bit width."""
    return {1: (16, 4), 2: (16, 2), 3: (8, 1), 4: (16, 1)}[bits]


def e_max(D):
    """Expected maximum |N(0,1)| over D i.i.d. draws (quadrature, float64)."""
    f = lambda t: 1.0 - special.erf(t / math.sqrt(2.0)) ** D
    val = 0.0
    edges = [0.0, 1.0, 2.0, 3.0, 4.0, 5.0, 6.0, 8.0, 12.0, 40.0]
    for a, b in zip(edges[:-1], edges[1:]):
        v, _ = integrate.quad(f, a, b, epsabs=1e-14, epsrel=1e-13, limit=200)
        val += v
    return val


def _enc_ue(s, mbits, bias, emax_code):
    s = float(s)
    if not (s > 0.0):
        return 0
    if math.isinf(s):
        return (emax_code << mbits) | ((1 << mbits) - 1)
    f, e = math.frexp(s)          # s = f * 2^e, f in [0.5, 1)
    e -= 1
    frac = 2.0 * f - 1.0          # s = 2^e (1 + frac)
    scaled = frac * (1 << mbits)
    m = int(np.rint(scaled))      # round half to even
    if m == (1 << mbits):
        m = 0
        e += 1
    code_e = e + bias
    if code_e < 1:
        return 0
    if code_e > emax_code:
        return (emax_code << mbits) | ((1 << mbits) - 1)
    return (code_e << mbits) | m


def _dec_ue(u, mbits, bias):
    u = int(u)
    if u == 0:
        return 0.0
    e = u >> mbits
    m = u & ((1 << mbits) - 1)
    return math.ldexp(1.0 + m / float(1 << mbits), e - bias)


def enc_ue7m9(s):
    return _enc_ue(s, 9, 63, 127)


def dec_ue7m9(u):
    return _dec_ue(u, 9, 63)


def enc_ue4m12(s):
    return _enc_ue(s, 12, 7, 15)


def dec_ue4m12(u):
    return _dec_ue(u, 12, 7)


UE4M12_ONE = 0x7000


def lite_lead(scale_mode):
    """Rslm4Lite: number of leading coordinates coded with the K = 8 codebook,
    whose freed top code bits carry the scales -- 16 for one UE7M9 scale,
    32 when the global UE4M12 scale is embedded as well (Sections "Codecs
    Description" and "Relative Quantization")."""
    return 32 if scale_mode == "global" else 16


def encode(x, R, C, bits, centroids=None, scale_mode="global", chunk=512, C_lead=None):
    """Encode rows of x relative to ``centroids`` (or 0) with rotation R.

    ``C_lead`` (Rslm4Lite, 4 bits only): the K = 8 1-D codebook used for the
    first ``lite_lead(scale_mode)`` coordinates instead of C.

    Returns a dict with ``codes`` (n, n_sub) int64, ``s_code`` / ``g_code``
    (n,) uint16 scale codes and the diagnostic values ``u`` (normalised
    rotated coordinates, zero padded), ``s`` and ``g`` (pre-rounding scales).
    """
    x = np.asarray(x, dtype=np.float64)
    n, D = x.shape
    C = np.asarray(C, dtype=np.float64)
    K, g = C.shape
    assert (K, g) == codec_shape(bits)
    n_sub = -(-D // g)
    D_pad = n_sub * g
    emax = e_max(D)
    lead = 0
    if C_lead is not None:
        C_lead = np.asarray(C_lead, dtype=np.float64)
        assert bits == 4 and C_lead.shape == (8, 1) and D >= 64
        lead = lite_lead(scale_mode)
    cen = np.zeros_like(x) if centroids is None else np.asarray(centroids, dtype=np.float64)
    codes = np.zeros((n, n_sub), dtype=np.int64)
    u_all = np.zeros((n, D_pad))
    s_pre = np.zeros(n)
    g_pre = np.ones(n)
    s_code = np.zeros(n, dtype=np.uint16)
    g_code = np.full(n, UE4M12_ONE, dtype=np.uint16)
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        r = x[lo:hi] - cen[lo:hi]
        z = r @ R.T                                   # z = R r, row-wise
        m = np.abs(z).max(axis=1)
        u = np.zeros((hi - lo, D_pad))
        nz = m > 0
        u[nz, :D] = z[nz] / (m[nz] / emax)[:, None]   # z / s_initial
        sub = u.reshape(hi - lo, n_sub, g)
        dist = ((sub[:, :, None, :] - C[None, None, :, :]) ** 2).sum(-1)
        cd = np.argmin(dist, axis=-1)                 # first minimum: lower k on ties
        chat = C[cd].reshape(hi - lo, D_pad)
        if lead:
            dl = ((sub[:, :lead, None, :] - C_lead[None, None, :, :]) ** 2).sum(-1)
            cd[:, :lead] = np.argmin(dl, axis=-1)
            chat[:, :lead] = C_lead[cd[:, :lead], 0]
        cd[~nz] = 0
        chat = chat[:, :D]
        rn = np.linalg.norm(r, axis=1)
        cn = np.linalg.norm(chat, axis=1)
        sh = np.zeros(hi - lo)
        for i in range(hi - lo):
            row = lo + i
            s = rn[i] / cn[i] if (nz[i] and cn[i] > 0) else 0.0
            su = enc_ue7m9(s)
            s_pre[row], s_code[row] = s, su
            sh[i] = dec_ue7m9(su)
        if scale_mode == "global":
            a = cen[lo:hi] + (sh[:, None] * chat) @ R        # c + R^T (s^ c^), row-wise
            an = np.linalg.norm(a, axis=1)
            xn = np.linalg.norm(x[lo:hi], axis=1)
            for i in range(hi - lo):
                gv = xn[i] / an[i] if an[i] > 0 else 0.0
                g_pre[lo + i], g_code[lo + i] = gv, enc_ue4m12(gv)
        codes[lo:hi] = cd
        u_all[lo:hi] = u
    return {"codes": codes, "s_code": s_code, "g_code": g_code,
            "u": u_all, "s": s_pre, "g": g_pre}


def canonical_code_bytes(D, bits):
    K, g = codec_shape(bits)
    w = int(K).bit_length() - 1
    return -(-(-(-D // g) * w) // 8)


def pack_canonical(codes, bits):
    """(n, n_sub) codes -> (n, bytes) uint8, code j at bits [w j, w j + w)."""
    K, _ = codec_shape(bits)
    w = int(K).bit_length() - 1
    codes = np.asarray(codes, dtype=np.int64)
    n, n_sub = codes.shape
    bitarr = ((codes[:, :, None] >> np.arange(w)[None, None, :]) & 1).reshape(n, n_sub * w)
    nbytes = -(-(n_sub * w) // 8)
    padded = np.zeros((n, nbytes * 8), dtype=np.uint8)
    padded[:, :n_sub * w] = bitarr
    return np.packbits(padded, axis=1, bitorder="little")


def unpack_canonical(packed, bits, n_sub):
    K, _ = codec_shape(bits)
    w = int(K).bit_length() - 1
    bitarr = np.unpackbits(np.asarray(packed, dtype=np.uint8), axis=1, bitorder="little")
    bitarr = bitarr[:, :n_sub * w].reshape(-1, n_sub, w).astype(np.int64)
    return (bitarr << np.arange(w)[None, None, :]).sum(-1)


def record_bytes(D, bits, scale_mode, lite=False):
    """Bytes of one packed record (table tab:rslm_codecs): the codes followed
    by a 2-byte scale suffix (two with the global scale); Rslm4Lite embeds
    its scales, ceil(D / 2) bytes."""
    if lite:
        return -(-D // 2)
    return canonical_code_bytes(D, bits) + (4 if scale_mode == "global" else 2)


def pack_records(codes, s_code, g_code, bits, scale_mode, lite=False):
    """Packed records (Section "Codecs Description": pack the codes and the
    scale factor).  Reading: scales are little-endian uint16 suffixes, the
    UE7M9 scale first, then the UE4M12 global scale.  Rslm4Lite: the leading
    lite_lead coordinates hold 3-bit codes and bit 3 of coordinate j's nibble
    holds bit j of the UE7M9 scale (j < 16) or bit j - 16 of the UE4M12 scale
    (16 <= j < 32), least significant bit first."""
    codes = np.asarray(codes, dtype=np.int64).copy()
    n = codes.shape[0]
    s_code = np.asarray(s_code, dtype=np.int64)
    g_code = np.asarray(g_code, dtype=np.int64)
    if lite:
        assert bits == 4
        lead = lite_lead(scale_mode)
        assert codes[:, :lead].max(initial=0) < 8
        for j in range(lead):
            word = s_code if j < 16 else g_code
            codes[:, j] |= ((word >> (j % 16)) & 1) << 3
        return pack_canonical(codes, bits)
    body = pack_canonical(codes, bits)
    suf = [s_code] + ([g_code] if scale_mode == "global" else [])
    tail = np.concatenate([np.stack([v & 0xFF, v >> 8], 1) for v in suf], 1).astype(np.uint8)
    return np.concatenate([body, tail.reshape(n, -1)], 1)


def unpack_records(rec, bits, D, scale_mode, lite=False):
    """Inverse of pack_records: (codes, s_code, g_code); g_code is the code of
    1.0 (0x7000) for local records."""
    K, g = codec_shape(bits)
    n_sub = -(-D // g)
    rec = np.asarray(rec, dtype=np.uint8)
    nb = canonical_code_bytes(D, bits)
    codes = unpack_canonical(rec[:, :nb], bits, n_sub)
    n = rec.shape[0]
    g_code = np.full(n, UE4M12_ONE, dtype=np.uint16)
    if lite:
        lead = lite_lead(scale_mode)
        top = (codes[:, :lead] >> 3) & 1
        codes[:, :lead] &= 7
        w = (top << np.arange(lead) % 16).astype(np.int64)
        s_code = w[:, :16].sum(1).astype(np.uint16)
        if lead == 32:
            g_code = w[:, 16:32].sum(1).astype(np.uint16)
        return codes, s_code, g_code
    tail = rec[:, nb:].astype(np.int64)
    s_code = (tail[:, 0] | (tail[:, 1] << 8)).astype(np.uint16)
    if scale_mode == "global":
        g_code = (tail[:, 2] | (tail[:, 3] << 8)).astype(np.uint16)
    return codes, s_code, g_code


def decode_rotated(codes, s_code, C, D, C_lead=None, lead=0):
    """s^ * C[codes] over the D valid coordinates (rotated space); the first
    ``lead`` coordinates decode through C_lead (Rslm4Lite)."""
    C = np.asarray(C, dtype=np.float64)
    n = codes.shape[0]
    chat = C[codes].reshape(n, -1)
    if lead:
        chat[:, :lead] = np.asarray(C_lead, dtype=np.float64)[codes[:, :lead], 0]
    chat = chat[:, :D]
    sh = np.array([dec_ue7m9(u) for u in s_code])
    return sh[:, None] * chat


def reconstruct(codes, s_code, g_code, C, R, centroids=None, C_lead=None, lead=0):
    """x~ = g^ (c + R^T s^ c^) in the original space."""
    rr = decode_rotated(codes, s_code, C, R.shape[0], C_lead, lead)
    base = 0.0 if centroids is None else np.asarray(centroids, dtype=np.float64)
    gh = np.array([dec_ue4m12(u) for u in g_code])
    return gh[:, None] * (base + rr @ R)


def first_stage_rotated(codes, s_code, g_code, C, R, centroids=None, C_lead=None, lead=0):
    """R a for the first-stage approximation a = x~1 = g^ (c + R^T s^ c^):
    R a = g^ (R c + s^ c^) (R is orthogonal), the base of the rescoring codec."""
    rr = decode_rotated(codes, s_code, C, R.shape[0], C_lead, lead)
    base = 0.0 if centroids is None else np.asarray(centroids, dtype=np.float64) @ R.T
    gh = np.array([dec_ue4m12(u) for u in g_code])
    return gh[:, None] * (base + rr)


def encode_rescore(x, R, enc1, C1, C2, bits2, centroids=None, scale_mode="global"):
    """Rescoring codec of Section "Relative Quantization": the second residual
    r2 = x - a, with a = x~1 the first-stage approximation, RSLM-encoded
    relative to a.

    Reading: the codec's rotation is a fixed table, so the first stage's R
    serves both stages and the second residual is quantised in the rotated
    space without a further rotation: the rows R x are encoded against the
    bases R a with R = I, which gives s2 = ||r2|| / ||C2[codes2]|| and, in
    the global mode, g2 = ||x|| / ||a + R^T s2^ c2^|| (the decoded s2^).
    Returns the dict of ``encode`` for the second stage.
    """
    x = np.asarray(x, dtype=np.float64)
    ra = first_stage_rotated(enc1["codes"], enc1["s_code"], enc1["g_code"], C1, R, centroids)
    eye = np.eye(x.shape[1])
    return encode(x @ R.T, eye, C2, bits2, centroids=ra, scale_mode=scale_mode)


def reconstruct_rescore(enc1, enc2, C1, C2, R, centroids=None):
    """x~2 = g2^ (a + R^T s2^ c2^) in the original space, a = x~1."""
    a = reconstruct(enc1["codes"], enc1["s_code"], enc1["g_code"], C1, R, centroids)
    rr = decode_rotated(enc2["codes"], enc2["s_code"], C2, R.shape[0])
    gh = np.array([dec_ue4m12(u) for u in enc2["g_code"]])
    return gh[:, None] * (a + rr @ R)

