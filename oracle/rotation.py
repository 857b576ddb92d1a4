"""Oracle: the block-wise cascaded Walsh-Hadamard rotation, as a dense matrix.

Follows Section "Pre-Quantization Transformations" of the paper:
  * "Fast Walsh Hadamard Transform": the Sylvester recursion for the
    unnormalised Hadamard matrix and the orthonormal H_n = H^_n / sqrt(n);
    blocks of B = 128, shrunk to the largest power of two <= D when D < 128;
    a final block of the same size overlapping the previous one, ending at D,
    when B does not divide D.
  * "Sign Flips and Dimension Permutation": 256 signs S1 tiled over the
    coordinates; a 128-element permutation P within a block (bit reversal for
    B < 128); the strided transpose x'[k*M + b] = x[b*B + P(k)] of the first
    M*B coordinates with the tail unchanged.
  * "Cascaded Rotation Pipeline": S1, block FWHT, permute+transpose, S2
    (S1 offset by 127), block FWHT; a single pass (S1 + block FWHT) for
    4-bit codecs with D <= 256.

This module never uses a butterfly: every block transform is a product with
the explicit Hadamard matrix, and ``rotation_matrix`` applies the steps to the
identity to obtain R (D x D, float64).

Readings where the paper is not explicit:
  * S2[i] = S1[(i + 127) mod 256];
  * each block application is orthonormal (scaled by 1/sqrt(B));
  * blocks are applied full blocks first in ascending order, then the
    overlapping block; the same block list in both passes;
  * ``passes`` 0 means no rotation at all (identity); the permutation and
    transpose are applied whenever two passes run (for D <= 128 the transpose
    with M = 1 reduces to the in-block permutation).
"""

import numpy as np


def block_size(D):
    """Active FWHT block size: 128, or the largest power of two <= D."""
    if D >= 128:
        return 128
    return 1 << (int(D).bit_length() - 1)


def block_list(D):
    """[(offset, B), ...]: the full blocks in order, then the overlap block."""
    B = block_size(D)
    M = D // B
    out = [(i * B, B) for i in range(M)]
    if D % B:
        out.append((D - B, B))
    return out


def resolve_passes(bits, D, passes=-1):
    """Explicit pass count, or the paper's rule when ``passes`` is -1."""
    if passes in (0, 1, 2):
        return passes
    return 1 if (bits == 4 and D <= 256) else 2


def hadamard(n):
    """Unnormalised Sylvester-Hadamard matrix of order n (power of two)."""
    H = np.ones((1, 1))
    while H.shape[0] < n:
        H = np.block([[H, H], [H, -H]])
    assert H.shape[0] == n, "order must be a power of two"
    return H


def intra_block_perm(B, perm128):
    """P for B == 128; the bit-reversal permutation on log2(B) bits otherwise."""
    if B == 128:
        return np.asarray(perm128, dtype=np.int64)
    nb = B.bit_length() - 1
    out = np.zeros(B, dtype=np.int64)
    for k in range(B):
        r = 0
        for t in range(nb):
            if k >> t & 1:
                r |= 1 << (nb - 1 - t)
        out[k] = r
    return out


def _block_pass(y, D):
    for off, B in block_list(D):
        y[off:off + B] = hadamard(B) @ y[off:off + B] / np.sqrt(B)
    return y


def rotate(x, passes, signs, perm128):
    """Apply the cascade to one vector x (length D), float64, step by step."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[0]
    if passes == 0:
        return x.copy()
    S1 = np.asarray(signs, dtype=np.float64)
    idx = np.arange(D)
    y = S1[idx % 256] * x
    y = _block_pass(y, D)
    if passes == 2:
        B = block_size(D)
        M = D // B
        P = intra_block_perm(B, perm128)
        t = y.copy()
        for b in range(M):
            for k in range(B):
                t[k * M + b] = y[b * B + P[k]]
        S2 = S1[(idx + 127) % 256]
        y = _block_pass(S2 * t, D)
    return y


def rotation_matrix(D, passes, signs, perm128):
    """R (D x D float64): column i is ``rotate(e_i)``; the inverse is R.T."""
    R = np.zeros((D, D))
    eye = np.eye(D)
    for i in range(D):
        R[:, i] = rotate(eye[i], passes, signs, perm128)
    return R
