"""Pins for the oracle's rotation (Section "Pre-Quantization Transformations").

Each test checks the oracle against something other than itself: a library
routine (scipy's Hadamard), algebraic invariants the paper states
(orthogonality, norm preservation, exact invertibility), hand-derived index
maps of the strided transpose, and the closed form of the single pass.
"""

import numpy as np
import pytest
import scipy.linalg

import oracle
import synth

S1 = synth.sign_table()
P = synth.permutation_table()


@pytest.mark.parametrize("n", [1, 2, 4, 8, 16, 32, 64, 128])
def test_hadamard_is_sylvester(n):
    H = oracle.hadamard(n)
    assert np.array_equal(H, scipy.linalg.hadamard(n))
    assert np.array_equal(H @ H.T, n * np.eye(n))
    assert np.array_equal(H, H.T)


def test_tables_shape():
    assert S1.shape == (256,) and set(np.unique(S1)) == {-1, 1}
    assert sorted(P.tolist()) == list(range(128))


@pytest.mark.parametrize("D,expect", [
    (96, [(0, 64), (32, 64)]),
    (100, [(0, 64), (36, 64)]),
    (128, [(0, 128)]),
    (300, [(0, 128), (128, 128), (172, 128)]),
    (768, [(i * 128, 128) for i in range(6)]),
    (2049, [(i * 128, 128) for i in range(16)] + [(1921, 128)]),
    (5, [(0, 4), (1, 4)]),
    (1, [(0, 1)]),
])
def test_block_list(D, expect):
    assert oracle.block_list(D) == expect


def test_bit_reversal():
    br = oracle.intra_block_perm(64, P)
    assert br[0] == 0 and br[1] == 32 and br[2] == 16 and br[3] == 48 and br[63] == 63
    assert sorted(br.tolist()) == list(range(64))
    assert np.array_equal(oracle.intra_block_perm(128, P), P)


def test_pass_rule():
    assert oracle.resolve_passes(4, 256) == 1
    assert oracle.resolve_passes(4, 257) == 2
    assert oracle.resolve_passes(3, 128) == 2
    assert oracle.resolve_passes(1, 64) == 2
    assert oracle.resolve_passes(4, 96, 2) == 2


@pytest.mark.parametrize("D", [1, 2, 4, 8, 64, 96, 98, 100, 101, 128, 256, 300])
@pytest.mark.parametrize("passes", [0, 1, 2])
def test_rotation_orthogonal(D, passes):
    R = oracle.rotation_matrix(D, passes, S1, P)
    assert np.abs(R @ R.T - np.eye(D)).max() < 1e-12
    x = np.random.default_rng(D).standard_normal(D)
    assert abs(np.linalg.norm(R @ x) - np.linalg.norm(x)) < 1e-12 * np.linalg.norm(x)


def test_single_pass_closed_form():
    # One block of 128: R = H_128 diag(S1[0:128]) / sqrt(128).
    R = oracle.rotation_matrix(128, 1, S1, P)
    expect = scipy.linalg.hadamard(128) * S1[:128][None, :] / np.sqrt(128)
    assert np.abs(R - expect).max() < 1e-14


def test_two_pass_single_block_closed_form():
    # D = 128 (M = 1): R = H D2 Pi H D1 / 128 with (Pi y)[k] = y[P[k]],
    # D2 = diag(S1[(i + 127) mod 256]).
    H = scipy.linalg.hadamard(128).astype(float)
    Pi = np.zeros((128, 128))
    Pi[np.arange(128), P] = 1.0
    D1 = np.diag(S1[:128].astype(float))
    D2 = np.diag(S1[(np.arange(128) + 127) % 256].astype(float))
    expect = H @ D2 @ Pi @ H @ D1 / 128.0
    R = oracle.rotation_matrix(128, 2, S1, P)
    assert np.abs(R - expect).max() < 1e-14


def test_overlap_block_order_d96():
    # D = 96, one pass: blocks [0,64) then [32,96); the second acts on the
    # first block's output, so R = G2 G1 with G1, G2 embedded H_64 / 8.
    H = scipy.linalg.hadamard(64) / 8.0
    G1 = np.eye(96); G1[:64, :64] = H
    G2 = np.eye(96); G2[32:, 32:] = H
    S = np.diag(S1[:96].astype(float))
    R = oracle.rotation_matrix(96, 1, S1, P)
    assert np.abs(R - G2 @ G1 @ S).max() < 1e-14
    assert np.abs(R - G1 @ G2 @ S).max() > 1e-3   # order matters


def _transpose_only(y, D):
    # the oracle's transpose isolated: run rotate() on a vector with the
    # FWHT replaced by identity is not possible, so rebuild the index map
    # from its definition x'[k M + b] = x[b B + P(k)].
    B = oracle.block_size(D)
    M = D // B
    Pk = oracle.intra_block_perm(B, P)
    out = y.copy()
    for b in range(M):
        for k in range(B):
            out[k * M + b] = y[b * B + Pk[k]]
    return out


@pytest.mark.parametrize("D", [256, 300, 768, 1024, 2049])
def test_transpose_is_bijection_and_tail_fixed(D):
    y = np.arange(D, dtype=float)
    t = _transpose_only(y, D)
    assert sorted(t.tolist()) == list(range(D))
    B = 128
    M = D // B
    assert np.array_equal(t[M * B:], y[M * B:])
    # hand-derived entries: x'[0] = x[P0], x'[1] = x[B + P0] (M >= 2)
    assert t[0] == P[0] and t[1] == B + P[0] and t[M] == P[1]


def test_two_pass_matches_stepwise_composition_d300():
    # R for D = 300 equals F2 D2 T F1 D1 with the transpose as a matrix.
    D = 300
    H = scipy.linalg.hadamard(128) / np.sqrt(128)

    def F():
        G = np.eye(D)
        for off, _ in oracle.block_list(D):
            E = np.eye(D)
            E[off:off + 128, off:off + 128] = H
            G = E @ G
        return G

    T = np.zeros((D, D))
    idx = _transpose_only(np.arange(D, dtype=float), D).astype(int)
    T[np.arange(D), idx] = 1.0
    D1 = np.diag(S1[np.arange(D) % 256].astype(float))
    D2 = np.diag(S1[(np.arange(D) + 127) % 256].astype(float))
    expect = F() @ D2 @ T @ F() @ D1
    R = oracle.rotation_matrix(D, 2, S1, P)
    assert np.abs(R - expect).max() < 1e-13


def test_inverse_is_reverse_order():
    D = 300
    R = oracle.rotation_matrix(D, 2, S1, P)
    x = np.random.default_rng(0).standard_normal(D)
    y = oracle.rotate(x, 2, S1, P)
    assert np.abs(R.T @ y - x).max() < 1e-12
