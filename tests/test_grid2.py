"""The candidate lists of the 2-D nearest-centroid grid (rslm_grid2_lists:
the lists that plans of 2-D codebooks build and that the two-stage encoder
searches instead of all K centroids).  For points everywhere in and beyond
the grid, including points within 1e-6 of every cell edge, the nearest code
(lowest on ties) must be in the point's cell list, and a strict scan of the
list in its ascending order must return it.  Host code only: no GPU needed."""

import ctypes as C

import numpy as np
import pytest

import oracle
import synth
from paper_2608_30384_amd import _lib as L

G = 32


def _lists(cb, emax):
    cbf = np.ascontiguousarray(cb, dtype=np.float32)
    out = np.zeros(G * G, np.uint16)
    so = np.zeros(2, np.float32)
    st = L.lib().rslm_grid2_lists(cbf.ctypes.data, cbf.shape[0], C.c_float(emax),
                                  out.ctypes.data, so.ctypes.data)
    return st, out.reshape(G, G), so


def _scan(tab, s, o, cb, u):
    """Nearest code by a full search, and by the strict scan of the cell list."""
    cb64 = cb.astype(np.float64)
    d = 0.5 * (cb64 ** 2).sum(1)[None, :] - u.astype(np.float64) @ cb64.T
    near = np.argmin(d, 1)                      # first (lowest) code on exact ties
    cell = np.clip(np.floor(u.astype(np.float64) * s + o), 0, G - 1).astype(int)
    lists = tab[cell[:, 0], cell[:, 1]].astype(np.int64)
    codes = (lists[:, None] >> (4 * np.arange(4))) & 15
    pick = codes[np.arange(len(u)), np.argmin(np.take_along_axis(d, codes, 1), 1)]
    return near, pick, codes


@pytest.mark.parametrize("D", [96, 128, 768, 1536, 2049])
def test_grid2_lists_hold_the_nearest_code(D):
    cb = synth.codebook(2)                      # the 2-bit codec's 2-D K = 16 codebook
    emax = np.float32(oracle.e_max(D))
    st, tab, (s, o) = _lists(cb, emax)
    assert st == 0
    assert s == np.float32(G) / (np.float32(2) * emax) and o == G // 2
    rng = np.random.default_rng(D)
    edges = (np.arange(G + 1) - float(o)) / float(s)
    u = np.vstack([rng.uniform(-1.3 * emax, 1.3 * emax, (60000, 2)),
                   rng.normal(size=(60000, 2)),
                   rng.choice(edges, (60000, 2)) + rng.normal(scale=1e-6, size=(60000, 2))])
    u = u.astype(np.float32)
    near, pick, codes = _scan(tab, s, o, cb, u)
    assert np.all(np.diff(codes, axis=1) >= 0) and codes.max() < len(cb)
    assert np.array_equal(pick, near), np.argwhere(pick != near)[:5]
    # most cells need one code, none more than four
    n_codes = np.array([[len(set((int(e) >> (4 * t)) & 15 for t in range(4))) for e in row]
                        for row in tab])
    assert n_codes.max() <= 4 and (n_codes == 1).mean() > 0.6


def test_grid2_lists_catch_a_dropped_code():
    """Removing one listed code from a cell that needs two makes the strict
    scan miss the nearest code for points of that cell (the check above is
    able to fail)."""
    cb = synth.codebook(2)
    emax = np.float32(oracle.e_max(768))
    st, tab, (s, o) = _lists(cb, emax)
    assert st == 0
    rng = np.random.default_rng(0)

    def points(i, j):
        lo = (np.array([i, j]) - float(o)) / float(s)
        return (lo + rng.uniform(0.05, 0.95, (4000, 2)) / float(s)).astype(np.float32)

    # a cell inside the grid whose points have two different nearest codes
    i, j = next((i, j) for i in range(1, G - 1) for j in range(1, G - 1)
                if len(set(_scan(tab, s, o, cb, points(i, j))[0])) >= 2)
    u = points(i, j)
    assert np.array_equal(*_scan(tab, s, o, cb, u)[:2])
    keep = int(tab[i, j]) & 15                  # first listed code only
    bad = tab.copy()
    bad[i, j] = keep | (keep << 4) | (keep << 8) | (keep << 12)
    near, pick, _ = _scan(bad, s, o, cb, u)
    assert not np.array_equal(pick, near)


def test_grid2_lists_arguments():
    cb = synth.codebook(2)
    assert _lists(cb, 3.0)[0] == 0
    assert _lists(cb[:0], 3.0)[0] == 1                     # K = 0
    assert _lists(cb, 0.0)[0] == 1                         # emax <= 0
    assert _lists(cb, float("nan"))[0] == 1
    nan_cb = cb.copy()
    nan_cb[3, 1] = np.nan
    assert _lists(nan_cb, 3.0)[0] == 1
    # sixteen codes crowded into one cell: some cell needs more than four
    ang = np.linspace(0, 2 * np.pi, 16, endpoint=False)
    crowd = (0.01 * np.stack([np.cos(ang), np.sin(ang)], 1)).astype(np.float32)
    assert _lists(crowd, 3.0)[0] == 2
