"""Parity of the IVF partition training on the GPU (Section "End-to-End
Comparison with Faiss and ScaNN", Setup: Euclidean k-means partitions) with
the float64 oracle.

* ``ivf_kmeans_update`` (one Lloyd centre update) against the oracle's
  update on the same points and the same assignment: the mean of each
  centre's points, a centre with no points unchanged.  Shapes cover empty
  centres, centres with thousands of points, dimensions that are not a
  multiple of the 256-coordinate workgroup and assignments outside the
  centre range (ignored).
* ``ivf.kmeans`` (assignment on ``ivf_assign_probe`` + this update) against
  ``oracle.kmeans`` from the same initial centres for the same number of
  iterations, on data whose every assignment along the oracle's trajectory
  has a clear margin (checked on the oracle side first), so the float32
  assignment must make the same choices and the centres agree to float32
  rounding.
"""

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def R():
    import paper_2608_30384_amd as R
    return R


def _t(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(DEV)


@pytest.mark.parametrize("n,dim,nlist", [(5000, 33, 40), (20000, 768, 16), (3001, 300, 500),
                                         (257, 4, 1), (4096, 1000, 64)])
def test_kmeans_update_parity(R, n, dim, nlist):
    rng = np.random.default_rng(n + dim)
    x = (rng.standard_normal((n, dim)) * rng.uniform(0.1, 3.0, dim) + 0.5).astype(np.float32)
    c0 = (rng.standard_normal((nlist, dim)) * 2.0).astype(np.float32)
    if nlist > 4:
        c0[-3:] = 1e3                                  # three centres no point is near
    a, _ = oracle.assign_l2(x, c0)
    ref = oracle.kmeans(x, nlist, iters=1, init=c0)   # assign, then the mean update
    assert (np.bincount(a, minlength=nlist) == 0).sum() >= (3 if nlist > 4 else 0)
    a32 = a.astype(np.int32)
    if n > 1000:
        a32[7] = nlist                                 # out of range: ignored by the update
        a32[8] = -1
        keep = np.ones(n, dtype=bool)
        keep[[7, 8]] = False
        ref = c0.astype(np.float64).copy()
        for p in range(nlist):
            sel = (a == p) & keep
            if sel.any():
                ref[p] = x[sel].astype(np.float64).mean(0)
    c = _t(c0)
    R.ivf_kmeans_update(_t(x), _t(a32), c)
    got = c.cpu().numpy().astype(np.float64)
    tol = 2.0 ** -24 * np.abs(ref) + 2.0 ** -50 * np.abs(x).max()
    assert np.all(np.abs(got - ref) <= tol), np.abs(got - ref).max()
    empty = np.bincount(a32[(a32 >= 0) & (a32 < nlist)], minlength=nlist) == 0
    assert np.array_equal(got[empty], c0[empty].astype(np.float64))


def _dists(x, c):
    x = x.astype(np.float64)
    return ((x[:, None, :] - c[None, :, :]) ** 2).sum(-1)


@pytest.mark.parametrize("dim,n_comp,extra", [(32, 16, False), (96, 24, True)])
def test_kmeans_matches_oracle(R, dim, n_comp, extra):
    from paper_2608_30384_amd import ivf
    seed = 40 + dim
    n, iters = 20000, 10
    x = synth.gmix(n, dim, n_comp, seed=seed, normalize=False)
    means = synth.gmix_means(dim, n_comp, seed)
    # initial centres: one data point per mixture component (the first row
    # nearest each component mean), plus a far centre that stays empty
    near, _ = oracle.assign_l2(x, means)
    init = np.stack([x[np.flatnonzero(near == p)[0]] for p in range(n_comp)]).astype(np.float64)
    if extra:
        init = np.vstack([init, np.full((1, dim), 50.0)])
    nlist = len(init)
    # every assignment along the oracle's trajectory has a clear margin
    for it in range(iters):
        c = oracle.kmeans(x, nlist, iters=it, init=init)
        d = np.sort(_dists(x, c), axis=1)
        scale = (x.astype(np.float64) ** 2).sum(1) + (c ** 2).sum(1).max()
        assert ((d[:, 1] - d[:, 0]) / scale).min() > 1e-4, it
    ref = oracle.kmeans(x, nlist, iters=iters, init=init)
    got = ivf.kmeans(_t(x), nlist, iters=iters, init=_t(init.astype(np.float32)))
    got = got.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(got - ref) <= 1e-6 * (np.abs(ref) + 1.0)), np.abs(got - ref).max()
    if extra:
        assert np.array_equal(got[-1], init[-1])
