"""Write ``synth/codebooks.json``: the fixed Lloyd-Max codebooks for N(0, I_g).

Run once (``python -m synth.make_codebooks``); the result is committed data.

* 1-D tables (K = 2, 4, 8, 16): Lloyd's fixed-point iteration on the exact
  normal density -- thresholds are midpoints of neighbouring levels and each
  level is the conditional mean of its cell, computed in closed form with the
  normal pdf/cdf -- run to convergence in float64.
* 2-D and 4-D tables (K = 16): k-means (Lloyd's algorithm) on seeded samples
  of N(0, I_g), seed 3, best of three initialisations, as the paper describes
  (k-means on a large synthetic normal sample).

Every centroid is then rounded to the nearest float16 value and stored as a
decimal that float32 reproduces exactly.  1-D tables are ascending; g > 1
tables are ordered by (radius, angle of the first two coordinates).
"""

import json
import os

import numpy as np
from scipy.stats import norm

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "codebooks.json")


def lloyd_max_1d(K, iters=20000, tol=1e-15):
    c = norm.ppf((np.arange(K) + 0.5) / K)
    for _ in range(iters):
        t = 0.5 * (c[1:] + c[:-1])
        lo = np.concatenate([[-np.inf], t])
        hi = np.concatenate([t, [np.inf]])
        mass = norm.cdf(hi) - norm.cdf(lo)
        new = (norm.pdf(lo) - norm.pdf(hi)) / mass
        if np.max(np.abs(new - c)) < tol:
            c = new
            break
        c = new
    return c


def kmeans_gauss(g, K, n, seed, iters, inits=3):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, g))
    xx = (x * x).sum(1)
    best = None
    for trial in range(inits):
        c = x[rng.choice(n, K, replace=False)].copy()
        for _ in range(iters):
            d = xx[:, None] - 2.0 * x @ c.T + (c * c).sum(1)[None, :]
            a = d.argmin(1)
            for k in range(K):
                sel = a == k
                if sel.any():
                    c[k] = x[sel].mean(0)
        d = xx[:, None] - 2.0 * x @ c.T + (c * c).sum(1)[None, :]
        mse = d.min(1).mean() / g
        if best is None or mse < best[0]:
            best = (mse, c.copy())
    return best[1]


def to_f16_exact(a):
    return np.asarray(a, dtype=np.float64).astype(np.float16).astype(np.float64)


def order_multi(c):
    r = np.sqrt((c * c).sum(1))
    ang = np.arctan2(c[:, 1], c[:, 0])
    idx = np.lexsort((ang, np.round(r, 6)))
    return c[idx]


def main():
    out = {}
    for K, key in [(2, "lm1d_k2"), (4, "lm1d_k4"), (8, "rslm3"), (16, "rslm4")]:
        c = to_f16_exact(lloyd_max_1d(K))
        c = np.sort(c)
        out[key] = {"K": K, "g": 1, "centroids": [float(v) for v in c]}
    for g, key in [(2, "rslm2"), (4, "rslm1")]:
        c = kmeans_gauss(g, 16, 1 << 21, seed=3, iters=150)
        c = order_multi(to_f16_exact(c))
        out[key] = {"K": 16, "g": g, "centroids": [float(v) for v in c.reshape(-1)]}
    with open(OUT, "w") as f:
        json.dump(out, f, indent=1)
    print("wrote", OUT)


if __name__ == "__main__":
    main()
