"""Seeded synthetic embedding collections.

Two families stand in for the paper's embedding datasets (which are not
available here):

* ``gmix`` -- an isotropic Gaussian mixture: component means ~ N(0, I_D),
  a uniformly chosen component per row, within-component noise sigma*N(0, I_D),
  optionally L2-normalised (the unit-norm, low-dimensional sets).
* ``aniso`` -- an anisotropic Gaussian with a power-law per-dimension variance
  spectrum sigma_d^2 proportional to (d+1)^-alpha (normalised so that
  E||x - mu||^2 = 1) plus a shared mean offset mu of norm 0.5, optionally
  L2-normalised (text-embedding-shaped sets, MIPS with varying norms).

Rows are generated in chunks of 2**20 with ``numpy.random.default_rng([seed,
chunk])`` so any row range regenerates independently of the others; the
component means / offset come from ``default_rng([mean_seed, 2**32 - 1])`` and
are shared by a collection and its queries.  ``aniso_torch`` produces the same
*distribution* on a GPU with torch's generator for collections too large to
create on the host (its rows differ from ``aniso``'s).
"""

import numpy as np

CHUNK = 1 << 20
_MEAN_STREAM = 2**32 - 1


def gmix_means(d, n_comp, mean_seed):
    return np.random.default_rng([mean_seed, _MEAN_STREAM]).standard_normal((n_comp, d))


def _chunks(start, n):
    end = start + n
    c0, c1 = start // CHUNK, (end + CHUNK - 1) // CHUNK
    for c in range(c0, c1):
        lo, hi = max(start, c * CHUNK), min(end, (c + 1) * CHUNK)
        yield c, lo - c * CHUNK, hi - c * CHUNK


def gmix(n, d, n_comp, sigma=0.3, seed=100, mean_seed=None, normalize=True, start=0):
    """Rows [start, start+n) of a Gaussian-mixture collection, float32 (n, d)."""
    mean_seed = seed if mean_seed is None else mean_seed
    mu = gmix_means(d, n_comp, mean_seed)
    out = np.empty((n, d), dtype=np.float32)
    pos = 0
    for c, a, b in _chunks(start, n):
        rows = min(CHUNK, b)
        rng = np.random.default_rng([seed, c])
        comp = rng.integers(0, n_comp, rows)
        x = mu[comp] + sigma * rng.standard_normal((rows, d))
        x = x[a:b]
        if normalize:
            x = x / np.linalg.norm(x, axis=1, keepdims=True)
        out[pos:pos + (b - a)] = x
        pos += b - a
    return out


def aniso_params(d, alpha=1.0, mean_seed=100):
    """Per-dimension standard deviations and the shared mean offset."""
    var = (np.arange(d) + 1.0) ** (-alpha)
    var /= var.sum()
    v = np.random.default_rng([mean_seed, _MEAN_STREAM]).standard_normal(d)
    mu = 0.5 * v / np.linalg.norm(v)
    return np.sqrt(var), mu


def aniso(n, d, alpha=1.0, seed=100, mean_seed=None, normalize=False, start=0):
    """Rows [start, start+n) of the anisotropic collection, float32 (n, d)."""
    mean_seed = seed if mean_seed is None else mean_seed
    sd, mu = aniso_params(d, alpha, mean_seed)
    out = np.empty((n, d), dtype=np.float32)
    pos = 0
    for c, a, b in _chunks(start, n):
        rows = min(CHUNK, b)
        rng = np.random.default_rng([seed, c])
        x = mu + sd * rng.standard_normal((rows, d))
        x = x[a:b]
        if normalize:
            x = x / np.linalg.norm(x, axis=1, keepdims=True)
        out[pos:pos + (b - a)] = x
        pos += b - a
    return out


def aniso_torch(n, d, alpha=1.0, seed=100, mean_seed=None, normalize=False,
                device="cuda", out=None, chunk=1 << 22):
    """Same distribution as ``aniso`` generated on ``device`` with torch.

    Writes into ``out`` (float32, (n, d)) when given.  Deterministic for a
    given seed, device and chunk size.
    """
    import torch

    mean_seed = seed if mean_seed is None else mean_seed
    sd, mu = aniso_params(d, alpha, mean_seed)
    sd_t = torch.tensor(sd, dtype=torch.float32, device=device)
    mu_t = torch.tensor(mu, dtype=torch.float32, device=device)
    if out is None:
        out = torch.empty((n, d), dtype=torch.float32, device=device)
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        blk = out[lo:hi]
        blk.normal_(generator=gen)
        blk.mul_(sd_t).add_(mu_t)
        if normalize:
            blk.div_(blk.norm(dim=1, keepdim=True))
    return out


TORCH_BLOCK = 1 << 22


def aniso_torch_block(b, d, alpha=1.0, seed=100, mean_seed=None, normalize=False,
                      device="cuda", out=None, block=TORCH_BLOCK):
    """Rows [b * block, (b + 1) * block) of a collection too large to hold
    at once (same distribution as ``aniso``), generated on ``device`` with a
    torch generator seeded by (seed, b), so any block regenerates on its own.
    """
    import torch

    mean_seed = seed if mean_seed is None else mean_seed
    sd, mu = aniso_params(d, alpha, mean_seed)
    sd_t = torch.tensor(sd, dtype=torch.float32, device=device)
    mu_t = torch.tensor(mu, dtype=torch.float32, device=device)
    if out is None:
        out = torch.empty((block, d), dtype=torch.float32, device=device)
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed) * 1_000_003 + int(b))
    out.normal_(generator=gen)
    out.mul_(sd_t).add_(mu_t)
    if normalize:
        out.div_(out.norm(dim=1, keepdim=True))
    return out


def queries_like(kind, n, d, data_seed=100, query_seed=200, **kw):
    """Queries drawn from the same distribution as a collection (same means)."""
    if kind == "gmix":
        return gmix(n, d, seed=query_seed, mean_seed=data_seed, **kw)
    if kind == "aniso":
        return aniso(n, d, seed=query_seed, mean_seed=data_seed, **kw)
    raise ValueError(kind)


def random_rows(n_total, k, seed=0):
    """k distinct row indices of [0, n_total), sorted, seeded."""
    idx = np.random.default_rng(seed).choice(n_total, size=k, replace=False)
    return np.sort(idx).astype(np.int64)
