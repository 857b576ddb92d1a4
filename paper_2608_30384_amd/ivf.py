"""IVF index construction around the librslm kernels.

Partition training runs in librslm (assignment by ``ivf_assign_probe``,
the centre update by ``ivf_kmeans_update``); the record layout of the
inverted lists is build-time bookkeeping done with torch tensor operations
(counting and sorting); every step of the codec itself (rotation, encoding,
SQ8) runs in librslm.  The paper's partitioning (Section "End-to-End
Comparison", Setup) is Euclidean k-means with random initialisation on a
sample of about 256 points per centre.
"""

import torch

from . import _lib as L
from .api import (Index, ivf_assign_probe, ivf_kmeans_update, rslm_encode,
                  rslm_encode_two_stage, rslm_fwht, rslm_sq8_encode, rslm_sq8_fit)


def kmeans(x, nlist, iters=10, seed=0, sample=None, init=None):
    """Euclidean k-means (Lloyd) on device: each iteration assigns every point
    to its nearest centre (``ivf_assign_probe``) and moves each centre to the
    mean of its points (``ivf_kmeans_update``; an empty centre stays).  The
    initial centres are ``init`` (nlist x dim) or nlist distinct points drawn
    with torch's generator seeded by ``seed``."""
    n = x.shape[0]
    gen = torch.Generator(device=x.device)
    gen.manual_seed(int(seed))
    if sample is not None and sample < n:
        xs = x[torch.randperm(n, generator=gen, device=x.device)[:sample]].contiguous()
    else:
        xs = x
    if init is None:
        c = xs[torch.randperm(xs.shape[0], generator=gen, device=x.device)[:nlist]].clone()
    else:
        c = init.to(device=x.device, dtype=torch.float32).clone().contiguous()
    a = torch.empty(xs.shape[0], dtype=torch.int32, device=x.device)
    for _ in range(iters):
        ivf_assign_probe(xs, c, 1, L.IVF_ASSIGN_L2, out_ids=a)
        ivf_kmeans_update(xs, a, c)
    return c.contiguous()


def layout(assign, nlist, tile=16):
    """Inverted-list record layout: lists padded to whole tiles of 16.

    Returns (list_offsets int64, list_sizes int32, src_row int64 per record
    (-1 = padding), rec_list int32 per record, ids int32 per record, total).
    Within a list, vectors keep their original order.
    """
    a = assign.long()
    n = a.numel()
    dev = a.device
    counts = torch.bincount(a, minlength=nlist)
    padded = (counts + tile - 1) // tile * tile
    offsets = torch.cumsum(padded, 0) - padded
    total = int(padded.sum().item())
    order = torch.argsort(a, stable=True)
    sl = a[order]
    starts = torch.cumsum(counts, 0) - counts
    rank = torch.arange(n, device=dev) - starts[sl]
    rec = offsets[sl] + rank
    src_row = torch.full((total,), -1, dtype=torch.int64, device=dev)
    src_row[rec] = order
    rec_list = torch.repeat_interleave(torch.arange(nlist, device=dev, dtype=torch.int32), padded)
    ids = torch.full((total,), -1, dtype=torch.int32, device=dev)
    ids[rec] = order.to(torch.int32)
    return offsets, counts.to(torch.int32), src_row, rec_list.contiguous(), ids, total


def build_index(plan, x, centroids, assign=None, resid_rot=None):
    """Assign, lay out and encode a collection; returns (Index, R c, assign)."""
    nlist = centroids.shape[0]
    if assign is None:
        assign, _ = ivf_assign_probe(x, centroids, 1, L.IVF_ASSIGN_L2)
    cen_rot = rslm_fwht(plan, centroids)
    offsets, sizes, src_row, rec_list, ids, total = layout(assign, nlist)
    codes = torch.zeros(plan.code_bytes(total), dtype=torch.uint8, device=x.device)
    scales = torch.zeros(total, dtype=torch.int32, device=x.device)
    rslm_encode(plan, x, codes, scales, n_records=total, src_row=src_row, rec_list=rec_list,
                centroids=centroids, centroids_rot=cen_rot, resid_rot=resid_rot)
    return Index(offsets, sizes, ids, codes, scales), cen_rot, assign


def build_sq8(resid_rot):
    """SQ8 rescoring codes of the rotated second residuals (row = vector id)."""
    lo, hi = rslm_sq8_fit(resid_rot)
    codes2 = rslm_sq8_encode(resid_rot, lo, hi)
    return codes2, lo, hi


def build_two_stage_blocked(plan, plan2, block, n, block_rows, centroids, on_assigned=None,
                            on_block=None):
    """Index a collection too large to hold as float32: ``block(b)`` returns
    rows [b * block_rows, ...) on the device (regenerated on demand).  Rows
    are assigned block by block, laid out, then encoded block by block into
    scan records (``plan``) and RSLM rescoring records (``plan2``, indexed by
    row) with ``rslm_encode_two_stage``: records of other blocks fall outside
    a block's row range and are skipped.  ``on_assigned()`` runs after the
    assignment pass and ``on_block(b, rows)`` after each block's encode.
    Returns (Index, codes2, scales2, R c)."""
    dev = centroids.device
    nlist = centroids.shape[0]
    nblk = (n + block_rows - 1) // block_rows
    assign = torch.empty(n, dtype=torch.int32, device=dev)
    for b in range(nblk):
        xs = block(b)
        ivf_assign_probe(xs, centroids, 1, L.IVF_ASSIGN_L2,
                         out_ids=assign[b * block_rows:b * block_rows + len(xs)])
    if on_assigned is not None:
        on_assigned()
    crot = rslm_fwht(plan, centroids)
    offsets, sizes, src_row, rec_list, ids, total = layout(assign, nlist)
    del assign
    codes = torch.zeros(plan.code_bytes(total), dtype=torch.uint8, device=dev)
    scales = torch.zeros(total, dtype=torch.int32, device=dev)
    codes2 = torch.zeros((n, plan2.canon_bytes), dtype=torch.uint8, device=dev)
    scales2 = torch.zeros(n, dtype=torch.int32, device=dev)
    for b in range(nblk):
        xs = block(b)
        lo = b * block_rows
        src_local = src_row - lo
        rslm_encode_two_stage(plan, plan2, xs, codes, scales, codes2[lo:lo + len(xs)],
                              scales2[lo:lo + len(xs)], n_records=total, src_row=src_local,
                              rec_list=rec_list, centroids=centroids, centroids_rot=crot)
        del src_local
        if on_block is not None:
            on_block(b, xs)
    return Index(offsets, sizes, ids, codes, scales), codes2, scales2, crot
