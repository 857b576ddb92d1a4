"""The allocation-free probe entry point (ivf_assign_probe_noalloc), called
through the C ABI: its outputs must equal ivf_assign_probe's (the same
kernels; here bit for bit) on two calls in a row, the second smaller (the
fixed scratch keeps the first call's contents), in both modes; a size beyond
the fixed scratch is rejected before any launch with outputs untouched."""

import ctypes as C

import numpy as np
import pytest

import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"


def _call(lib, x, cen, nprobe, mode, ids, sc, stream):
    return lib.ivf_assign_probe_noalloc(C.c_void_p(x.data_ptr()), x.shape[0], x.shape[1],
                                        C.c_void_p(cen.data_ptr()), cen.shape[0], nprobe, mode,
                                        C.c_void_p(ids.data_ptr()), C.c_void_p(sc.data_ptr()),
                                        stream)


def _reference(R, x, cen, nprobe, mode):
    return R.ivf_assign_probe(x, cen, nprobe, mode)


@pytest.mark.parametrize("mode_name", ["probe", "assign"])
def test_noalloc_matches_the_workspace_entry_point(mode_name):
    import paper_2608_30384_amd as R
    from paper_2608_30384_amd import _lib as L
    lib = L.lib()
    limit = lib.ivf_assign_probe_noalloc_limit()
    assert limit == (64 << 20) + (256 << 10)
    mode = R.IVF_PROBE_IP if mode_name == "probe" else R.IVF_ASSIGN_L2
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    # first call: the capacity batch's probe (1,024 x 16,384 dots: the
    # whole fixed scratch); second call: a smaller, ragged one
    shapes = [(1024, 768, 16384, 128), (37, 96, 3001, 50)] if mode_name == "probe" else \
             [(50000, 768, 4096, 1), (333, 100, 700, 1)]
    for n, dim, nlist, nprobe in shapes:
        rng = np.random.default_rng(n + dim)
        x = torch.from_numpy(synth.aniso(n, dim, seed=n)).to(DEV)
        cen = torch.from_numpy(rng.standard_normal((nlist, dim)).astype(np.float32)).to(DEV)
        shape = (n, nprobe) if mode == R.IVF_PROBE_IP else (n,)
        ids = torch.full(shape, -7, dtype=torch.int32, device=DEV)
        sc = torch.full(shape, 7.0, dtype=torch.float32, device=DEV)
        assert _call(lib, x, cen, nprobe, mode, ids, sc, stream) == 0
        ref_ids, ref_sc = _reference(R, x, cen, nprobe, mode)
        torch.cuda.synchronize()
        assert torch.equal(ids, ref_ids)
        assert torch.equal(sc, ref_sc)


def test_noalloc_rejects_sizes_beyond_its_scratch():
    import paper_2608_30384_amd as R
    from paper_2608_30384_amd import _lib as L
    lib = L.lib()
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    n, dim, nlist, nprobe = 1028, 64, 16384, 8          # 1,028 x 16,384 dots: too many
    limit = lib.ivf_assign_probe_noalloc_limit()
    assert lib.ivf_assign_probe_workspace(n, dim, nlist, nprobe, R.IVF_PROBE_IP) > limit
    assert lib.ivf_assign_probe_workspace(n - 1, dim, nlist, nprobe, R.IVF_PROBE_IP) <= limit
    x = torch.zeros((n, dim), dtype=torch.float32, device=DEV)
    cen = torch.zeros((nlist, dim), dtype=torch.float32, device=DEV)
    ids = torch.full((n, nprobe), -7, dtype=torch.int32, device=DEV)
    sc = torch.full((n, nprobe), 7.0, dtype=torch.float32, device=DEV)
    assert _call(lib, x, cen, nprobe, R.IVF_PROBE_IP, ids, sc, stream) == 4
    torch.cuda.synchronize()
    assert bool((ids == -7).all()) and bool((sc == 7.0).all())
