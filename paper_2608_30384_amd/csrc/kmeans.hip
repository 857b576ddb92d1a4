// IVF partition training: one Lloyd update of the partition centres.
//
// Paper, Section "End-to-End Comparison with Faiss and ScaNN", Setup: the
// collection is partitioned by Euclidean k-means (about 256 sample points
// per centre).  One iteration assigns every point to its nearest centre
// (ivf_assign_probe, IVF_ASSIGN_L2) and then moves each centre to the mean of
// its points; a centre with no points keeps its position.  This file is the
// second half of the iteration.
//
// GPU design.  The point indices are counting-sorted by centre (counts by
// integer atomics, one exclusive scan, placement through a per-centre
// cursor), so each centre's points are one contiguous run of indices.  Then
// one workgroup per (centre, 256 coordinates) walks its run: each thread owns
// one coordinate and adds the points' values in float64 (a point's row is
// read as one coalesced 1 KiB segment per workgroup), and divides once by
// the count.  With float64 sums, the order in which atomics placed a
// centre's points only moves the sum by float64 roundings; the result is
// rounded to float32 once.
#include "rslm_internal.h"

namespace rslm {

constexpr int kKmThreads = 256;
constexpr int kKmScanThreads = 1024;

struct KmWs {
  int32_t *counts, *cursor, *offsets, *order;
  size_t bytes;
};

static size_t km_align(size_t b) { return (b + 255) / 256 * 256; }

static KmWs km_ws_layout(void *base, int64_t n, int nlist) {
  KmWs w{};
  char *p = static_cast<char *>(base);
  size_t off = 0;
  auto take = [&](size_t b) {
    char *r = p ? p + off : nullptr;
    off += km_align(b);
    return reinterpret_cast<int32_t *>(r);
  };
  w.counts = take(size_t(nlist) * 4);
  w.cursor = take(size_t(nlist) * 4);
  w.offsets = take(size_t(nlist + 1) * 4);
  w.order = take(size_t(n > 0 ? n : 1) * 4);
  w.bytes = off;
  return w;
}

__global__ void __launch_bounds__(kKmThreads) k_km_zero(int32_t *__restrict__ counts,
                                                        int32_t *__restrict__ cursor, int nlist) {
  const int i = blockIdx.x * kKmThreads + threadIdx.x;
  if (i < nlist) {
    counts[i] = 0;
    cursor[i] = 0;
  }
}

// Points per centre; assignments outside [0, nlist) are ignored.
__global__ void __launch_bounds__(kKmThreads) k_km_count(const int32_t *__restrict__ assign,
                                                         int64_t n, int nlist,
                                                         int32_t *__restrict__ counts) {
  const int64_t stride = int64_t(gridDim.x) * kKmThreads;
  for (int64_t i = int64_t(blockIdx.x) * kKmThreads + threadIdx.x; i < n; i += stride) {
    const int a = assign[i];
    if (a >= 0 && a < nlist) atomicAdd(&counts[a], 1);
  }
}

// Exclusive prefix of the counts (one workgroup): thread t sums a run of
// consecutive centres, the runs' totals are scanned by wavefront shuffles and
// then across the wavefronts, and each thread writes its run's offsets.
__global__ void __launch_bounds__(kKmScanThreads) k_km_scan(const int32_t *__restrict__ counts,
                                                            int nlist,
                                                            int32_t *__restrict__ offsets) {
  __shared__ int32_t part[kKmScanThreads / 64];
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int per = (nlist + kKmScanThreads - 1) / kKmScanThreads;
  const int a = min(nlist, t * per), b = min(nlist, a + per);
  int sum = 0;
  for (int i = a; i < b; ++i) sum += counts[i];
  int incl = sum;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int v = __shfl_up(incl, off, 64);
    if (lane >= off) incl += v;
  }
  if (lane == 63) part[wv] = incl;
  __syncthreads();
  int before = 0, total = 0;
  for (int w = 0; w < kKmScanThreads / 64; ++w) {
    before += w < wv ? part[w] : 0;
    total += part[w];
  }
  int run = before + incl - sum;
  for (int i = a; i < b; ++i) {
    offsets[i] = run;
    run += counts[i];
  }
  if (t == 0) offsets[nlist] = total;
}

// Point i takes the next slot of its centre's run.
__global__ void __launch_bounds__(kKmThreads) k_km_place(const int32_t *__restrict__ assign,
                                                         int64_t n, int nlist,
                                                         const int32_t *__restrict__ offsets,
                                                         int32_t *__restrict__ cursor,
                                                         int32_t *__restrict__ order) {
  const int64_t stride = int64_t(gridDim.x) * kKmThreads;
  for (int64_t i = int64_t(blockIdx.x) * kKmThreads + threadIdx.x; i < n; i += stride) {
    const int a = assign[i];
    if (a >= 0 && a < nlist) order[offsets[a] + atomicAdd(&cursor[a], 1)] = int32_t(i);
  }
}

// Workgroup (centre L, coordinate block y): thread d' sums coordinate
// d = 256 y + d' over the centre's points in float64 (four rows in flight),
// then writes the mean; an empty centre is left as it is.
__global__ void __launch_bounds__(kKmThreads) k_km_mean(const float *__restrict__ x, int dim,
                                                        const int32_t *__restrict__ offsets,
                                                        const int32_t *__restrict__ counts,
                                                        const int32_t *__restrict__ order,
                                                        float *__restrict__ centroids) {
  const int L = blockIdx.x;
  const int d = blockIdx.y * kKmThreads + threadIdx.x;
  const int cnt = counts[L];
  if (cnt <= 0 || d >= dim) return;
  const int32_t *run = order + offsets[L];
  double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
  int j = 0;
  for (; j + 4 <= cnt; j += 4) {
    const float v0 = x[int64_t(run[j]) * dim + d];
    const float v1 = x[int64_t(run[j + 1]) * dim + d];
    const float v2 = x[int64_t(run[j + 2]) * dim + d];
    const float v3 = x[int64_t(run[j + 3]) * dim + d];
    s0 += double(v0);
    s1 += double(v1);
    s2 += double(v2);
    s3 += double(v3);
  }
  for (; j < cnt; ++j) s0 += double(x[int64_t(run[j]) * dim + d]);
  centroids[int64_t(L) * dim + d] = float(((s0 + s1) + (s2 + s3)) / double(cnt));
}

}  // namespace rslm

using namespace rslm;

extern "C" {

size_t ivf_kmeans_update_workspace(int64_t n, int32_t nlist) {
  if (n < 0 || nlist < 1) return 0;
  return km_ws_layout(nullptr, n, nlist).bytes;
}

int ivf_kmeans_update(const float *x, int64_t n, int32_t dim, const int32_t *assign,
                      int32_t nlist, float *centroids, void *ws, size_t ws_bytes,
                      void *stream) {
  if (n < 0 || n > 0x7fffffff || dim < 1 || dim > (1 << 20) || nlist < 1 || nlist > 65536)
    return RSLM_ERR_INVALID_ARG;
  if (!centroids) return RSLM_ERR_INVALID_ARG;
  if (n == 0) return RSLM_OK;
  if (!x || !assign) return RSLM_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(x) & 3) || (reinterpret_cast<uintptr_t>(assign) & 3) ||
      (reinterpret_cast<uintptr_t>(centroids) & 3))
    return RSLM_ERR_INVALID_ARG;
  if (!ws || ws_bytes < ivf_kmeans_update_workspace(n, nlist)) return RSLM_ERR_WORKSPACE;
  const KmWs w = km_ws_layout(ws, n, nlist);
  hipStream_t s = as_stream(stream);
  int st;
  hipLaunchKernelGGL(k_km_zero, dim3(unsigned((nlist + kKmThreads - 1) / kKmThreads)),
                     dim3(kKmThreads), 0, s, w.counts, w.cursor, nlist);
  if ((st = check_launch())) return st;
  const unsigned grid = unsigned(std::min<int64_t>((n + kKmThreads - 1) / kKmThreads, 4096));
  hipLaunchKernelGGL(k_km_count, dim3(grid), dim3(kKmThreads), 0, s, assign, n, nlist, w.counts);
  if ((st = check_launch())) return st;
  hipLaunchKernelGGL(k_km_scan, dim3(1), dim3(kKmScanThreads), 0, s, w.counts, nlist, w.offsets);
  if ((st = check_launch())) return st;
  hipLaunchKernelGGL(k_km_place, dim3(grid), dim3(kKmThreads), 0, s, assign, n, nlist, w.offsets,
                     w.cursor, w.order);
  if ((st = check_launch())) return st;
  hipLaunchKernelGGL(k_km_mean, dim3(unsigned(nlist), unsigned((dim + kKmThreads - 1) / kKmThreads)),
                     dim3(kKmThreads), 0, s, x, dim, w.offsets, w.counts, w.order, centroids);
  return check_launch();
}

}  // extern "C"
