// IVF routing: assignment of vectors to their nearest partition centre and
// probing of the partitions with the largest dot product with a query
// (paper, Section "End-to-End Comparison", Setup: Euclidean partitions,
// routing by the dot product with the centres).
//
// Both modes are a dense [n x D] x [D x nlist] contraction in float32 on the
// matrix cores (v_mfma_f32_16x16x4_f32).  Probing writes the dots (64 x 64
// output tiles) and selects the top-nprobe per row.  Assignment keeps a
// running (distance, id) minimum per row across all centre tiles (128 x 128
// output tiles), never writing the product; rows that are not whole 16-byte
// runs take a vector-ALU tile (64 x 64, 4 x 4 outputs per thread) instead.
#include <mutex>

#include "rslm_internal.h"
#include "select_dev.h"

namespace rslm {

constexpr int kTM = 64, kTN = 64, kTK = 16;

__global__ void k_row_norms(const float *__restrict__ c, int n, int D, float *__restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (row >= n) return;
  float s = 0.f;
  for (int i = lane; i < D; i += 64) {
    const float v = c[int64_t(row) * D + i];
    s += v * v;
  }
  s = wave_sum(s);
  if (lane == 0) out[row] = s;
}

// Loads a 64-row x 16-column slice of a row-major matrix (rows r0.., cols
// k0..) transposed into lds[16][64 + 4] (zero outside the matrix).
__device__ __forceinline__ void load_slice(const float *__restrict__ m, int64_t rows, int D,
                                           int64_t r0, int k0, float (*lds)[kTM + 4]) {
  // 256 threads x 4 elements
  const int t = threadIdx.x;
  const int r = t >> 2;          // 0..63
  const int kk = (t & 3) * 4;    // 0,4,8,12
  const int64_t gr = r0 + r;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int gk = k0 + kk + e;
    float v = 0.f;
    if (gr < rows && gk < D) v = m[gr * D + gk];
    lds[kk + e][r] = v;
  }
}

// acc[i][j] = sum_k A[r0 + ty*4 + i][k] * B[c0 + tx*4 + j][k]
__device__ __forceinline__ void tile_product(const float *__restrict__ A, int64_t n,
                                             const float *__restrict__ Bm, int nb, int D,
                                             int64_t r0, int c0, float (*As)[kTM + 4],
                                             float (*Bs)[kTM + 4], float acc[4][4]) {
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
  for (int k0 = 0; k0 < D; k0 += kTK) {
    load_slice(A, n, D, r0, k0, As);
    load_slice(Bm, nb, D, c0, k0, Bs);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kTK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += a[i] * b[j];
    }
    __syncthreads();
  }
}

__global__ void __launch_bounds__(256) k_assign(const float *__restrict__ x, int64_t n, int D,
                                                const float *__restrict__ cen, int nlist,
                                                const float *__restrict__ cnorm,
                                                int32_t *__restrict__ out_ids,
                                                float *__restrict__ out_d) {
  __shared__ float As[kTK][kTM + 4];
  __shared__ float Bs[kTK][kTM + 4];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int64_t r0 = int64_t(blockIdx.x) * kTM;
  float best[4];
  int bid[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    best[i] = 3.4e38f;
    bid[i] = 0x7fffffff;
  }
  float acc[4][4];
  for (int c0 = 0; c0 < nlist; c0 += kTN) {
    tile_product(x, n, cen, nlist, D, r0, c0, As, Bs, acc);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = c0 + tx * 4 + j;
      if (c < nlist) {
        const float cn = cnorm[c];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float v = cn - 2.f * acc[i][j];   // ||c||^2 - 2 <x, c>
          if (v < best[i]) {                      // columns visited in increasing order
            best[i] = v;
            bid[i] = c;
          }
        }
      }
    }
  }
  // reduce over the 16 threads (tx) sharing each row: lexicographic (value, id)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    for (int off = 8; off >= 1; off >>= 1) {
      const float ov = __shfl_xor(best[i], off, 64);
      const int oi = __shfl_xor(bid[i], off, 64);
      if (ov < best[i] || (ov == best[i] && oi < bid[i])) {
        best[i] = ov;
        bid[i] = oi;
      }
    }
  }
  if (tx == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t r = r0 + ty * 4 + i;
      if (r < n) {
        out_ids[r] = bid[i];
        if (out_d) {
          float xx = 0.f;
          for (int k = 0; k < D; ++k) {
            const float v = x[r * D + k];
            xx += v * v;
          }
          out_d[r] = xx + best[i];
        }
      }
    }
  }
}

// Probe dots on the matrix cores (v_mfma_f32_16x16x4_f32, full float32):
// a 32 x 32 output tile per 256-thread workgroup, each wavefront one 16 x 16
// MFMA tile, K staged through LDS in slabs of 32.
typedef float floatx4_t __attribute__((ext_vector_type(4)));
constexpr int kMT = 32, kMK = 32;

__device__ __forceinline__ void stage32(const float *__restrict__ m, int64_t rows, int D,
                                        int64_t r0, int k0, float (*lds)[kMK + 1]) {
  const int t = threadIdx.x;        // 256 threads x 4 elements = 32 rows x 32 k
  const int r = t >> 3;
  const int kk = (t & 7) * 4;
  const int64_t gr = r0 + r;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int gk = k0 + kk + e;
    lds[r][kk + e] = (gr < rows && gk < D) ? m[gr * D + gk] : 0.f;
  }
}

__global__ void __launch_bounds__(256) k_dots_mfma(const float *__restrict__ x, int64_t n, int D,
                                                   const float *__restrict__ cen, int nlist,
                                                   float *__restrict__ dots) {
  __shared__ float As[kMT][kMK + 1];
  __shared__ float Bs[kMT][kMK + 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t r0 = int64_t(blockIdx.y) * kMT;
  const int c0 = blockIdx.x * kMT;
  const int wr = (wave >> 1) * 16, wc = (wave & 1) * 16;   // this wave's 16 x 16 block
  const int ml = lane & 15, kl = lane >> 4;
  floatx4_t acc = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < D; k0 += kMK) {
    stage32(x, n, D, r0, k0, As);
    stage32(cen, nlist, D, c0, k0, Bs);
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < kMK; ks += 4) {
      const float a = As[wr + ml][ks + kl];     // A[m][k]: lane -> (m = lane % 16, k = lane / 16)
      const float b = Bs[wc + ml][ks + kl];     // B[k][n]: lane -> (k = lane / 16, n = lane % 16)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
    }
    __syncthreads();
  }
  // lane holds C[4 (lane / 16) + i][lane % 16]
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t r = r0 + wr + 4 * kl + i;
    const int c = c0 + wc + ml;
    if (r < n && c < nlist) dots[r * nlist + c] = acc[i];
  }
}

// Assignment on the matrix cores (v_mfma_f32_16x16x4f32, full float32) for
// D a multiple of 4 and 16-byte aligned operands.  A workgroup owns 128 rows
// and walks the centres in tiles of 128 (tile128), in increasing order.  After
// each centre tile the distances ||c||^2 - 2 <x, c> update a (distance, id)
// minimum per row and lane (centres visited in increasing order with a
// strict comparison, so the smallest id wins a tie); lanes and the two
// wavefronts sharing a row are merged lexicographically at the end.
constexpr int kAM = 128, kAN = 128, kAK = 32, kAS = kAK + 4;

__device__ __forceinline__ float4 ld4_or_zero(const float *p, bool in) {
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (in) v = *reinterpret_cast<const float4 *>(p);
  return v;
}

// The 128 x 128 product tile of rows (staging offsets aoff, four per thread)
// and centres [c0, c0 + 128) on the matrix cores: four wavefronts of 4 x 4
// v_mfma_f32_16x16x4f32 tiles, k staged through LDS in slabs of 32 (rows
// padded to 36 floats, so that the 16-byte operand reads of eight consecutive
// lanes fall on distinct banks) with the next slab prefetched into registers.
// Within a half slab of 16 both operands use the same permutation of k: lane
// (m, h) supplies k = 4 h + t to MFMA step t, so one 16-byte read covers four
// steps.  Lane (m, h) of wavefront (wr, wc) ends with C[4 h + e][m] of tile
// (i, j): row wr + 16 i + 4 h + e, centre c0 + wc + 16 j + m.
__device__ __forceinline__ void tile128(const float *__restrict__ x, const int64_t (&aoff)[4],
                                        int D, const float *__restrict__ cen, int nlist, int c0,
                                        float (*As)[kAS], float (*Bs)[kAS],
                                        floatx4_t (&acc)[4][4]) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = (wave >> 1) * 64, wc = (wave & 1) * 64;
  const int m = lane & 15, h = lane >> 4;
  const int srow = tid >> 3, scol = (tid & 7) * 4;
  const int nslab = (D + kAK - 1) / kAK;
  int64_t boff[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) boff[u] = int64_t(min(c0 + srow + 32 * u, nlist - 1)) * D + scol;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  float4 pa[4], pb[4];
  const bool in0 = scol < D;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    pa[u] = ld4_or_zero(x + aoff[u], in0);
    pb[u] = ld4_or_zero(cen + boff[u], in0);
  }
  for (int sl = 0; sl < nslab; ++sl) {
    __syncthreads();   // the previous slab's operand reads are done
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      *reinterpret_cast<float4 *>(&As[srow + 32 * u][scol]) = pa[u];
      *reinterpret_cast<float4 *>(&Bs[srow + 32 * u][scol]) = pb[u];
    }
    __syncthreads();
    if (sl + 1 < nslab) {
      const int kn = (sl + 1) * kAK;
      const bool in = kn + scol < D;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        pa[u] = ld4_or_zero(x + aoff[u] + kn, in);
        pb[u] = ld4_or_zero(cen + boff[u] + kn, in);
      }
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      float4 a4[4], b4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a4[i] = *reinterpret_cast<const float4 *>(&As[wr + 16 * i + m][16 * s + 4 * h]);
        b4[i] = *reinterpret_cast<const float4 *>(&Bs[wc + 16 * i + m][16 * s + 4 * h]);
      }
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float av = t == 0 ? a4[i].x : t == 1 ? a4[i].y : t == 2 ? a4[i].z : a4[i].w;
            const float bv = t == 0 ? b4[j].x : t == 1 ? b4[j].y : t == 2 ? b4[j].z : b4[j].w;
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[i][j], 0, 0, 0);
          }
    }
  }
}

__global__ void __launch_bounds__(256) k_assign_mfma(const float *__restrict__ x, int64_t n,
                                                     int D, const float *__restrict__ cen,
                                                     int nlist, const float *__restrict__ cnorm,
                                                     int32_t *__restrict__ out_ids,
                                                     float *__restrict__ out_d) {
  __shared__ float As[kAM][kAS];
  __shared__ float Bs[kAN][kAS];
  __shared__ float red_v[kAM];
  __shared__ int32_t red_i[kAM];
  __shared__ float xx_s[kAM];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = (wave >> 1) * 64, wc = (wave & 1) * 64;
  const int m = lane & 15, h = lane >> 4;
  const int64_t r0 = int64_t(blockIdx.x) * kAM;
  // staging: thread t moves the float4s (row t / 8 + 32 u, column 4 (t % 8)),
  // u = 0..3, of a 128 x 32 slab; rows past the end are clamped (their
  // products are computed and never used)
  const int srow = tid >> 3, scol = (tid & 7) * 4;
  int64_t aoff[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int64_t r = r0 + srow + 32 * u;
    aoff[u] = (r < n ? r : n - 1) * D + scol;
  }
  float best[16];
  int32_t bid[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    best[r] = 3.4e38f;
    bid[r] = 0x7fffffff;
  }
  for (int c0 = 0; c0 < nlist; c0 += kAN) {
    floatx4_t acc[4][4];
    tile128(x, aoff, D, cen, nlist, c0, As, Bs, acc);
    // lane holds C[4 h + e][m] of each 16 x 16 tile: row wr + 16 i + 4 h + e,
    // centre c0 + wc + 16 j + m
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = c0 + wc + 16 * j + m;
      const float cn = c < nlist ? cnorm[c] : __builtin_inff();
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float v = cn - 2.f * acc[i][j][e];   // ||c||^2 - 2 <x, c>
          if (v < best[4 * i + e]) {
            best[4 * i + e] = v;
            bid[4 * i + e] = c;
          }
        }
    }
  }
  // merge the 16 lanes (m) holding the same rows: lexicographic (value, id)
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    for (int off = 1; off < 16; off <<= 1) {
      const float ov = __shfl_xor(best[r], off, 64);
      const int oi = __shfl_xor(bid[r], off, 64);
      if (ov < best[r] || (ov == best[r] && oi < bid[r])) {
        best[r] = ov;
        bid[r] = oi;
      }
    }
  }
  if (wc && m == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        red_v[wr + 16 * i + 4 * h + e] = best[4 * i + e];
        red_i[wr + 16 * i + 4 * h + e] = bid[4 * i + e];
      }
  }
  if (out_d) {   // ||x||^2 of the workgroup's rows: 32 rows per wavefront
    for (int rr = 0; rr < 32; ++rr) {
      const int rl = wave * 32 + rr;
      const int64_t row = r0 + rl < n ? r0 + rl : n - 1;
      float s = 0.f;
      for (int k = 4 * lane; k < D; k += 256) {
        const float4 v = *reinterpret_cast<const float4 *>(x + row * D + k);
        s += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
      }
      s = wave_sum(s);
      if (lane == 0) xx_s[rl] = s;
    }
  }
  __syncthreads();
  if (wc || m) return;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int rl = wr + 16 * i + 4 * h + e;
      float v = best[4 * i + e];
      int32_t id = bid[4 * i + e];
      const float ov = red_v[rl];
      const int32_t oi = red_i[rl];
      if (ov < v || (ov == v && oi < id)) {
        v = ov;
        id = oi;
      }
      const int64_t r = r0 + rl;
      if (r < n) {
        out_ids[r] = id;
        if (out_d) out_d[r] = xx_s[rl] + v;
      }
    }
}

// Probe dots for many rows (D a multiple of 4, 16-byte aligned operands): one
// 128 x 128 tile (tile128) per workgroup, written out.
__global__ void __launch_bounds__(256) k_dots_big(const float *__restrict__ x, int n, int D,
                                                  const float *__restrict__ cen, int nlist,
                                                  float *__restrict__ dots) {
  __shared__ float As[kAM][kAS];
  __shared__ float Bs[kAN][kAS];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = (wave >> 1) * 64, wc = (wave & 1) * 64;
  const int m = lane & 15, h = lane >> 4;
  const int r0 = blockIdx.y * kAM, c0 = blockIdx.x * kAN;
  const int srow = tid >> 3, scol = (tid & 7) * 4;
  int64_t aoff[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) aoff[u] = int64_t(min(r0 + srow + 32 * u, n - 1)) * D + scol;
  floatx4_t acc[4][4];
  tile128(x, aoff, D, cen, nlist, c0, As, Bs, acc);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = r0 + wr + 16 * i + 4 * h + e;
        const int c = c0 + wc + 16 * j + m;
        if (r < n && c < nlist) dots[int64_t(r) * nlist + c] = acc[i][j][e];
      }
}

// Probe dots for D a multiple of 4 and 16-byte aligned operands: a 64 x 64
// output tile per workgroup, each of the four wavefronts a 32 x 32 block as
// 2 x 2 MFMA tiles; k staged through LDS in slabs of 32 with the next slab
// prefetched into registers, the same permuted k within half slabs as the
// assignment kernel.  Every centre row is read from L2 by n / 64 workgroups.
constexpr int kPT = 64;

__global__ void __launch_bounds__(256) k_dots_tiled(const float *__restrict__ x, int n, int D,
                                                    const float *__restrict__ cen, int nlist,
                                                    float *__restrict__ dots) {
  __shared__ float As[kPT][kAS];
  __shared__ float Bs[kPT][kAS];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = (wave >> 1) * 32, wc = (wave & 1) * 32;
  const int m = lane & 15, h = lane >> 4;
  const int r0 = blockIdx.y * kPT, c0 = blockIdx.x * kPT;
  // staging: thread t moves the float4s (row t / 8 + 32 u, column 4 (t % 8)),
  // u = 0, 1, of a 64 x 32 slab; rows past the end are clamped
  const int srow = tid >> 3, scol = (tid & 7) * 4;
  int64_t aoff[2], boff[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    aoff[u] = int64_t(min(r0 + srow + 32 * u, n - 1)) * D + scol;
    boff[u] = int64_t(min(c0 + srow + 32 * u, nlist - 1)) * D + scol;
  }
  floatx4_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  const int nslab = (D + kAK - 1) / kAK;
  float4 pa[2], pb[2];
  const bool in0 = scol < D;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    pa[u] = ld4_or_zero(x + aoff[u], in0);
    pb[u] = ld4_or_zero(cen + boff[u], in0);
  }
  for (int sl = 0; sl < nslab; ++sl) {
    __syncthreads();   // the previous slab's operand reads are done
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      *reinterpret_cast<float4 *>(&As[srow + 32 * u][scol]) = pa[u];
      *reinterpret_cast<float4 *>(&Bs[srow + 32 * u][scol]) = pb[u];
    }
    __syncthreads();
    if (sl + 1 < nslab) {
      const int kn = (sl + 1) * kAK;
      const bool in = kn + scol < D;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        pa[u] = ld4_or_zero(x + aoff[u] + kn, in);
        pb[u] = ld4_or_zero(cen + boff[u] + kn, in);
      }
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      float4 a4[2], b4[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        a4[i] = *reinterpret_cast<const float4 *>(&As[wr + 16 * i + m][16 * s + 4 * h]);
        b4[i] = *reinterpret_cast<const float4 *>(&Bs[wc + 16 * i + m][16 * s + 4 * h]);
      }
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const float av = t == 0 ? a4[i].x : t == 1 ? a4[i].y : t == 2 ? a4[i].z : a4[i].w;
            const float bv = t == 0 ? b4[j].x : t == 1 ? b4[j].y : t == 2 ? b4[j].z : b4[j].w;
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[i][j], 0, 0, 0);
          }
    }
  }
  // lane holds C[4 h + e][m] of each 16 x 16 tile
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = r0 + wr + 16 * i + 4 * h + e;
        const int c = c0 + wc + 16 * j + m;
        if (r < n && c < nlist) dots[int64_t(r) * nlist + c] = acc[i][j][e];
      }
}

struct IdentityId {
  __device__ int32_t operator()(int i) const { return i; }
};

// Top-nprobe of one row of dots (nlist <= 16,384): 1,024 threads hold the
// row in registers.  The dots are binned linearly over [min, max] of the row
// (1,024 bins; the bin index is a non-decreasing function of the dot, so "bin
// >= b" is an up-set of the order), the bin holding the nprobe-th largest dot
// is found, and every dot in it or above is sorted on (dot desc, list asc).
// Value bins spread the row evenly, unlike the leading bits of the float
// keys, which most dots share (LDS atomics on a few bins serialise).  If the
// boundary bin is crowded (equal or clustered dots), 8-bit radix passes over
// the keys take over, and beyond that the block selection.
constexpr int kPSelThreads = 1024;
constexpr int kPSelPer = 16;
constexpr int kPSelBins = 1024;

__global__ void __launch_bounds__(kPSelThreads) k_probe_select_reg(const float *__restrict__ dots,
                                                                   int nlist, int nprobe,
                                                                   int32_t *__restrict__ out_ids,
                                                                   float *__restrict__ out_s) {
  __shared__ SelectSmem sm;   // hist during the counting passes, buf afterwards
  __shared__ float red[2][kPSelThreads / 64];
  const int tid = threadIdx.x, nt = blockDim.x;
  const int64_t row = blockIdx.x;
  const float *d = dots + row * nlist;
  float val[kPSelPer];
  uint32_t key[kPSelPer];
  float lo = __builtin_inff(), hi = -__builtin_inff();
#pragma unroll
  for (int v = 0; v < kPSelPer; ++v) {
    const int i = v * nt + tid;
    val[v] = (i < nlist) ? d[i] : 0.f;
    key[v] = (i < nlist) ? order_key(val[v]) : 0u;   // every real key is > 0
    if (i < nlist) {
      lo = fminf(lo, val[v]);
      hi = fmaxf(hi, val[v]);
    }
  }
  lo = -wave_max(-lo);
  hi = wave_max(hi);
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = lo;
    red[1][tid >> 6] = hi;
  }
  __syncthreads();
  lo = red[0][0];
  hi = red[1][0];
  for (int w = 1; w < nt / 64; ++w) {
    lo = fminf(lo, red[0][w]);
    hi = fmaxf(hi, red[1][w]);
  }
  const float scale = (hi > lo) ? float(kPSelBins) / (hi - lo) : 0.f;
  auto bin_of = [&](float x) { return min(kPSelBins - 1, int((x - lo) * scale)); };
  bool collect_by_bin = false;
  int bbin = 0;
  uint32_t edge = 0;
  if (scale > 0.f && scale < 3.0e38f) {
    for (int b = tid; b < kPSelBins; b += nt) sm.hist[b] = 0;
    __syncthreads();
#pragma unroll
    for (int v = 0; v < kPSelPer; ++v)
      if (v * nt + tid < nlist) atomicAdd(&sm.hist[bin_of(val[v])], 1u);
    find_boundary(sm, kPSelBins, 0u, uint32_t(nprobe));
    bbin = int(sm.bcast[0]);
    collect_by_bin = sm.bcast[1] + sm.hist[bbin] <= uint32_t(kSelCap);
    __syncthreads();
  }
  if (!collect_by_bin) {
    uint32_t prefix = 0, above = 0;
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int b = tid; b < 256; b += nt) sm.hist[b] = 0;
      __syncthreads();
#pragma unroll
      for (int v = 0; v < kPSelPer; ++v) {
        const int i = v * nt + tid;
        if (i < nlist && (shift == 24 || (key[v] >> (shift + 8)) == prefix))
          atomicAdd(&sm.hist[(key[v] >> shift) & 255u], 1u);
      }
      find_boundary(sm, 256, above, uint32_t(nprobe));
      const uint32_t bb = sm.bcast[0];
      const uint32_t in_bin = sm.hist[bb];
      above = sm.bcast[1];
      prefix = (prefix << 8) | bb;
      edge = prefix << shift;
      __syncthreads();
      if (above + in_bin <= uint32_t(kSelCap)) break;
      if (shift == 0) {   // more than kSelCap equal keys at the boundary
        block_topk(d, nlist, nprobe, IdentityId(), out_s + row * nprobe, out_ids + row * nprobe,
                   sm);
        return;
      }
    }
  }
  if (tid == 0) sm.count = 0;
  __syncthreads();
#pragma unroll
  for (int v = 0; v < kPSelPer; ++v) {
    const int i = v * nt + tid;
    const bool take = collect_by_bin ? bin_of(val[v]) >= bbin : key[v] >= edge;
    if (i < nlist && take) sm.buf[atomicAdd(&sm.count, 1u)] = composite(key[v], i);
  }
  __syncthreads();
  emit_sorted(sm, int(sm.count), nprobe, out_s + row * nprobe, out_ids + row * nprobe);
}

// Top-nprobe for rows longer than the register-resident kernel holds.
__global__ void __launch_bounds__(kSelThreads) k_probe_select(const float *__restrict__ dots,
                                                              int nlist, int nprobe,
                                                              int32_t *__restrict__ out_ids,
                                                              float *__restrict__ out_s) {
  __shared__ SelectSmem sm;
  const int64_t row = blockIdx.x;
  block_topk(dots + row * nlist, nlist, nprobe, IdentityId(), out_s + row * nprobe,
             out_ids + row * nprobe, sm);
}

// ------------------------------------------------------------- fixed scratch
// Scratch of ivf_assign_probe_noalloc: a static device array, one per GPU
// the library runs on, held until the process ends.  Host code never uses
// its name as an address: the device address is looked up once per device
// (hipGetSymbolAddress, with that device current) and kept in g_scratch_ptr.
constexpr size_t kProbeScratchBytes = (size_t(64) << 20) + (size_t(256) << 10);
static __device__ __align__(256) unsigned char scratch[kProbeScratchBytes];

constexpr int kMaxDevices = 64;
static void *g_scratch_ptr[kMaxDevices] = {nullptr};
static std::mutex g_scratch_mu;

// Device address of this GPU's scratch (looked up on first use); nullptr
// with *status set when the lookup fails.
static void *scratch_of_current_device(int *status) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    *status = set_hip_error(e);
    return nullptr;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    *status = RSLM_ERR_UNSUPPORTED;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      *status = set_hip_error(e != hipSuccess ? e : hipErrorInvalidSymbol);
      return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
  }
  *status = RSLM_OK;
  return g_scratch_ptr[dev];
}

}  // namespace rslm

using namespace rslm;

extern "C" {

size_t ivf_assign_probe_workspace(int64_t n, int32_t dim, int32_t nlist, int32_t nprobe,
                                  int mode) {
  (void)dim;
  (void)nprobe;
  if (n < 0 || nlist < 1) return 0;
  const size_t norms = (size_t(nlist) * sizeof(float) + 255) / 256 * 256;
  if (mode == IVF_ASSIGN_L2) return norms;
  const size_t dots = size_t(n) * size_t(nlist) * sizeof(float);
  return norms + (dots + 255) / 256 * 256;
}

int ivf_assign_probe(const float *x, int64_t n, int32_t dim, const float *centroids,
                     int32_t nlist, int32_t nprobe, int mode, int32_t *out_ids,
                     float *out_scores, void *ws, size_t ws_bytes, void *stream) {
  if (n < 0 || dim < 1 || nlist < 1 || nlist > 65536) return RSLM_ERR_INVALID_ARG;
  if (mode != IVF_ASSIGN_L2 && mode != IVF_PROBE_IP) return RSLM_ERR_INVALID_ARG;
  if (mode == IVF_ASSIGN_L2 && nprobe != 1) return RSLM_ERR_INVALID_ARG;
  if (mode == IVF_PROBE_IP && (nprobe < 1 || nprobe > nlist || nprobe > kMaxNprobe))
    return RSLM_ERR_INVALID_ARG;
  if (n == 0) return RSLM_OK;
  if (!x || !centroids || !out_ids || (mode == IVF_PROBE_IP && !out_scores))
    return RSLM_ERR_INVALID_ARG;
  if (!ws || ws_bytes < ivf_assign_probe_workspace(n, dim, nlist, nprobe, mode))
    return RSLM_ERR_WORKSPACE;
  hipStream_t s = as_stream(stream);
  if (mode == IVF_ASSIGN_L2) {
    float *cnorm = static_cast<float *>(ws);
    hipLaunchKernelGGL(k_row_norms, dim3((nlist + 3) / 4), dim3(256), 0, s, centroids, nlist,
                       dim, cnorm);
    int st = check_launch();
    if (st) return st;
    const bool aligned16 = (reinterpret_cast<uintptr_t>(x) % 16 == 0) &&
                           (reinterpret_cast<uintptr_t>(centroids) % 16 == 0);
    if (dim % 4 == 0 && aligned16) {   // rows are whole, aligned float4 runs
      const int64_t grid = (n + kAM - 1) / kAM;
      if (grid > 0x7fffffff) return RSLM_ERR_INVALID_ARG;
      hipLaunchKernelGGL(k_assign_mfma, dim3(unsigned(grid)), dim3(256), 0, s, x, n, dim,
                         centroids, nlist, cnorm, out_ids, out_scores);
      return check_launch();
    }
    const int64_t grid = (n + kTM - 1) / kTM;
    if (grid > 0x7fffffff) return RSLM_ERR_INVALID_ARG;
    hipLaunchKernelGGL(k_assign, dim3(unsigned(grid)), dim3(256), 0, s, x, n, dim, centroids,
                       nlist, cnorm, out_ids, out_scores);
    return check_launch();
  }
  const size_t norms = (size_t(nlist) * sizeof(float) + 255) / 256 * 256;
  float *dots = reinterpret_cast<float *>(static_cast<char *>(ws) + norms);
  const int64_t gy32 = (n + kMT - 1) / kMT;
  if (gy32 > 65535) return RSLM_ERR_INVALID_ARG;
  int st;
  const bool aligned16 = (reinterpret_cast<uintptr_t>(x) % 16 == 0) &&
                         (reinterpret_cast<uintptr_t>(centroids) % 16 == 0);
  const int64_t big_tiles = ((n + kAM - 1) / kAM) * ((nlist + kAN - 1) / kAN);
  if (dim % 4 == 0 && aligned16 && big_tiles >= 1024) {   // enough 128 x 128 tiles
    hipLaunchKernelGGL(k_dots_big, dim3(unsigned((nlist + kAN - 1) / kAN),
                                        unsigned((n + kAM - 1) / kAM)),
                       dim3(256), 0, s, x, int(n), dim, centroids, nlist, dots);
  } else if (dim % 4 == 0 && aligned16) {   // rows are whole, aligned float4 runs
    hipLaunchKernelGGL(k_dots_tiled, dim3(unsigned((nlist + kPT - 1) / kPT),
                                          unsigned((n + kPT - 1) / kPT)),
                       dim3(256), 0, s, x, int(n), dim, centroids, nlist, dots);
  } else {
    hipLaunchKernelGGL(k_dots_mfma, dim3((nlist + kMT - 1) / kMT, unsigned(gy32)), dim3(256), 0, s,
                       x, n, dim, centroids, nlist, dots);
  }
  if ((st = check_launch())) return st;
  if (n > 0x7fffffff) return RSLM_ERR_INVALID_ARG;
  if (nlist <= kPSelThreads * kPSelPer)
    hipLaunchKernelGGL(k_probe_select_reg, dim3(unsigned(n)), dim3(kPSelThreads), 0, s, dots, nlist,
                       nprobe, out_ids, out_scores);
  else
    hipLaunchKernelGGL(k_probe_select, dim3(unsigned(n)), dim3(kSelThreads), 0, s, dots, nlist,
                       nprobe, out_ids, out_scores);
  return check_launch();
}

}  // extern "C"

extern "C" {

int ivf_assign_probe_noalloc(const float *x, int64_t n, int32_t dim, const float *centroids,
                             int32_t nlist, int32_t nprobe, int mode, int32_t *out_ids,
                             float *out_scores, void *stream) {
  // the same validation as ivf_assign_probe, then the fixed scratch's limit
  if (n < 0 || dim < 1 || nlist < 1 || nlist > 65536) return RSLM_ERR_INVALID_ARG;
  if (mode != IVF_ASSIGN_L2 && mode != IVF_PROBE_IP) return RSLM_ERR_INVALID_ARG;
  if (mode == IVF_ASSIGN_L2 && nprobe != 1) return RSLM_ERR_INVALID_ARG;
  if (mode == IVF_PROBE_IP && (nprobe < 1 || nprobe > nlist || nprobe > kMaxNprobe))
    return RSLM_ERR_INVALID_ARG;
  if (n == 0) return RSLM_OK;
  if (!x || !centroids || !out_ids || (mode == IVF_PROBE_IP && !out_scores))
    return RSLM_ERR_INVALID_ARG;
  const size_t need = ivf_assign_probe_workspace(n, dim, nlist, nprobe, mode);
  if (need > kProbeScratchBytes) return RSLM_ERR_WORKSPACE;
  int st = RSLM_OK;
  void *ws = scratch_of_current_device(&st);
  if (!ws) return st;
  return ivf_assign_probe(x, n, dim, centroids, nlist, nprobe, mode, out_ids, out_scores, ws,
                          kProbeScratchBytes, stream);
}

size_t ivf_assign_probe_noalloc_limit(void) { return kProbeScratchBytes; }

}  // extern "C"
