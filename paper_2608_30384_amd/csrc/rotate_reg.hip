// Register-resident rotation and 1-D encoder for dimensions that are a
// multiple of the 128-element block (D = 128 NB, NB = 1, 2, 3, 4, 6, 8, 12, 16).
//
// Same arithmetic as the general path (paper, Section "Pre-Quantization
// Transformations": S1, block FWHT, permutation + strided transpose, S2,
// block FWHT), different mapping: lane l of a wavefront holds elements
// e = l + 64 j (j < J = D / 64), so element bits 0..5 are the lane and bit 6
// of the block index is j's parity.  The six lane-bit butterfly stages use
// cross-lane exchanges, the seventh is in registers, and LDS is touched only
// by the strided transpose between the passes.  With 1-D codebooks the
// quantiser, norms, packing (an OR over the 8 lanes of each 8-coordinate
// group) and the rotated second residual stay in registers as well.
#include "rslm_internal.h"

namespace rslm {

__device__ __forceinline__ int px_r(int i) { return i + (i >> 5); }

__device__ __forceinline__ void wave_sync_r() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Orthonormal FWHT of every 128-block of the register vector.
template <int J>
__device__ __forceinline__ void fwht128_reg(float (&x)[J], int lane) {
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) {
    const float sg = (lane & s) ? -1.f : 1.f;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const float p = __shfl_xor(x[j], s, 64);
      x[j] = fmaf(sg, x[j], p);   // lane bit clear: x + p; set: p - x
    }
  }
  constexpr float kInv = 0.08838834764831845f;   // 1 / sqrt(128)
#pragma unroll
  for (int j = 0; j < J; j += 2) {
    const float a = x[j], b = x[j + 1];
    x[j] = (a + b) * kInv;
    x[j + 1] = (a - b) * kInv;
  }
}

// Per-lane sign words: element j of the lane takes sign word w[j mod 4]
// (the sign index pattern repeats every 256 = 4 x 64 elements).
struct SignWords {
  uint32_t w[4];
};
__device__ __forceinline__ SignWords sign_words(uint32_t bits) {
  SignWords s;
#pragma unroll
  for (int t = 0; t < 4; ++t) s.w[t] = ((bits >> t) & 1u) << 31;
  return s;
}
__device__ __forceinline__ float flipw(float v, const SignWords &s, int j) {
  return __uint_as_float(__float_as_uint(v) ^ s.w[j & 3]);
}

// LDS float at a byte offset (the transpose table holds padded byte offsets)
__device__ __forceinline__ float &lds_at(float *buf, uint32_t byte_off) {
  return *reinterpret_cast<float *>(reinterpret_cast<char *>(buf) + byte_off);
}

// Forward rotation of x (already multiplied by S1) through buf (LDS, >= D +
// D/32 floats) for the transpose; ts[o] = byte offset in buf of the source of
// output o.
template <int J>
__device__ __forceinline__ void rotate_fwd_reg(float (&x)[J], const RotParams &rp,
                                               const uint16_t *ts, const SignWords &s2, float *buf,
                                               int lane) {
  if (rp.passes == 0) return;
  fwht128_reg<J>(x, lane);
  if (rp.passes == 1) return;
#pragma unroll
  for (int j = 0; j < J; ++j) buf[px_r(lane + 64 * j)] = x[j];
  wave_sync_r();
#pragma unroll
  for (int j = 0; j < J; ++j) x[j] = flipw(lds_at(buf, ts[lane + 64 * j]), s2, j);
  wave_sync_r();
  fwht128_reg<J>(x, lane);
}

// Inverse rotation R^T (without the final S1, applied by the caller).
template <int J>
__device__ __forceinline__ void rotate_inv_reg(float (&x)[J], const RotParams &rp,
                                               const uint16_t *ts, const SignWords &s2, float *buf,
                                               int lane) {
  if (rp.passes == 0) return;
  fwht128_reg<J>(x, lane);
  if (rp.passes == 1) return;
#pragma unroll
  for (int j = 0; j < J; ++j) lds_at(buf, ts[lane + 64 * j]) = flipw(x[j], s2, j);
  wave_sync_r();
#pragma unroll
  for (int j = 0; j < J; ++j) x[j] = buf[px_r(lane + 64 * j)];
  wave_sync_r();
  fwht128_reg<J>(x, lane);
}

// Workgroup prologue: LDS copy of the transpose source table (D entries), as
// byte offsets into the padded per-wave buffer.
// D = 64 J entries, 256 threads: all loads first (clamped index), then the
// stores.
template <int J>
__device__ __forceinline__ void load_tsrc_r(const RotParams &rp, uint16_t *ts) {
  constexpr int D = 64 * J, kU = (D + 255) / 256;
  if (rp.passes == 2) {
    int16_t tv[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) tv[u] = rp.tsrc[min(int(threadIdx.x) + 256 * u, D - 1)];
#pragma unroll
    for (int u = 0; u < kU; ++u)
      if (int(threadIdx.x) + 256 * u < D) ts[threadIdx.x + 256 * u] = uint16_t(4 * px_r(tv[u]));
  }
  __syncthreads();
}

template <int J>
__global__ void __launch_bounds__(256) k_rotate_reg(const float *__restrict__ x, float *y,
                                                    int64_t n, RotParams rp, int inverse,
                                                    int dstride) {
  extern __shared__ float lds[];
  __shared__ uint16_t ts[64 * J];
  load_tsrc_r<J>(rp, ts);
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int64_t row = int64_t(blockIdx.x) * (blockDim.x >> 6) + wid;
  if (row >= n) return;   // no workgroup barriers below
  float *buf = lds + wid * dstride;
  const uint2 sm = lane_sign_masks(rp, lane);
  const SignWords s1 = sign_words(rp.passes > 0 ? sm.x : 0u), s2 = sign_words(sm.y);
  const float *xr = x + row * (64 * J);
  float v[J];
#pragma unroll
  for (int j = 0; j < J; ++j) v[j] = xr[lane + 64 * j];
  if (!inverse) {
#pragma unroll
    for (int j = 0; j < J; ++j) v[j] = flipw(v[j], s1, j);
    rotate_fwd_reg<J>(v, rp, ts, s2, buf, lane);
  } else {
    rotate_inv_reg<J>(v, rp, ts, s2, buf, lane);
#pragma unroll
    for (int j = 0; j < J; ++j) v[j] = flipw(v[j], s1, j);
  }
  float *yr = y + row * (64 * J);
#pragma unroll
  for (int j = 0; j < J; ++j) yr[lane + 64 * j] = v[j];
}

// ---------------------------------------------------------------------------
// Encoder for 1-D codebooks (3 and 4 bits) at D = 128 NB, four vectors per
// wavefront.  Row rho = lane / 16 of the wavefront holds one vector; lane r =
// lane % 16 of the row holds, of every 128-block b, the 8 consecutive
// coordinates 128 b + 8 r + i (i < 8).  In a block, coordinate bits 0..2 are
// the register index i and bits 3..6 are r, so three butterfly stages are in
// registers and four exchange lanes inside the row through DPP (quad_perm for
// lane xor 1 and 2, half-mirror + quad_perm for xor 4, row_ror:8 for xor 8);
// row reductions are four DPP steps.  The strided transpose between the two
// passes goes through a per-vector LDS buffer.  Codes of a lane's 8
// coordinates form one packed word, stored straight into the tile layout.

constexpr int kDppQuadXor1 = 0xB1;   // quad_perm [1, 0, 3, 2]
constexpr int kDppQuadXor2 = 0x4E;   // quad_perm [2, 3, 0, 1]
constexpr int kDppQuadRev = 0x1B;    // quad_perm [3, 2, 1, 0]
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppRowRor4 = 0x124;
constexpr int kDppRowRor8 = 0x128;

template <int CTRL>
__device__ __forceinline__ float dppf(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, true));
}
// value of lane r ^ 4 of the row: half-mirror (r ^ 7) then quad reverse (^ 3)
__device__ __forceinline__ float dpp_xor4(float v) {
  return dppf<kDppQuadRev>(dppf<kDppHalfMirror>(v));
}
__device__ __forceinline__ float row_sum16(float v) {
  v += dppf<kDppQuadXor1>(v);
  v += dppf<kDppQuadXor2>(v);
  v += dppf<kDppRowRor4>(v);   // quads now uniform: + the next quad
  v += dppf<kDppRowRor8>(v);   // + the two others
  return v;
}
__device__ __forceinline__ float row_max16(float v) {
  v = fmaxf(v, dppf<kDppQuadXor1>(v));
  v = fmaxf(v, dppf<kDppQuadXor2>(v));
  v = fmaxf(v, dppf<kDppRowRor4>(v));
  v = fmaxf(v, dppf<kDppRowRor8>(v));
  return v;
}

// The four lane stages of the 8 elements z[o..o+7] of one block, each a DPP
// multiply-add v_fmac_f32_dpp (z += sg[k] * z of the partner lane: lane r ^ 1,
// r ^ 2, r ^ 4, r ^ 8 of the 16-lane row; r ^ 4 as a half-mirror move then a
// quad reversal).  The compiler does not fold a DPP move into the multiplied
// operand of a multiply-add, so the stages are written out here.  A DPP
// operand must not have been written by the two preceding VALU instructions:
// the block opens and closes with two wait states, and inside it every DPP
// read is at least seven instructions after the write of its register.
#define RSLM_DPP_FMAC(I, SG, SRC, CTRL) \
  "v_fmac_f32_dpp %" #I ", %" #SRC ", %" #SG " " CTRL " row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
#define RSLM_DPP_STAGE(SG, CTRL)                                                           \
  RSLM_DPP_FMAC(0, SG, 0, CTRL) RSLM_DPP_FMAC(1, SG, 1, CTRL) RSLM_DPP_FMAC(2, SG, 2, CTRL) \
  RSLM_DPP_FMAC(3, SG, 3, CTRL) RSLM_DPP_FMAC(4, SG, 4, CTRL) RSLM_DPP_FMAC(5, SG, 5, CTRL) \
  RSLM_DPP_FMAC(6, SG, 6, CTRL) RSLM_DPP_FMAC(7, SG, 7, CTRL)
#define RSLM_DPP_MIRROR(T, I) \
  "v_mov_b32_dpp %" #T ", %" #I " row_half_mirror row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
__device__ __forceinline__ void lane_stages8(float *z, int o, const float (&sg)[4]) {
  float t0, t1, t2, t3, t4, t5, t6, t7;   // half-mirrored copies (stage r ^ 4)
  asm volatile(
      "s_nop 1\n\t"
      RSLM_DPP_STAGE(16, "quad_perm:[1,0,3,2]")
      RSLM_DPP_STAGE(17, "quad_perm:[2,3,0,1]")
      RSLM_DPP_MIRROR(8, 0) RSLM_DPP_MIRROR(9, 1) RSLM_DPP_MIRROR(10, 2) RSLM_DPP_MIRROR(11, 3)
      RSLM_DPP_MIRROR(12, 4) RSLM_DPP_MIRROR(13, 5) RSLM_DPP_MIRROR(14, 6) RSLM_DPP_MIRROR(15, 7)
      RSLM_DPP_FMAC(0, 18, 8, "quad_perm:[3,2,1,0]") RSLM_DPP_FMAC(1, 18, 9, "quad_perm:[3,2,1,0]")
      RSLM_DPP_FMAC(2, 18, 10, "quad_perm:[3,2,1,0]") RSLM_DPP_FMAC(3, 18, 11, "quad_perm:[3,2,1,0]")
      RSLM_DPP_FMAC(4, 18, 12, "quad_perm:[3,2,1,0]") RSLM_DPP_FMAC(5, 18, 13, "quad_perm:[3,2,1,0]")
      RSLM_DPP_FMAC(6, 18, 14, "quad_perm:[3,2,1,0]") RSLM_DPP_FMAC(7, 18, 15, "quad_perm:[3,2,1,0]")
      RSLM_DPP_STAGE(19, "row_ror:8")
      "s_nop 1"
      : "+v"(z[o + 0]), "+v"(z[o + 1]), "+v"(z[o + 2]), "+v"(z[o + 3]), "+v"(z[o + 4]),
        "+v"(z[o + 5]), "+v"(z[o + 6]), "+v"(z[o + 7]), "=&v"(t0), "=&v"(t1), "=&v"(t2),
        "=&v"(t3), "=&v"(t4), "=&v"(t5), "=&v"(t6), "=&v"(t7)
      : "v"(sg[0]), "v"(sg[1]), "v"(sg[2]), "v"(sg[3]));
}
#undef RSLM_DPP_MIRROR
#undef RSLM_DPP_STAGE
#undef RSLM_DPP_FMAC

// Unnormalised FWHT of every 128-block of the row's vector; sg[k] = -1 where
// bit k of r is set.  A lane stage computes own + sg[k] partner, so the
// exchanged value is the multiplied operand and the exchange folds into the
// multiply-add (one DPP multiply-add per element and stage).  In a lane with
// bit k set that is partner - own, the negative of the butterfly's
// difference: after the four lane stages lane r holds (-1)^popcount(r) times
// the transform, which the caller folds into a later sign or scale.
template <int E>
__device__ __forceinline__ void fwht_rows(float (&z)[E], const float (&sg)[4]) {
#pragma unroll
  for (int b = 0; b < E / 8; ++b) {
#pragma unroll
    for (int s = 1; s < 8; s <<= 1) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        if (i & s) continue;
        const float a = z[8 * b + i], c = z[8 * b + i + s];
        z[8 * b + i] = a + c;
        z[8 * b + i + s] = a - c;
      }
    }
  }
  // lane stages, one block at a time
#pragma unroll
  for (int b = 0; b < E / 8; ++b) lane_stages8(z, 8 * b, sg);
}

// sign bit (bit 31) of coordinate 128 b + 8 r + i from the lane's 16-bit
// mask: bit 8 (b mod 2) + i (the sign tables repeat every 256 coordinates)
__device__ __forceinline__ uint32_t sgnbit(uint32_t m, int b, int i) {
  return ((m >> (8 * (b & 1) + i)) & 1u) << 31;
}

// Quantiser grid buckets the register-path encoder holds in LDS (the plan's
// grids for the Lloyd-Max codebooks have 128; larger grids take the general
// path).
constexpr int kQuantBuckets = 128;

// Stand-in centre rows (zeros) for records encoded without a centre.
__device__ __align__(16) const float kZeroRow[2048] = {};

// S2 selects the output of the second residual R x - g^ (R c + s^ c^):
//   0: float32 rows (resid, when given);
//   1: the second (rescoring) RSLM stage with a 2-D K = 16 codebook (the
//      2-bit codec): the pairs (8 r + 2 k, 8 r + 2 k + 1) of a block are
//      sub-vectors 64 b + 4 r + k, so a lane's four codes of a block are 16
//      consecutive bits of the canonical record at byte 32 b + 2 r;
//   2: SQ8 codes with the ranges sq8_lo / sq8_hi, 8 bytes per lane and block.
// LITE (Rslm4Lite): the lanes holding the first cp.lead coordinates (block 0,
// r < cp.lead / 8) quantise on the K = 8 codebook's bucket grid and
// thresholds (padded with +inf, so codes stay 0..7) and decode with that
// codebook; their stored code words carry the scale bits in bit 3 of each
// nibble.
template <int NB, int BITS, int S2, bool LITE = false>
__global__ void __launch_bounds__(256) k_encode_rows(
    const float *__restrict__ x, int64_t n_rows, const int64_t *__restrict__ src_row,
    const int32_t *__restrict__ rec_list, int64_t n_records, const float *__restrict__ cen,
    const float *__restrict__ cen_rot, int nlist, uint8_t *__restrict__ codes,
    uint32_t *__restrict__ scales, float *__restrict__ resid, RotParams rp, CodecParams cp,
    uint8_t *__restrict__ codes2, uint32_t *__restrict__ scales2, CodecParams cp2,
    const float *__restrict__ sq8_lo, const float *__restrict__ sq8_hi) {
  constexpr bool TWO = S2 == 1;
  constexpr int D = 128 * NB;
  constexpr int E = 8 * NB;
  constexpr int K = 1 << BITS;
  constexpr int kVecStride = D + 4;   // floats per vector buffer (offset of 4 banks per row)
  __shared__ float buf[16 * kVecStride];
  __shared__ float cbs[16], thr[16];
  // Rslm4Lite: K = 8 codebook of the leading lanes
  __shared__ float cb8[LITE ? 16 : 1], thr8[LITE ? 16 : 1];
  // second codebook: (first, second coordinate, |C_k|^2 / 2) per code, and
  // the candidate lists of its nearest-centroid grid
  __shared__ float4 cb2[TWO ? 16 : 1];
  __shared__ uint16_t g2t[TWO ? kGrid2 * kGrid2 : 1];
  __shared__ uint32_t rmask[16];
  // per lane r: bit 8 b + i (word b / 4) = sign of element (b, i) after the
  // transpose: S2 of the target coordinate times the lane sign (-1)^popcount
  // that the first pass left on its source coordinate
  constexpr int kTmWords = (NB + 3) / 4;   // 4 blocks of 8 sign bits per word
  __shared__ uint32_t tmask[16][kTmWords];
  // quantiser grids: thresholds below each bucket (cp.qn, cp.qn_lead <=
  // kQuantBuckets)
  __shared__ uint8_t qtab[kQuantBuckets];
  __shared__ uint8_t qtab8[LITE ? kQuantBuckets : 1];

  __shared__ uint16_t ts[D];
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int rho = lane >> 4, r = lane & 15;
  if (TWO && threadIdx.x < 16)
    cb2[threadIdx.x] = make_float4(cp2.cb[2 * threadIdx.x], cp2.cb[2 * threadIdx.x + 1],
                                   cp2.cbh[threadIdx.x], 0.f);
  if (TWO) {   // all loads first, then the stores (kGrid2^2 is a multiple of 256)
    static_assert(kGrid2 * kGrid2 % 256 == 0, "grid table copy");
    uint16_t gv[TWO ? kGrid2 * kGrid2 / 256 : 1];
#pragma unroll
    for (int u = 0; u < (TWO ? kGrid2 * kGrid2 / 256 : 1); ++u) gv[u] = cp2.g2tab[threadIdx.x + 256 * u];
#pragma unroll
    for (int u = 0; u < (TWO ? kGrid2 * kGrid2 / 256 : 1); ++u) g2t[threadIdx.x + 256 * u] = gv[u];
  }
  if (LITE && threadIdx.x < 16) {
    cb8[threadIdx.x] = (threadIdx.x < 8) ? cp.cb_lead[threadIdx.x] : 0.f;
    thr8[threadIdx.x] = cp.thr_lead[threadIdx.x];
  }
  if (threadIdx.x < 16) {
    cbs[threadIdx.x] = cp.cb[threadIdx.x];
    // sorted decision thresholds, padded with +inf (the comparison after the
    // bucket lookup never passes beyond the last one)
    thr[threadIdx.x] = (int(threadIdx.x) + 1 < K) ? cp.thr[threadIdx.x] : __builtin_inff();
    // S1 sign bits of coordinates 128 p + 8 t + i (p < 2: the signs repeat
    // every 256 coordinates)
    uint32_t m = 0;
    for (int pi = 0; pi < 16; ++pi) {
      const int c = 128 * (pi >> 3) + 8 * int(threadIdx.x) + (pi & 7);
      m |= sign_bit(rp.s1mask, c) << pi;
    }
    rmask[threadIdx.x] = m;
    if (rp.passes == 2) {
      uint32_t tm[kTmWords] = {};
      for (int b = 0; b < NB; ++b)
        for (int i = 0; i < 8; ++i) {
          const int o = 128 * b + 8 * int(threadIdx.x) + i;
          const int src_lane = (rp.tsrc[o] >> 3) & 15;
          const uint32_t bit = sign_bit(rp.s1mask, o + 127) ^ (__popc(src_lane) & 1u);
          tm[b >> 2] |= bit << (8 * (b & 3) + i);
        }
      for (int t = 0; t < kTmWords; ++t) tmask[threadIdx.x][t] = tm[t];
    }
  }
  if (rp.passes == 2) {   // all loads first (clamped index), then the stores
    constexpr int kU = (D + 255) / 256;
    int16_t tv[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) tv[u] = rp.tsrc[min(int(threadIdx.x) + 256 * u, D - 1)];
#pragma unroll
    for (int u = 0; u < kU; ++u)
      if (int(threadIdx.x) + 256 * u < D) ts[threadIdx.x + 256 * u] = uint16_t(4 * tv[u]);
  }

  for (int j = threadIdx.x; j < cp.qn; j += blockDim.x) {
    int cnt = 0;
#pragma unroll
    for (int k = 0; k + 1 < K; ++k) cnt += quant_bucket(cp.thr[k], cp.qs, cp.qo, cp.qn) < j;
    qtab[j] = uint8_t(cnt);
  }
  if (LITE)
    for (int j = threadIdx.x; j < cp.qn_lead; j += blockDim.x) {
      int cnt = 0;
#pragma unroll
      for (int k = 0; k < 7; ++k)
        cnt += quant_bucket(cp.thr_lead[k], cp.qs_lead, cp.qo_lead, cp.qn_lead) < j;
      qtab8[j] = uint8_t(cnt);
    }
  __syncthreads();
  const int64_t rec = (int64_t(blockIdx.x) * (blockDim.x >> 6) + wid) * 4 + rho;
  int64_t row = -1;
  int L = -1;
  if (rec < n_records) {
    row = src_row ? src_row[rec] : rec;
    if (row >= n_rows) row = -1;
    if (cen && row >= 0) {
      L = rec_list[rec];
      if (L < 0 || L >= nlist) row = -1;
    }
  }
  // A row without a vector leaves; rows never exchange data, and no
  // workgroup barrier follows.
  if (row < 0) return;
  const uint32_t m1 = rmask[r];
  const float sg[4] = {(r & 1) ? -1.f : 1.f, (r & 2) ? -1.f : 1.f, (r & 4) ? -1.f : 1.f,
                       (r & 8) ? -1.f : 1.f};

  // residual r = x - c, its sums, and S1
  const float *xr = x + row * D + 8 * r;
  const float *cr = ((L >= 0) ? cen + int64_t(L) * D : kZeroRow) + 8 * r;
  float z[E];
  float xx = 0.f, rr = 0.f, cc = 0.f;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const float4 xv = *reinterpret_cast<const float4 *>(xr + 128 * b + 4 * h);
      const float4 cv4 = *reinterpret_cast<const float4 *>(cr + 128 * b + 4 * h);
      const float xa[4] = {xv.x, xv.y, xv.z, xv.w};
      const float ca[4] = {cv4.x, cv4.y, cv4.z, cv4.w};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int i = 4 * h + t;
        const float d = xa[t] - ca[t];
        xx = fmaf(xa[t], xa[t], xx);
        rr = fmaf(d, d, rr);
        cc = fmaf(ca[t], ca[t], cc);
        const uint32_t sb = (rp.passes > 0) ? sgnbit(m1, b, i) : 0u;
        z[8 * b + i] = __uint_as_float(__float_as_uint(d) ^ sb);
      }
    }
    if (b % 2 == 1) __builtin_amdgcn_sched_barrier(0);   // at most 2 blocks of loads in flight
  }
  // reduce right away: a late use lets the compiler sink the accumulation
  // chains and keep every input alive until then
  xx = row_sum16(xx);
  rr = row_sum16(rr);
  cc = row_sum16(cc);
  // rotation: FWHT, [permute + strided transpose, S2, FWHT]; 1/sqrt(128) per pass
  float scale = 1.f;
  if (rp.passes > 0) {
    fwht_rows<E>(z, sg);
    scale = rp.inv_sqrt_b;
    if (rp.passes == 2) {
      float *vb = buf + (4 * wid + rho) * kVecStride;
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          *reinterpret_cast<float4 *>(vb + 128 * b + 8 * r + 4 * h) =
              make_float4(z[8 * b + 4 * h], z[8 * b + 4 * h + 1], z[8 * b + 4 * h + 2],
                          z[8 * b + 4 * h + 3]);
      wave_sync_r();
      uint32_t tm[kTmWords];
#pragma unroll
      for (int t = 0; t < kTmWords; ++t) tm[t] = tmask[r][t];
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const uint4 t8 = *reinterpret_cast<const uint4 *>(ts + 128 * b + 8 * r);
        const uint32_t tw[4] = {t8.x, t8.y, t8.z, t8.w};
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const uint32_t off = (tw[i >> 1] >> (16 * (i & 1))) & 0xffffu;
          const uint32_t sb = ((tm[b >> 2] >> (8 * (b & 3) + i)) & 1u) << 31;
          z[8 * b + i] = __uint_as_float(__float_as_uint(lds_at(vb, off)) ^ sb);
        }
      }
      wave_sync_r();
      fwht_rows<E>(z, sg);
      scale = rp.inv_sqrt_b * rp.inv_sqrt_b;
    }
    if (__popc(r) & 1) scale = -scale;   // the lane sign of the last pass
  }
  float m = 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    z[e] *= scale;
    m = fmaxf(m, fabsf(z[e]));
  }
  m = row_max16(m);
  const float inv_s0 = (m > 0.f) ? cp.emax / m : 0.f;

  // nearest centroid of the sorted 1-D codebook = number of thresholds below
  // u: the count below u's bucket on the quantiser grid plus one comparison
  // with the next threshold (the grid has at most one per bucket).  Only the
  // packed words are kept; centroid values are looked up again where needed
  // (registers, not recomputation, bound this kernel).  ||c^||^2 and
  // <R c, c^> accumulate here, the rotated centre streamed one block ahead.
  const bool has_rc = L >= 0 && cen_rot;
  const float *rcr = (has_rc ? cen_rot + int64_t(L) * D : kZeroRow) + 8 * r;
  uint32_t word[NB];
  float cn2 = 0.f, rcd = 0.f;
  const bool lead_lane = LITE && r < cp.lead / 8;   // block 0 of these lanes is on cb8
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const bool lb = LITE && b == 0 && lead_lane;
    float *tb = lb ? thr8 : thr;
    float *cbb = lb ? cb8 : cbs;
    const uint8_t *qt = lb ? qtab8 : qtab;
    const float qs = lb ? cp.qs_lead : cp.qs, qo = lb ? cp.qo_lead : cp.qo;
    const int qn = lb ? cp.qn_lead : cp.qn;
    uint32_t code[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float u = z[8 * b + i] * inv_s0;
      const uint32_t base = qt[quant_bucket(u, qs, qo, qn)];
      code[i] = base + ((u > tb[base]) ? 1u : 0u);
    }
    word[b] = 0u;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      word[b] |= code[i] << (BITS * i);
      const float v = cbb[code[i]];
      cn2 = fmaf(v, v, cn2);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  // a zero residual has codes 0 (its cn2 and rcd are multiplied by s^ = 0)
  if (!(m > 0.f))
#pragma unroll
    for (int b = 0; b < NB; ++b) word[b] = 0u;
  cn2 = row_sum16(cn2);
  // centroid value of a code (a zero residual has codes 0 and s^ = 0, so the
  // value its codes decode to is always multiplied by 0)
  auto centroid = [&](int b, int i) {
    float *cbb = (LITE && b == 0 && lead_lane) ? cb8 : cbs;
    return lds_at(cbb, 4u * ((word[b] >> (BITS * i)) & uint32_t(K - 1)));
  };
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const float4 v = *reinterpret_cast<const float4 *>(rcr + 128 * b + 4 * h);
      const float va[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int t = 0; t < 4; ++t) rcd = fmaf(va[t], centroid(b, 4 * h + t), rcd);
    }
  rcd = row_sum16(rcd);
  const float s = (m > 0.f && cn2 > 0.f) ? sqrtf(rr / cn2) : 0.f;
  const uint32_t su = enc_ue7m9(s);
  const float sh = dec_ue7m9(su);
  uint32_t gu = 0x7000u;
  const float den2 = cc + 2.f * sh * rcd + sh * sh * cn2;   // ||c + R^T s^ c^||^2
  if (cp.global) {
    const float gv = (den2 > 0.f) ? sqrtf(xx / den2) : 0.f;
    gu = enc_ue4m12(gv);
  }
  if (r == 0) scales[rec] = su | (gu << 16);

  // packed words into the scan tile layout: group G = 16 b + r of record n
  // goes to lane stream 16 (r & 3) + n at byte c BITS, c = G / 4 = 4 b + r / 4
  uint8_t *tile = codes + (rec >> 4) * int64_t(cp.tile_bytes);
  const int n = int(rec & 15);
  uint32_t emb = 0u;   // Rslm4Lite: scale byte of this lane spread into bit 3 of each nibble
  if (LITE && lead_lane) {
    const uint32_t byte = ((r < 2 ? su : gu) >> (8 * (r & 1))) & 0xffu;
#pragma unroll
    for (int i = 0; i < 8; ++i) emb |= ((byte >> i) & 1u) << (4 * i + 3);
  }
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int c = 4 * b + (r >> 2);
    if (BITS == 4) {
      const int off = 4 * c;   // 4 bytes inside one 16-byte unit
      *reinterpret_cast<uint32_t *>(tile + ((off >> 4) * 64 + 16 * (r & 3) + n) * 16 + (off & 15)) =
          (b == 0) ? (word[b] | emb) : word[b];
    } else {
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        const int off = 3 * c + t;
        tile[((off >> 4) * 64 + 16 * (r & 3) + n) * 16 + (off & 15)] = uint8_t(word[b] >> (8 * t));
      }
    }
  }
  if (TWO) {
    // second residual r2 = R x - R a, R a = g^ (R c + s^ c^), kept in z.
    // The rotated centre is read again where it is needed rather than kept
    // (opaque zero offsets stop the compiler from holding earlier loads).
    const float gh = dec_ue4m12(gu);
    float m2 = 0.f, rr2 = 0.f;
    int off1 = 0;
    asm volatile("" : "+v"(off1));
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float4 v = *reinterpret_cast<const float4 *>(rcr + off1 + 128 * b + 4 * h);
        const float va[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int e = 8 * b + 4 * h + t;
          const float d = z[e] + va[t] - gh * (va[t] + sh * centroid(b, 4 * h + t));
          z[e] = d;
          m2 = fmaxf(m2, fabsf(d));
          rr2 = fmaf(d, d, rr2);
        }
      }
    m2 = row_max16(m2);
    rr2 = row_sum16(rr2);
    const float inv2 = (m2 > 0.f) ? cp2.emax / m2 : 0.f;
    // Nearest 2-D centroid: argmin_k |c_k|^2 / 2 - <u, c_k> (lower k on
    // ties) over the (at most four) codes listed for u's cell of the grid,
    // in ascending order with a strict comparison: the same code as a scan
    // of all K (the lists hold every code that can be nearest in the cell).
    // With the codes of a block: ||c2^||^2, <c^, c2^> and <R c, c2^>.  A
    // zero r2 (m2 = 0) gets codes 0 and s2^ = 0, which removes these sums
    // from g2^, so they need no guard.
    uint32_t w2[NB];
    float cn22 = 0.f, c12 = 0.f, rc2 = 0.f;
    int off2 = 0;
    asm volatile("" : "+v"(off2));
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const float4 ra = *reinterpret_cast<const float4 *>(rcr + off2 + 128 * b);
      const float4 rb = *reinterpret_cast<const float4 *>(rcr + off2 + 128 * b + 4);
      float nu0[4], nu1[4], best[4];
      uint32_t code[4];
      uint32_t cell[4];
#pragma unroll
      for (int k2 = 0; k2 < 4; ++k2) {
        const float u0 = z[8 * b + 2 * k2] * inv2, u1 = z[8 * b + 2 * k2 + 1] * inv2;
        nu0[k2] = -u0;
        nu1[k2] = -u1;
        best[k2] = 3.4e38f;
        code[k2] = 0u;
        const int gx = int(__builtin_amdgcn_fmed3f(fmaf(u0, cp2.g2s, cp2.g2o), 0.f, float(kGrid2 - 1)));
        const int gy = int(__builtin_amdgcn_fmed3f(fmaf(u1, cp2.g2s, cp2.g2o), 0.f, float(kGrid2 - 1)));
        cell[k2] = g2t[gx * kGrid2 + gy];
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
#pragma unroll
        for (int k2 = 0; k2 < 4; ++k2) {
          const uint32_t k = (cell[k2] >> (4 * t)) & 15u;
          const float4 ck = cb2[k];
          const float d = fmaf(nu1[k2], ck.y, fmaf(nu0[k2], ck.x, ck.z));
          code[k2] = (d < best[k2]) ? k : code[k2];
          best[k2] = fminf(best[k2], d);
        }
      }
      const float rcv[8] = {ra.x, ra.y, ra.z, ra.w, rb.x, rb.y, rb.z, rb.w};
      uint32_t wb = word[b];   // first-stage codes, looked up again
      asm volatile("" : "+v"(wb));
      w2[b] = 0u;
#pragma unroll
      for (int k2 = 0; k2 < 4; ++k2) {
        const uint32_t cd = code[k2];
        w2[b] |= cd << (4 * k2);
        const float4 cc = cb2[cd];
        const float c0 = cc.x, c1 = cc.y;
        cn22 = fmaf(c0, c0, fmaf(c1, c1, cn22));
        const float e0 = lds_at(cbs, 4u * ((wb >> (BITS * 2 * k2)) & uint32_t(K - 1)));
        const float e1 = lds_at(cbs, 4u * ((wb >> (BITS * (2 * k2 + 1))) & uint32_t(K - 1)));
        c12 = fmaf(e0, c0, fmaf(e1, c1, c12));
        rc2 = fmaf(rcv[2 * k2], c0, fmaf(rcv[2 * k2 + 1], c1, rc2));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if (!(m2 > 0.f))
#pragma unroll
      for (int b = 0; b < NB; ++b) w2[b] = 0u;
    cn22 = row_sum16(cn22);
    const float rad = gh * row_sum16(fmaf(sh, c12, rc2));   // <R a, c2^>
    const float s2 = (m2 > 0.f && cn22 > 0.f) ? sqrtf(rr2 / cn22) : 0.f;
    const uint32_t su2 = enc_ue7m9(s2);
    const float sh2 = dec_ue7m9(su2);
    uint32_t gu2 = 0x7000u;
    if (cp2.global) {
      const float dd = gh * gh * den2 + 2.f * sh2 * rad + sh2 * sh2 * cn22;
      gu2 = enc_ue4m12((dd > 0.f) ? sqrtf(xx / dd) : 0.f);
    }
    if (r == 0) scales2[row] = su2 | (gu2 << 16);
    uint8_t *dst = codes2 + row * int64_t(cp2.canon_bytes) + 2 * r;
#pragma unroll
    for (int b = 0; b < NB; ++b) *reinterpret_cast<uint16_t *>(dst + 32 * b) = uint16_t(w2[b]);
  }
  if (S2 == 2) {
    // SQ8 codes of the second residual (the rslm_sq8_encode arithmetic)
    const float gh = dec_ue4m12(gu);
    uint8_t *dst = codes2 + row * D + 8 * r;   // indexed by source row
    const float *lo_r = sq8_lo + 8 * r, *hi_r = sq8_hi + 8 * r;
    // lo and 255 / (hi - lo) of every dimension (sq8_inv), staged once per
    // wavefront in its vector buffers (free after the rotation) by the lanes
    // still running, instead of a reciprocal per coordinate: the four rows
    // share the dimensions
    float *sq_inv = buf + 4 * wid * kVecStride, *sq_lo = sq_inv + D;
    static_assert(2 * D <= 4 * kVecStride, "ranges fit the wavefront's vector buffers");
    if constexpr (!LITE) {
      wave_sync_r();   // the wavefront is done with its vector buffers
      const uint64_t act = __ballot(1);
      const int n_act = __popcll(act);
      const int me = __popcll(act & ((uint64_t(1) << lane) - 1u));
      if (n_act == 64) {
        // every lane: dimensions lane + 64 j, loads of four j in flight
#pragma unroll
        for (int j0 = 0; j0 < D / 64; j0 += 4) {
          float l4[4], h4[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            l4[t] = sq8_lo[lane + 64 * (j0 + t)];
            h4[t] = sq8_hi[lane + 64 * (j0 + t)];
          }
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            sq_inv[lane + 64 * (j0 + t)] = sq8_inv(l4[t], h4[t]);
            sq_lo[lane + 64 * (j0 + t)] = l4[t];
          }
        }
      } else {
        for (int d = me; d < D; d += n_act) {
          sq_inv[d] = sq8_inv(sq8_lo[d], sq8_hi[d]);
          sq_lo[d] = sq8_lo[d];
        }
      }
      wave_sync_r();
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      uint32_t word2[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float4 v = *reinterpret_cast<const float4 *>(rcr + 128 * b + 4 * h);
        const float4 l4 = *reinterpret_cast<const float4 *>(
            (LITE ? lo_r : sq_lo + 8 * r) + 128 * b + 4 * h);
        const float va[4] = {v.x, v.y, v.z, v.w};
        const float la[4] = {l4.x, l4.y, l4.z, l4.w};
        float ia[4];
        if constexpr (!LITE) {
          const float4 i4 = *reinterpret_cast<const float4 *>(sq_inv + 128 * b + 8 * r + 4 * h);
          ia[0] = i4.x;
          ia[1] = i4.y;
          ia[2] = i4.z;
          ia[3] = i4.w;
        } else {
          const float4 h4 = *reinterpret_cast<const float4 *>(hi_r + 128 * b + 4 * h);
          const float ha[4] = {h4.x, h4.y, h4.z, h4.w};
#pragma unroll
          for (int t = 0; t < 4; ++t) ia[t] = sq8_inv(la[t], ha[t]);
        }
        uint32_t wv = 0u;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int e = 8 * b + 4 * h + t;
          const float o = z[e] + va[t] - gh * (va[t] + sh * centroid(b, 4 * h + t));
          wv = sq8_code_put(wv, o, la[t], ia[t], t);
        }
        word2[h] = wv;
      }
      *reinterpret_cast<uint2 *>(dst + 128 * b) = make_uint2(word2[0], word2[1]);
    }
  }
  if (S2 == 0 && resid) {
    const float gh = dec_ue4m12(gu);
    float *out = resid + row * D + 8 * r;   // indexed by source row
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float4 v = *reinterpret_cast<const float4 *>(rcr + 128 * b + 4 * h);
        const float va[4] = {v.x, v.y, v.z, v.w};
        float o[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int e = 8 * b + 4 * h + t;
          o[t] = z[e] + va[t] - gh * (va[t] + sh * centroid(b, 4 * h + t));
        }
        *reinterpret_cast<float4 *>(out + 128 * b + 4 * h) = make_float4(o[0], o[1], o[2], o[3]);
      }
  }
}

// Launchers: return false when D is not handled here.
#define RSLM_REG_SWITCH(NB, CALL) \
  switch (NB) {                   \
    case 1: CALL(2); break;       \
    case 2: CALL(4); break;       \
    case 3: CALL(6); break;       \
    case 4: CALL(8); break;       \
    case 6: CALL(12); break;      \
    case 8: CALL(16); break;      \
    case 12: CALL(24); break;     \
    case 16: CALL(32); break;     \
    default: return false;        \
  }

bool reg_path_ok(const RotParams &rp) {
  if (rp.B != 128 || rp.overlap || rp.D % 128) return false;
  const int nb = rp.D / 128;
  return nb == 1 || nb == 2 || nb == 3 || nb == 4 || nb == 6 || nb == 8 || nb == 12 || nb == 16;
}

static int reg_dstride(int D) { return (D + (D >> 5) + 4 + 3) / 4 * 4; }

bool launch_rotate_reg(const rslm_plan *p, const float *x, float *y, int64_t n, int inverse,
                       hipStream_t s) {
  if (!reg_path_ok(p->rot)) return false;
  const int dstride = reg_dstride(p->rot.D);
  const int waves = 4;
  const size_t shm = size_t(waves) * dstride * sizeof(float);
  const unsigned grid = unsigned((n + waves - 1) / waves);
#define CALL(J)                                                                            \
  hipLaunchKernelGGL((k_rotate_reg<J>), dim3(grid), dim3(64 * waves), shm, s, x, y, n, p->rot, \
                     inverse, dstride)
  RSLM_REG_SWITCH(p->rot.D / 128, CALL)
#undef CALL
  return true;
}

bool launch_encode_reg(const rslm_plan *p, const rslm_plan *p2, const float *x, int64_t n_rows,
                       const int64_t *src_row, const int32_t *rec_list, int64_t n_records,
                       const float *cen, const float *cen_rot, int nlist, uint8_t *codes,
                       uint32_t *scales, float *resid, uint8_t *codes2, uint32_t *scales2,
                       const float *sq8_lo, const float *sq8_hi, hipStream_t s) {
  if (!reg_path_ok(p->rot) || p->codec.g != 1 || p->codec.d_pad != p->rot.D) return false;
  const int s2 = p2 ? 1 : (sq8_lo ? 2 : 0);
  // the RSLM second stage here is the 2-D K = 16 codec only
  if (s2 == 1 && (p2->codec.g != 2 || p2->codec.K != 16 || p2->codec.n_sub * 2 != p->rot.D ||
                  p2->codec.canon_bytes * 4 != p->rot.D || resid || !p2->codec.g2tab))
    return false;
  if (s2 != 0 && p->codec.bits != 4) return false;
  const bool lite = p->codec.lead > 0;
  if (lite && s2 == 1) return false;   // Lite with an RSLM second stage: general path
  // codebooks whose thresholds no quantiser grid separates: general path
  if (p->codec.qn == 0 || (lite && p->codec.qn_lead == 0)) return false;
  if (p->codec.qn > kQuantBuckets || (lite && p->codec.qn_lead > kQuantBuckets)) return false;
  // 16-byte vector loads and stores of every row
  if ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(cen) |
       reinterpret_cast<uintptr_t>(cen_rot) | reinterpret_cast<uintptr_t>(resid) |
       reinterpret_cast<uintptr_t>(sq8_lo) | reinterpret_cast<uintptr_t>(sq8_hi)) % 16)
    return false;
  if (s2 == 1 && (reinterpret_cast<uintptr_t>(codes2) % 2)) return false;
  if (s2 == 2 && (reinterpret_cast<uintptr_t>(codes2) % 8 || resid)) return false;
  const int64_t groups = (n_records + 15) / 16;   // 16 vectors per 256-thread workgroup
  if (groups > 0x7fffffff) return false;
  const unsigned grid = unsigned(groups);
  const CodecParams &cp2 = p2 ? p2->codec : p->codec;
#define CALL_B(NB, B, ...)                                                                      \
  hipLaunchKernelGGL((k_encode_rows<NB, B, __VA_ARGS__>), dim3(grid), dim3(256), 0, s, x, n_rows,  \
                     src_row,                                                                    \
                     rec_list, n_records, cen, cen_rot, nlist, codes, scales, resid, p->rot,      \
                     p->codec, codes2, scales2, cp2, sq8_lo, sq8_hi)
#define CALL(J)                  \
  if (s2 == 1)                   \
    CALL_B((J) / 2, 4, 1);       \
  else if (s2 == 2 && lite)      \
    CALL_B((J) / 2, 4, 2, true); \
  else if (s2 == 2)              \
    CALL_B((J) / 2, 4, 2);       \
  else if (lite)                 \
    CALL_B((J) / 2, 4, 0, true); \
  else if (p->codec.bits == 4)   \
    CALL_B((J) / 2, 4, 0);       \
  else                           \
    CALL_B((J) / 2, 3, 0)
  RSLM_REG_SWITCH(p->rot.D / 128, CALL)
#undef CALL
#undef CALL_B
  return true;
}

}  // namespace rslm
