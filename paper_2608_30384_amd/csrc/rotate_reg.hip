// Register-resident rotation and 1-D encoder for dimensions that are a
// multiple of the 128-element block (D = 128 NB, NB = 1, 2, 3, 4, 6, 8).
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
__device__ __forceinline__ void load_tsrc_r(const RotParams &rp, uint16_t *ts) {
  if (rp.passes == 2)
    for (int k = threadIdx.x; k < rp.D; k += blockDim.x)
      ts[k] = uint16_t(4 * px_r(rp.tsrc[k]));
  __syncthreads();
}

template <int J>
__global__ void __launch_bounds__(256) k_rotate_reg(const float *__restrict__ x, float *y,
                                                    int64_t n, RotParams rp, int inverse,
                                                    int dstride) {
  extern __shared__ float lds[];
  __shared__ uint16_t ts[64 * J];
  load_tsrc_r(rp, ts);
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

// Byte address of group G (coordinates [8G, 8G + 8)) of record rec in the
// scan tile layout (see the general encoder for the layout).
__device__ __forceinline__ int64_t tile_addr_r(int64_t rec, int G, int t, const CodecParams &cp) {
  const int64_t tile = rec >> 4;
  const int n = int(rec & 15);
  const int c = G >> 2, r = G & 3;
  const int off = c * cp.bits + t;
  return tile * cp.tile_bytes + int64_t((off >> 4) * 64 + r * 16 + n) * 16 + (off & 15);
}

// Encoder for 1-D codebooks (3 and 4 bits), registers only after the loads.
template <int J, int BITS>
__global__ void __launch_bounds__(256) k_encode_reg(
    const float *__restrict__ x, int64_t n_rows, const int64_t *__restrict__ src_row,
    const int32_t *__restrict__ rec_list, int64_t n_records, const float *__restrict__ cen,
    const float *__restrict__ cen_rot, int nlist, uint8_t *__restrict__ codes,
    uint32_t *__restrict__ scales, float *__restrict__ resid, RotParams rp, CodecParams cp,
    int dstride) {
  constexpr int D = 64 * J;
  constexpr int K = 1 << BITS;
  extern __shared__ float lds[];
  __shared__ float cbs[16], thr[16];
  __shared__ uint16_t ts[D];
  const int lane = threadIdx.x & 63;
  // record, source row and list are the same for the whole wavefront; kept
  // in scalar registers so every address below is scalar base + lane offset
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nw = blockDim.x >> 6;
  if (threadIdx.x < 16) {
    cbs[threadIdx.x] = cp.cb[threadIdx.x];
    // sorted decision thresholds, padded with +inf for the binary search
    thr[threadIdx.x] = (int(threadIdx.x) + 1 < cp.K) ? cp.thr[threadIdx.x] : __builtin_inff();
  }
  load_tsrc_r(rp, ts);
  const int64_t rec = int64_t(blockIdx.x) * nw + wid;
  int64_t row = -1;
  int L = -1;
  if (rec < n_records) {
    if (src_row) {
      const int64_t sr = src_row[rec];
      row = int64_t((uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(int(uint64_t(sr) >> 32)))) << 32) |
                    uint32_t(__builtin_amdgcn_readfirstlane(int(uint32_t(sr)))));
    } else {
      row = rec;
    }
    if (row >= n_rows) row = -1;
    if (cen && row >= 0) {
      L = __builtin_amdgcn_readfirstlane(rec_list[rec]);
      if (L < 0 || L >= nlist) row = -1;
    }
  }
  if (row < 0) return;   // no workgroup barriers below
  float *buf = lds + wid * dstride;
  const uint2 sm = lane_sign_masks(rp, lane);
  const SignWords s1 = sign_words(rp.passes > 0 ? sm.x : 0u), s2 = sign_words(sm.y);

  // residual r = x - c, its sums, and S1
  const float *xr = x + row * D;
  const float *cr = (L >= 0) ? cen + int64_t(L) * D : xr;   // branch-free: weight 0 without c
  const float cw = (L >= 0) ? 1.f : 0.f;
  const bool has_rc = L >= 0 && cen_rot;
  const float *rcr = has_rc ? cen_rot + int64_t(L) * D : xr;
  const float rcw = has_rc ? 1.f : 0.f;
  float z[J], rc[J];
  float xx = 0.f, rr = 0.f, cc = 0.f;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const float xv = xr[lane + 64 * j];
    const float cv = cr[lane + 64 * j] * cw;
    rc[j] = rcr[lane + 64 * j] * rcw;
    const float r = xv - cv;
    xx += xv * xv;
    rr += r * r;
    cc += cv * cv;
    z[j] = flipw(r, s1, j);
  }
  rotate_fwd_reg<J>(z, rp, ts, s2, buf, lane);

  // EVT scale and 1-D Lloyd-Max codes
  float m = 0.f;
#pragma unroll
  for (int j = 0; j < J; ++j) m = fmaxf(m, fabsf(z[j]));
  m = wave_max(m);
  const float inv_s0 = (m > 0.f) ? cp.emax / m : 0.f;
  // Nearest centroid of the sorted 1-D codebook = number of thresholds below
  // u, by an unrolled binary search over the sorted thresholds; c4 is 4 x the
  // code (the byte offset of its centroid and thresholds in LDS).
  uint32_t c4[J];
#pragma unroll
  for (int j = 0; j < J; ++j) c4[j] = 0u;
#pragma unroll
  for (int half = K >> 1; half >= 1; half >>= 1) {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const float u = z[j] * inv_s0;
      c4[j] += (u > lds_at(thr, c4[j] + 4u * (half - 1))) ? 4u * half : 0u;
    }
  }
  float cv[J];
  float cn2 = 0.f, rcd = 0.f;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    c4[j] = (m > 0.f) ? c4[j] : 0u;
    cv[j] = (m > 0.f) ? lds_at(cbs, c4[j]) : 0.f;
    cn2 += cv[j] * cv[j];
    rcd += rc[j] * cv[j];
  }
  xx = wave_sum(xx);
  rr = wave_sum(rr);
  cc = wave_sum(cc);
  cn2 = wave_sum(cn2);
  rcd = wave_sum(rcd);
  const float s = (m > 0.f && cn2 > 0.f) ? sqrtf(rr / cn2) : 0.f;
  const uint32_t su = enc_ue7m9(s);
  const float sh = dec_ue7m9(su);
  uint32_t gu = 0x7000u;
  if (cp.global) {
    const float den2 = cc + 2.f * sh * rcd + sh * sh * cn2;
    const float gv = (den2 > 0.f) ? sqrtf(xx / den2) : 0.f;
    gu = enc_ue4m12(gv);
  }
  if (lane == 0) scales[rec] = su | (gu << 16);

  // pack: group G = 8 j + lane / 8 holds the codes of lanes 8 (lane / 8) .. + 7
#pragma unroll
  for (int j = 0; j < J; ++j) {
    uint32_t val = (c4[j] >> 2) << (BITS * (lane & 7));
    val |= __shfl_xor(val, 1, 64);
    val |= __shfl_xor(val, 2, 64);
    val |= __shfl_xor(val, 4, 64);
    if ((lane & 7) == 0) {
      const int G = 8 * j + (lane >> 3);
      if (BITS == 4) {
        *reinterpret_cast<uint32_t *>(codes + tile_addr_r(rec, G, 0, cp)) = val;
      } else {
        for (int t = 0; t < 3; ++t) codes[tile_addr_r(rec, G, t, cp)] = uint8_t(val >> (8 * t));
      }
    }
  }
  // padding groups of the tile layout (d_pad > D) carry code 0
  for (int G = (D >> 3) + lane; G < (cp.d_pad >> 3); G += 64) {
    if (BITS == 4) *reinterpret_cast<uint32_t *>(codes + tile_addr_r(rec, G, 0, cp)) = 0u;
    else for (int t = 0; t < 3; ++t) codes[tile_addr_r(rec, G, t, cp)] = 0;
  }
  if (resid) {
    const float gh = dec_ue4m12(gu);
    float *out = resid + row * D;   // indexed by source row
#pragma unroll
    for (int j = 0; j < J; ++j) out[lane + 64 * j] = z[j] + rc[j] - gh * (rc[j] + sh * cv[j]);
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
    default: return false;        \
  }

bool reg_path_ok(const RotParams &rp) {
  if (rp.B != 128 || rp.overlap || rp.D % 128) return false;
  const int nb = rp.D / 128;
  return nb == 1 || nb == 2 || nb == 3 || nb == 4 || nb == 6 || nb == 8;
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

bool launch_encode_reg(const rslm_plan *p, const float *x, int64_t n_rows, const int64_t *src_row,
                       const int32_t *rec_list, int64_t n_records, const float *cen,
                       const float *cen_rot, int nlist, uint8_t *codes, uint32_t *scales,
                       float *resid, hipStream_t s) {
  if (!reg_path_ok(p->rot) || p->codec.g != 1) return false;
  const int dstride = reg_dstride(p->rot.D);
  const int waves = 4;
  const size_t shm = size_t(waves) * dstride * sizeof(float);
  const unsigned grid = unsigned((n_records + waves - 1) / waves);
#define CALL_B(J, B)                                                                           \
  hipLaunchKernelGGL((k_encode_reg<J, B>), dim3(grid), dim3(64 * waves), shm, s, x, n_rows,       \
                     src_row, rec_list, n_records, cen, cen_rot, nlist, codes, scales, resid,       \
                     p->rot, p->codec, dstride)
#define CALL(J)          \
  if (p->codec.bits == 4) \
    CALL_B(J, 4);         \
  else                    \
    CALL_B(J, 3)
  RSLM_REG_SWITCH(p->rot.D / 128, CALL)
#undef CALL
#undef CALL_B
  return true;
}

}  // namespace rslm
