// Internal definitions of librslm: the plan object, launch helpers and small
// device utilities shared by the kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/rslm.h"

namespace rslm {

constexpr int kWave = 64;
constexpr int kTileRecords = 16;        // records per scan tile (MFMA N)
constexpr int kMaxDim = 4096;
constexpr int kMaxK = 1024;             // top-k bound
constexpr int kMaxNprobe = 1024;

// Per-plan parameters needed on the device, passed by value to kernels.
struct RotParams {
  int D;          // dimension
  int B;          // FWHT block size
  int logB;
  int n_full;     // floor(D / B)
  int overlap;    // 1 iff D % B != 0
  int passes;     // 0, 1, 2
  float inv_sqrt_b;
  const float *s1;     // device, 256 signs (+1/-1) as float
  const int16_t *pi;   // device, intra-block permutation of size B
  const int16_t *tsrc; // device, D entries: source of output o of the strided transpose
  uint32_t s1mask[8];  // bit i set <=> S1[i] = -1
};

// Sign bit of S1[j & 255] from the plan's mask with a branch-free select
// chain (the word index is per lane).
__device__ __forceinline__ uint32_t sign_bit(const uint32_t (&m)[8], int j) {
  j &= 255;
  const int w = j >> 5;
  uint32_t word = m[0];
#pragma unroll
  for (int i = 1; i < 8; ++i) word = (w == i) ? m[i] : word;
  return (word >> (j & 31)) & 1u;
}

// Per-lane sign masks for elements i = lane + 64 t: bit (t mod 4) of the
// first word is S1[i mod 256], of the second S2[i] = S1[(i + 127) mod 256]
// (the index pattern repeats every 4 steps of 64).
__device__ __forceinline__ uint2 lane_sign_masks(const RotParams &rp, int lane) {
  uint32_t a = 0, b = 0;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    a |= sign_bit(rp.s1mask, lane + 64 * t) << t;
    b |= sign_bit(rp.s1mask, lane + 64 * t + 127) << t;
  }
  return make_uint2(a, b);
}

__device__ __forceinline__ float flip(float v, uint32_t mask, int t) {
  return __uint_as_float(__float_as_uint(v) ^ (((mask >> (t & 3)) & 1u) << 31));
}

struct CodecParams {
  int D, bits, K, g, w;       // w = log2 K
  int n_sub;                  // ceil(D / g)
  int d_pad;                  // multiple of 32
  int n_chunks;               // d_pad / 32
  int lane_bytes;             // bytes of one lane's stream in a tile
  int tile_bytes;             // 64 * lane_bytes
  int canon_bytes;
  int global;                 // scale mode
  float emax;                 // E_max(D) as float
  float cb[64];               // codebook, K*g values
  float thr[16];              // 1-D decision thresholds (K-1 used)
  float cbh[16];              // |C_k|^2 / 2 (unused k: a huge value)
  int lead;                   // Rslm4Lite: leading coordinates on cb_lead (16 or 32), else 0
  int record_bytes;           // packed record: canon_bytes + scale suffix (Lite: none)
  float cb_lead[8];           // Rslm4Lite: K = 8 codebook of the leading coordinates
  float thr_lead[16];         // its 7 thresholds, padded with +inf
  // 1-D quantiser grids (quant_bucket) over the thresholds of cb / cb_lead:
  // each bucket holds at most one threshold; qn = 0: no such grid
  float qs, qo, qs_lead, qo_lead;
  int qn, qn_lead;
  // 2-D codebooks: a kGrid2 x kGrid2 grid of cells over [-emax, emax]^2
  // (cell of u: floor(clamp(u_d g2s + g2o, 0, kGrid2 - 1)) per coordinate),
  // each cell listing, in ascending order, at most four codes that can be
  // nearest to some point of it (4 bits each, the last repeated); g2tab is
  // device memory of the plan, null when some cell needs more than four
  float g2s, g2o;
  const uint16_t *g2tab;
};

constexpr int kGrid2 = RSLM_GRID2;

// Bucket of u on a uniform grid of qn buckets: floor(clamp(u qs + qo, 0,
// qn - 1)), one fused multiply-add.  Non-decreasing in u, so with at most one
// decision threshold per bucket the number of thresholds below u is the
// number whose bucket is lower, plus one comparison with the next threshold.
// The plan (host) and the encoders (device) evaluate the same expression.
__host__ __device__ inline int quant_bucket(float u, float qs, float qo, int qn) {
#if defined(__HIP_DEVICE_COMPILE__)
  // the same clamp as one median-of-three (equal for every non-NaN value; a
  // NaN bucket is one of the bounds or converts to 0)
  return int(__builtin_amdgcn_fmed3f(fmaf(u, qs, qo), 0.0f, float(qn - 1)));
#else
  return int(fminf(fmaxf(fmaf(u, qs, qo), 0.0f), float(qn - 1)));
#endif
}

}  // namespace rslm

struct rslm_plan {
  int device;
  rslm::RotParams rot;
  rslm::CodecParams codec;
  double emax;
  int8_t signs[256];
  int32_t perm[128];
  // device allocations owned by the plan
  float *d_s1 = nullptr;
  int16_t *d_pi = nullptr;
  int16_t *d_tsrc = nullptr;
  uint32_t *d_dtab = nullptr;   // compact decode table (see scan.hip)
  uint16_t *d_g2tab = nullptr;  // candidate lists of the 2-D nearest-centroid grid
  int dtab_entries = 0;
  int dtab_words = 0;           // 32-bit words per entry
};

namespace rslm {

int set_hip_error(hipError_t e);     // records e, returns RSLM_ERR_HIP
int check_launch();                  // hipGetLastError -> status
bool device_ok();                    // current device is gfx950

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

// Register-resident rotation / 1-D encoder for D = 128 NB (rotate_reg.hip);
// false when the plan is not handled there.
bool launch_rotate_reg(const rslm_plan *p, const float *x, float *y, int64_t n, int inverse,
                       hipStream_t s);
// Optional second output: the RSLM rescoring stage of rslm_encode_two_stage
// (p2, codes2, scales2), or the SQ8 codes of rslm_encode_sq8 (sq8_lo,
// sq8_hi, codes2); neither: p2 == nullptr and sq8_lo == nullptr.
bool launch_encode_reg(const rslm_plan *p, const rslm_plan *p2, const float *x, int64_t n_rows,
                       const int64_t *src_row, const int32_t *rec_list, int64_t n_records,
                       const float *cen, const float *cen_rot, int nlist, uint8_t *codes,
                       uint32_t *scales, float *resid, uint8_t *codes2, uint32_t *scales2,
                       const float *sq8_lo, const float *sq8_hi, hipStream_t s);

// ---- device helpers ------------------------------------------------------

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// UE7M9: u = e << 9 | m encodes 2^(e-63) (1 + m/512), e in [1,127]; u = 0 is 0.
// Round to nearest even on 10 significant bits from float32, saturate on
// overflow, flush values below 2^-62 to 0.
__device__ __forceinline__ uint32_t enc_ue7m9(float s) {
  if (!(s > 0.0f)) return 0u;
  uint32_t b = __float_as_uint(s);
  if (b >= 0x7f800000u) return (127u << 9) | 511u;
  b += 0x1fffu + ((b >> 14) & 1u);
  b >>= 14;                             // (fp32 exponent << 9) | mantissa9
  int e = int(b >> 9) - 64;
  if (e < 1) return 0u;
  if (e > 127) return (127u << 9) | 511u;
  return (uint32_t(e) << 9) | (b & 511u);
}

__device__ __forceinline__ float dec_ue7m9(uint32_t u) {
  return u ? __uint_as_float((u << 14) + (64u << 23)) : 0.0f;
}

// UE4M12: u = e << 12 | m encodes 2^(e-7) (1 + m/4096), e in [1,15].
__device__ __forceinline__ uint32_t enc_ue4m12(float s) {
  if (!(s > 0.0f)) return 0u;
  uint32_t b = __float_as_uint(s);
  if (b >= 0x7f800000u) return (15u << 12) | 4095u;
  b += 0x3ffu + ((b >> 11) & 1u);
  b >>= 11;
  int e = int(b >> 12) - 120;
  if (e < 1) return 0u;
  if (e > 15) return (15u << 12) | 4095u;
  return (uint32_t(e) << 12) | (b & 4095u);
}

__device__ __forceinline__ float dec_ue4m12(uint32_t u) {
  return u ? __uint_as_float((u << 11) + (120u << 23)) : 0.0f;
}

// SQ8 code of v for the range [lo, hi]: clamp(rne((v - lo) / step), 0, 255)
// with step = (hi - lo) / 255, evaluated as (v - lo) * inv, inv = 255 / (hi -
// lo) with the hardware reciprocal (1 ulp); an empty range has inv = 0, which
// gives code 0 (a NaN product is clamped to 0 as well).  Encoders that code
// many rows against the same ranges compute inv once per coordinate.
__device__ __forceinline__ float sq8_inv(float lo, float hi) {
  const float w = hi - lo;
  return (w > 0.0f) ? __builtin_amdgcn_rcpf(w) * 255.0f : 0.0f;
}
__device__ __forceinline__ uint32_t sq8_code_inv(float v, float lo, float inv) {
  return uint32_t(fminf(fmaxf(rintf((v - lo) * inv), 0.0f), 255.0f));
}
__device__ __forceinline__ uint32_t sq8_code(float v, float lo, float hi) {
  return sq8_code_inv(v, lo, sq8_inv(lo, hi));
}
// sq8_code_inv(v, lo, inv) written into byte t of w, the other bytes kept:
// v_cvt_pk_u8_f32 rounds to nearest even and saturates to [0, 255] (NaN gives
// 0), the rounding and clamp above in one instruction.
__device__ __forceinline__ uint32_t sq8_code_put(uint32_t w, float v, float lo, float inv, int t) {
  return __builtin_amdgcn_cvt_pk_u8_f32((v - lo) * inv, uint32_t(t), w);
}

// Float -> uint32 whose unsigned order equals the float order.
__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float key_to_float(uint32_t k) {
  uint32_t b = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return __uint_as_float(b);
}

}  // namespace rslm
