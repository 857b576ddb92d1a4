// Block-wise cascaded Walsh-Hadamard rotation and the fused RSLM encoder.
//
// Rotation (paper, Section "Pre-Quantization Transformations"): signs S1,
// orthonormal FWHT on blocks of B (full blocks, then one block overlapping
// the previous one and ending at D), then for two passes the in-block
// permutation with the strided transpose x'[k M + b] = x[b B + P(k)], signs
// S2 = S1 offset by 127, and the block FWHT again.
//
// GPU mapping: one wavefront per vector; the vector lives in LDS and each
// radix-8 round loads 8 elements per lane, runs three butterfly stages in
// registers and stores them back, so a 128-block needs three LDS round
// trips (3 + 3 + 1 stages).  The encoder fuses residual, rotation, EVT
// scale, Lloyd-Max assignment, norm correction, both 16-bit scales, packing
// into the scan tile layout and the rotated second residual.
#include "rslm_internal.h"

namespace rslm {

// LDS index of vector element i: one pad word per 32 elements so that the
// strided butterfly accesses of a round fall into distinct banks.
__device__ __forceinline__ int px(int i) { return i + (i >> 5); }
__host__ __device__ constexpr int padded_len(int n) { return n + (n >> 5) + 1; }

// Each wavefront owns its vector, and LDS operations of one wavefront take
// effect in issue order, so a wavefront-scope fence (a compiler ordering
// point) is all the synchronisation the rotation needs.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// W: lanes per vector (the encoder gives small vectors fewer lanes); lane is
// the lane's index among them.
template <int R, int W = kWave>
__device__ __forceinline__ void fwht_round(float *v, int off, int nblk, int B, int logB, int s,
                                           bool last, float scale, int lane) {
  constexpr int G = 1 << R;
  const int h = 1 << s;
  const int lg = logB - R;   // groups per block: 2^lg
  const int total = nblk << lg;
  for (int gi = lane; gi < total; gi += W) {
    const int blk = gi >> lg;
    const int t = gi & ((1 << lg) - 1);
    const int low = t & (h - 1);
    const int high = t >> s;
    const int base = off + blk * B + ((high << (s + R)) | low);
    float e[G];
#pragma unroll
    for (int m = 0; m < G; ++m) e[m] = v[px(base + m * h)];
#pragma unroll
    for (int st = 0; st < R; ++st) {
#pragma unroll
      for (int m = 0; m < G; ++m) {
        if (!(m & (1 << st))) {
          const float a = e[m], b = e[m | (1 << st)];
          e[m] = a + b;
          e[m | (1 << st)] = a - b;
        }
      }
    }
    if (last) {
#pragma unroll
      for (int m = 0; m < G; ++m) e[m] *= scale;
    }
#pragma unroll
    for (int m = 0; m < G; ++m) v[px(base + m * h)] = e[m];
  }
}

// Orthonormal FWHT of nblk adjacent blocks of size B starting at off, by the
// calling wavefront.
template <int W = kWave>
__device__ __forceinline__ void fwht_blocks(float *v, int off, int nblk, const RotParams &rp,
                                            int lane) {
  const int B = rp.B, logB = rp.logB;
  if (logB == 0) return;  // B == 1: identity
  for (int s = 0; s < logB; s += 3) {
    const int R = (logB - s) < 3 ? (logB - s) : 3;
    const bool last = (s + R) == logB;
    if (R == 3) fwht_round<3, W>(v, off, nblk, B, logB, s, last, rp.inv_sqrt_b, lane);
    else if (R == 2) fwht_round<2, W>(v, off, nblk, B, logB, s, last, rp.inv_sqrt_b, lane);
    else fwht_round<1, W>(v, off, nblk, B, logB, s, last, rp.inv_sqrt_b, lane);
    wave_sync();
  }
}

// One pass of block transforms.  Forward: full blocks, then the overlap
// block.  Reverse (inverse rotation): overlap block first.
template <int W = kWave>
__device__ __forceinline__ void fwht_pass(float *v, const RotParams &rp, int lane, bool reverse) {
  if (!reverse) {
    if (rp.n_full) fwht_blocks<W>(v, 0, rp.n_full, rp, lane);
    if (rp.overlap) fwht_blocks<W>(v, rp.D - rp.B, 1, rp, lane);
  } else {
    if (rp.overlap) fwht_blocks<W>(v, rp.D - rp.B, 1, rp, lane);
    if (rp.n_full) fwht_blocks<W>(v, 0, rp.n_full, rp, lane);
  }
}

// Sign bits of the elements lane + W t of a vector spread over W lanes, bit t
// for t < 256 / W (the sign tables repeat every 256 coordinates); x: S1,
// y: S2 (S1 offset by 127).  W = 64 gives lane_sign_masks.
template <int W>
__device__ __forceinline__ uint2 sub_sign_masks(const RotParams &rp, int lane) {
  static_assert(W >= 8 && W <= kWave && 256 % W == 0, "lanes per vector");
  uint32_t a = 0, b = 0;
#pragma unroll
  for (int t = 0; t < 256 / W; ++t) {
    a |= sign_bit(rp.s1mask, lane + W * t) << t;
    b |= sign_bit(rp.s1mask, lane + W * t + 127) << t;
  }
  return make_uint2(a, b);
}
template <int W>
__device__ __forceinline__ float flip_w(float v, uint32_t mask, int t) {
  return __uint_as_float(__float_as_uint(v) ^ (((mask >> (t & (256 / W - 1))) & 1u) << 31));
}
// Sum / maximum over the W lanes of a vector (aligned groups of W lanes).
template <int W>
__device__ __forceinline__ float sub_sum(float v) {
#pragma unroll
  for (int off = W / 2; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}
template <int W>
__device__ __forceinline__ float sub_max(float v) {
#pragma unroll
  for (int off = W / 2; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// Source of output o of the strided transpose, (o mod M) B + P(o / M) below
// M B (M = n_full), o above: the plan's table of it (a division per element
// otherwise).
__device__ __forceinline__ int transpose_src(int o, const RotParams &rp) {
  return int(rp.tsrc[o]);
}

// Forward rotation of the vector held in v (already multiplied by S1 when
// passes > 0; element i at v[px(i)]).  Returns the buffer holding the result.
template <int W = kWave>
__device__ float *rotate_forward(float *v, float *w, const RotParams &rp,
                                 uint32_t s2bits, int lane) {
  if (rp.passes == 0) return v;
  fwht_pass<W>(v, rp, lane, false);
  if (rp.passes == 1) return v;
#pragma unroll 4
  for (int o = lane, t = 0; o < rp.D; o += W, ++t)
    w[px(o)] = flip_w<W>(v[px(transpose_src(o, rp))], s2bits, t);
  wave_sync();
  fwht_pass<W>(w, rp, lane, false);
  return w;
}

// Inverse rotation R^T of the vector in v; the result excludes the final S1
// multiplication, which the caller applies on output.
__device__ float *rotate_inverse(float *v, float *w, const RotParams &rp,
                                 uint32_t s2bits, int lane) {
  if (rp.passes == 0) return v;
  if (rp.passes == 1) {
    fwht_pass(v, rp, lane, true);
    return v;
  }
  fwht_pass(v, rp, lane, true);
#pragma unroll 4
  for (int o = lane, t = 0; o < rp.D; o += kWave, ++t)
    w[px(transpose_src(o, rp))] = flip(v[px(o)], s2bits, t);
  wave_sync();
  fwht_pass(w, rp, lane, true);
  return w;
}

// ---------------------------------------------------------------- rslm_fwht
__global__ void __launch_bounds__(256) k_rotate(const float *__restrict__ x, float *y, int64_t n,
                                                RotParams rp, int inverse, int dstride) {
  extern __shared__ float lds[];
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int64_t row = int64_t(blockIdx.x) * (blockDim.x >> 6) + wid;
  if (row >= n) return;   // no workgroup barriers below
  float *v = lds + wid * 2 * dstride;
  float *w = v + dstride;
  const int D = rp.D;
  const uint2 sm = lane_sign_masks(rp, lane);
  const uint32_t s1in = (!inverse && rp.passes > 0) ? sm.x : 0u;
  const uint32_t s1out = (inverse && rp.passes > 0) ? sm.x : 0u;
  const float *xr = x + row * D;
#pragma unroll 4
  for (int i = lane, t = 0; i < D; i += kWave, ++t) v[px(i)] = flip(xr[i], s1in, t);
  wave_sync();
  const float *res = inverse ? rotate_inverse(v, w, rp, sm.y, lane)
                             : rotate_forward(v, w, rp, sm.y, lane);
  float *yr = y + row * D;
#pragma unroll 4
  for (int i = lane, t = 0; i < D; i += kWave, ++t) yr[i] = flip(res[px(i)], s1out, t);
}

// --------------------------------------------------------------- rslm_encode
// Byte address inside the scan tile layout of the bits of coordinates
// [8G, 8G + 8) of record rec: the tile holds 16 records; lane l = r * 16 + n
// (n = record within the tile, r = G mod 4) owns a stream of lane_bytes
// bytes stored as 16-byte units interleaved across the 64 lanes; chunk
// c = G / 4 contributes `bits` bytes at stream offset c * bits.
__device__ __forceinline__ int64_t tile_byte_addr(int64_t rec, int G, int t, const CodecParams &cp) {
  const int64_t tile = rec >> 4;
  const int n = int(rec & 15);
  const int c = G >> 2, r = G & 3;
  const int lane_id = r * 16 + n;
  const int off = c * cp.bits + t;
  return tile * cp.tile_bytes + int64_t((off >> 4) * 64 + lane_id) * 16 + (off & 15);
}

__device__ __forceinline__ void store_group(uint8_t *codes, int64_t rec, int G, uint32_t val,
                                            const CodecParams &cp) {
  const int b = cp.bits;
  if (b == 4) {
    *reinterpret_cast<uint32_t *>(codes + tile_byte_addr(rec, G, 0, cp)) = val;
  } else if (b == 2) {
    *reinterpret_cast<uint16_t *>(codes + tile_byte_addr(rec, G, 0, cp)) = uint16_t(val);
  } else if (b == 1) {
    codes[tile_byte_addr(rec, G, 0, cp)] = uint8_t(val);
  } else {
    for (int t = 0; t < 3; ++t) codes[tile_byte_addr(rec, G, t, cp)] = uint8_t(val >> (8 * t));
  }
}

// Register rotation for D = 96 on 8 lanes per vector (the plan's blocks of 64:
// [0, 64) and the overlapping [32, 96)).  Lane l holds elements l + 8 t,
// t < 12, in e[t]; in a block starting at element 8 t0, bits 0-2 of the
// in-block index are the lane and bits 3-5 are t - t0.  The butterfly stages
// run in the order of the LDS rounds (bits 0, 1, 2, then 3, 4, 5; the scale
// last), so the results are those of the general path bit for bit.
template <int CTRL>
__device__ __forceinline__ float dpp8(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, true));
}
// value of lane l ^ m of the 8-lane group (quad_perm for m = 1, 2; for m = 4
// a half-row mirror, l ^ 7, then a quad reversal, ^ 3)
template <int M>
__device__ __forceinline__ float lane_xor8(float v) {
  if constexpr (M == 1) return dpp8<0xB1>(v);
  else if constexpr (M == 2) return dpp8<0x4E>(v);
  else return dpp8<0x1B>(dpp8<0x141>(v));
}
template <int M>
__device__ __forceinline__ void lane_stage8(float (&e)[12], int t0, int sl) {
  const float sg = (sl & M) ? -1.f : 1.f;   // upper lane: partner - own
#pragma unroll
  for (int k = 0; k < 8; ++k) e[t0 + k] = fmaf(e[t0 + k], sg, lane_xor8<M>(e[t0 + k]));
}
__device__ __forceinline__ void fwht64_r8(float (&e)[12], int t0, int sl, float scale) {
  lane_stage8<1>(e, t0, sl);
  lane_stage8<2>(e, t0, sl);
  lane_stage8<4>(e, t0, sl);
#pragma unroll
  for (int h = 1; h < 8; h <<= 1)
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (!(k & h)) {
        const float a = e[t0 + k], b = e[t0 + k + h];
        e[t0 + k] = a + b;
        e[t0 + k + h] = a - b;
      }
#pragma unroll
  for (int k = 0; k < 8; ++k) e[t0 + k] *= scale;
}

// VPW vectors per wavefront, W = 64 / VPW lanes each (small D: a wavefront
// per vector would leave most lanes idle in every butterfly round).
template <int VPW>
__global__ void __launch_bounds__(256) k_encode(
    const float *__restrict__ x, int64_t n_rows, const int64_t *__restrict__ src_row,
    const int32_t *__restrict__ rec_list, int64_t n_records, const float *__restrict__ cen,
    const float *__restrict__ cen_rot, int nlist, uint8_t *__restrict__ codes,
    uint32_t *__restrict__ scales, float *__restrict__ resid, RotParams rp, CodecParams cp,
    int dstride, uint8_t *__restrict__ codes2, uint32_t *__restrict__ scales2,
    CodecParams cp2, const float *__restrict__ sq8_lo, const float *__restrict__ sq8_hi) {
  extern __shared__ float lds[];
  __shared__ float cbs[64], cbs2[64], cbl[8];
  // 1-D quantiser grid (cp.qn > 0): thresholds below each bucket, and the
  // sorted thresholds padded with +inf
  __shared__ uint8_t qtab[512];
  __shared__ float thr_s[16];
  constexpr int W = kWave / VPW;
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const int sl = lane & (W - 1);            // lane within the vector's W lanes
  const int vid = wid * VPW + lane / W;     // vector slot of the workgroup
  const int nv = nw * VPW;
  if (threadIdx.x < 64) {
    cbs[threadIdx.x] = cp.cb[threadIdx.x];
    cbs2[threadIdx.x] = cp2.cb[threadIdx.x];
  }
  if (threadIdx.x < 8) cbl[threadIdx.x] = cp.cb_lead[threadIdx.x];
  if (cp.g == 1 && cp.qn > 0) {
    if (threadIdx.x < 16)
      thr_s[threadIdx.x] = (int(threadIdx.x) + 1 < cp.K) ? cp.thr[threadIdx.x] : __builtin_inff();
    for (int j = threadIdx.x; j < cp.qn; j += blockDim.x) {
      int cnt = 0;
      for (int k = 0; k + 1 < cp.K; ++k) cnt += quant_bucket(cp.thr[k], cp.qs, cp.qo, cp.qn) < j;
      qtab[j] = uint8_t(cnt);
    }
  }
  __syncthreads();   // publishes the tables above
  const int64_t rec = int64_t(blockIdx.x) * nv + vid;
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
  // no workgroup barriers below; the W lanes of a vector leave together and
  // never exchange data with another vector's lanes
  if (row < 0) return;
  float *v = lds + vid * 2 * dstride;
  float *w = v + dstride;
  uint8_t *cl = reinterpret_cast<uint8_t *>(lds + nv * 2 * dstride) + vid * dstride;
  // second-stage codes follow the first-stage ones (allocated only with codes2)
  uint8_t *cl2 = reinterpret_cast<uint8_t *>(lds + nv * 2 * dstride) + (nv + vid) * dstride;
  const int D = rp.D;
  float xx = 0.f, rr = 0.f, cc = 0.f;
  const uint2 sm = sub_sign_masks<W>(rp, sl);
  const uint32_t s1in = (rp.passes > 0) ? sm.x : 0u;
  const float *xr = x + row * D;
  // branch-free loads: without a centre read x's row and weight it by 0
  const float *cr = (L >= 0) ? cen + int64_t(L) * D : xr;
  const float cw = (L >= 0) ? 1.f : 0.f;
  const float *z = v;
  bool rotated = false;
  if constexpr (W == 8) {
    if (D == 96 && rp.B == 64 && rp.passes == 2) {
      // residual and both passes in registers; the transpose through v
      float e[12];
#pragma unroll
      for (int t = 0; t < 12; ++t) {
        const int i = sl + 8 * t;
        const float xv = xr[i];
        const float cv = cr[i] * cw;
        const float r = xv - cv;
        xx += xv * xv;
        rr += r * r;
        cc += cv * cv;
        e[t] = flip_w<W>(r, s1in, t);
      }
      fwht64_r8(e, 0, sl, rp.inv_sqrt_b);
      fwht64_r8(e, 4, sl, rp.inv_sqrt_b);
#pragma unroll
      for (int t = 0; t < 12; ++t) v[px(sl + 8 * t)] = e[t];
      wave_sync();
#pragma unroll
      for (int t = 0; t < 12; ++t) e[t] = flip_w<W>(v[px(transpose_src(sl + 8 * t, rp))], sm.y, t);
      fwht64_r8(e, 0, sl, rp.inv_sqrt_b);
      fwht64_r8(e, 4, sl, rp.inv_sqrt_b);
#pragma unroll
      for (int t = 0; t < 12; ++t) w[px(sl + 8 * t)] = e[t];
      wave_sync();
      z = w;
      rotated = true;
    }
  }
  if (!rotated) {
  #pragma unroll 4
    for (int i = sl, t = 0; i < D; i += W, ++t) {
      const float xv = xr[i];
      const float cv = cr[i] * cw;
      const float r = xv - cv;
      xx += xv * xv;
      rr += r * r;
      cc += cv * cv;
      v[px(i)] = flip_w<W>(r, s1in, t);
    }
    wave_sync();
    z = rotate_forward<W>(v, w, rp, sm.y, sl);
  }

  float m = 0.f;
#pragma unroll 4
  for (int i = sl; i < D; i += W) m = fmaxf(m, fabsf(z[px(i)]));
  m = sub_max<W>(m);
  const float inv_s0 = (m > 0.f) ? cp.emax / m : 0.f;
  const bool has_rc = L >= 0 && cen_rot;
  const float *rc = has_rc ? cen_rot + int64_t(L) * D : x + row * D;   // any valid row
  const float rcw = has_rc ? 1.f : 0.f;
  const int g = cp.g;
  float cn2 = 0.f, rcd = 0.f;
#pragma unroll 4
  for (int j = sl; j < cp.n_sub; j += W) {
    int code = 0;
    if (m > 0.f) {
      if (g == 1 && j < cp.lead) {   // Rslm4Lite leading coordinate: K = 8
        const float u = z[px(j)] * inv_s0;
#pragma unroll
        for (int k = 0; k < 7; ++k) code += (u > cp.thr_lead[k]) ? 1 : 0;
      } else if (g == 1 && cp.qn > 0) {
        // thresholds below u's bucket, plus one comparison with the next
        // threshold (the grid has at most one per bucket): the same count
        // as comparing u with every threshold
        const float u = z[px(j)] * inv_s0;
        const int base = qtab[quant_bucket(u, cp.qs, cp.qo, cp.qn)];
        code = base + ((u > thr_s[base]) ? 1 : 0);
      } else if (g == 1) {
        const float u = z[px(j)] * inv_s0;
#pragma unroll
        for (int k = 0; k < 15; ++k) code += (k + 1 < cp.K && u > cp.thr[k]) ? 1 : 0;
      } else {
        float u[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int i = j * g + t;
          u[t] = (t < g && i < D) ? z[px(i)] * inv_s0 : 0.f;
        }
        float best = 3.4e38f;
        for (int k = 0; k < 16; ++k) {
          float d = 0.f;
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            if (t < g) {
              const float e = u[t] - cp.cb[k * g + t];
              d += e * e;
            }
          }
          if (d < best) {
            best = d;
            code = k;
          }
        }
      }
      for (int t = 0; t < g; ++t) {
        const int i = j * g + t;
        const float cv = (i < D) ? ((i < cp.lead) ? cbl[code] : cbs[code * g + t]) : 0.f;
        cn2 += cv * cv;
        rcd += rc[i < D ? i : 0] * rcw * cv;
      }
    }
    cl[j] = uint8_t(code);
  }
  xx = sub_sum<W>(xx);
  rr = sub_sum<W>(rr);
  cc = sub_sum<W>(cc);
  cn2 = sub_sum<W>(cn2);
  rcd = sub_sum<W>(rcd);
  const float s = (m > 0.f && cn2 > 0.f) ? sqrtf(rr / cn2) : 0.f;
  const uint32_t su = enc_ue7m9(s);
  const float sh = dec_ue7m9(su);
  uint32_t gu = 0x7000u;
  const float den2 = cc + 2.f * sh * rcd + sh * sh * cn2;   // ||c + R^T s^ c^||^2
  if (cp.global) {
    const float gv = (den2 > 0.f) ? sqrtf(xx / den2) : 0.f;
    gu = enc_ue4m12(gv);
  }
  if (sl == 0) scales[rec] = su | (gu << 16);
  __builtin_amdgcn_wave_barrier();  // codes in cl are written by other lanes
  // first-stage centroid value of valid coordinate i (0 for a zero residual)
  const int lg = g >> 1;   // log2 g: sub-vectors of 1, 2 or 4 coordinates
  auto cval = [&](int i) {
    if (!(m > 0.f)) return 0.f;
    return (i < cp.lead) ? cbl[cl[i]] : cbs[cl[i >> lg] * g + (i & (g - 1))];
  };

  if (codes2 && !sq8_lo) {
    // Second stage: r2 = R x - R a with R a = g^ (R c + s^ c^), quantised in
    // the rotated space with the second codebook (no further rotation).
    const float gh = dec_ue4m12(gu);
    float *r2 = (z == v) ? w : v;   // the buffer the rotation left free
    float m2 = 0.f, rr2 = 0.f;
#pragma unroll 4
    for (int i = sl; i < D; i += W) {
      const float cv = cval(i);
      const float rcv = rc[i] * rcw;
      const float d = z[px(i)] + rcv - gh * (rcv + sh * cv);
      r2[px(i)] = d;
      m2 = fmaxf(m2, fabsf(d));
      rr2 += d * d;
    }
    wave_sync();
    m2 = sub_max<W>(m2);
    rr2 = sub_sum<W>(rr2);
    const float inv2 = (m2 > 0.f) ? cp2.emax / m2 : 0.f;
    const int g2 = cp2.g;
    float cn22 = 0.f, rad = 0.f;   // ||c2^||^2 and <R a, c2^> / g^
#pragma unroll 2
    for (int j = sl; j < cp2.n_sub; j += W) {
      int code = 0;
      if (m2 > 0.f) {
        if (g2 == 1) {
          const float u = r2[px(j)] * inv2;
#pragma unroll
          for (int k = 0; k < 15; ++k) code += (k + 1 < cp2.K && u > cp2.thr[k]) ? 1 : 0;
        } else {
          float u[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const int i = j * g2 + t;
            u[t] = (t < g2 && i < D) ? r2[px(i)] * inv2 : 0.f;
          }
          float best = 3.4e38f;
          for (int k = 0; k < 16; ++k) {
            float d = 0.f;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              if (t < g2) {
                const float e = u[t] - cbs2[k * g2 + t];
                d += e * e;
              }
            }
            if (d < best) {
              best = d;
              code = k;
            }
          }
        }
        for (int t = 0; t < g2; ++t) {
          const int i = j * g2 + t;
          if (i >= D) break;
          const float c2 = cbs2[code * g2 + t];
          const float c1 = cval(i);
          cn22 += c2 * c2;
          rad += (rc[i] * rcw + sh * c1) * c2;
        }
      }
      cl2[j] = uint8_t(code);
    }
    cn22 = sub_sum<W>(cn22);
    rad = sub_sum<W>(rad) * gh;
    const float s2 = (m2 > 0.f && cn22 > 0.f) ? sqrtf(rr2 / cn22) : 0.f;
    const uint32_t su2 = enc_ue7m9(s2);
    const float sh2 = dec_ue7m9(su2);
    uint32_t gu2 = 0x7000u;
    if (cp2.global) {
      const float dd = gh * gh * den2 + 2.f * sh2 * rad + sh2 * sh2 * cn22;
      gu2 = enc_ue4m12((dd > 0.f) ? sqrtf(xx / dd) : 0.f);
    }
    if (sl == 0) scales2[row] = su2 | (gu2 << 16);
    __builtin_amdgcn_wave_barrier();   // cl2 is written by other lanes
    // canonical bit stream: code j at bits [w j, w j + w)
    uint8_t *dst = codes2 + row * int64_t(cp2.canon_bytes);
    const int w2 = cp2.w;
    for (int t = sl; t < cp2.canon_bytes; t += W) {
      uint32_t val = 0;
      for (int b = 0; b < 8; ++b) {
        const int p = 8 * t + b;
        const int j = p / w2;
        if (j < cp2.n_sub) val |= ((uint32_t(cl2[j]) >> (p - j * w2)) & 1u) << b;
      }
      dst[t] = uint8_t(val);
    }
  }

  // pack: group G covers coordinates [8G, 8G + 8) = sub-vectors [8G/g, 8G/g + 8/g)
  const int n_groups = cp.d_pad >> 3;
  const int per = 8 / g;
  for (int G = sl; G < n_groups; G += W) {
    uint32_t val = 0;
    for (int t = 0; t < per; ++t) {
      const int j = G * per + t;
      uint32_t code = (j < cp.n_sub) ? cl[j] : 0u;
      if (j < cp.lead) code |= (((j < 16 ? su : gu) >> (j & 15)) & 1u) << 3;   // Rslm4Lite
      val |= code << (cp.w * t);
    }
    store_group(codes, rec, G, val, cp);
  }
  if (resid || sq8_lo) {
    // the rotated second residual, as floats and / or as SQ8 codes (the
    // rslm_sq8_encode arithmetic), both indexed by source row
    const float gh = dec_ue4m12(gu);
  #pragma unroll 4
    for (int i = sl; i < D; i += W) {
      const float cv = cval(i);
      const float rcv = rc[i] * rcw;
      const float o = z[px(i)] + rcv - gh * (rcv + sh * cv);
      if (resid) resid[row * D + i] = o;
      if (sq8_lo)
        codes2[row * D + i] = uint8_t(sq8_code_put(0u, o, sq8_lo[i], sq8_inv(sq8_lo[i], sq8_hi[i]), 0));
    }
  }
}

// --------------------------------------------------------------- rslm_decode
// Decompress: x~ = g^ (c + R^T s^ C[code]) per record, one wavefront per
// record through LDS: the decoded rotated residual s^ C[code] is placed in
// the vector buffer, rotated back (blocks in reverse, inverse transpose, S1
// last) and scaled.
__global__ void __launch_bounds__(256) k_decode(const uint8_t *__restrict__ codes,
                                                const uint32_t *__restrict__ scales, int64_t n,
                                                const int32_t *__restrict__ rec_list,
                                                const float *__restrict__ cen, int nlist,
                                                float *__restrict__ out, RotParams rp,
                                                CodecParams cp, int dstride) {
  extern __shared__ float lds[];
  __shared__ float cbs[64], cbl[8];
  if (threadIdx.x < 64) cbs[threadIdx.x] = cp.cb[threadIdx.x];
  if (threadIdx.x < 8) cbl[threadIdx.x] = cp.cb_lead[threadIdx.x];
  __syncthreads();   // publishes cbs / cbl
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int64_t rec = int64_t(blockIdx.x) * (blockDim.x >> 6) + wid;
  if (rec >= n) return;   // no workgroup barriers below
  float *v = lds + wid * 2 * dstride;
  float *w = v + dstride;
  const int D = rp.D, g = cp.g;
  const uint32_t sc = scales[rec];
  const float sh = dec_ue7m9(sc & 0xffffu);
  const float gh = cp.global ? dec_ue4m12(sc >> 16) : 1.f;
  int L = -1;
  if (cen) {
    L = rec_list[rec];
    if (L < 0 || L >= nlist) L = -1;
  }
  const int per = 8 / g;   // sub-vectors per group of 8 coordinates
  const int lg = g >> 1;   // log2 g: sub-vectors of 1, 2 or 4 coordinates
#pragma unroll 4
  for (int i = lane; i < D; i += kWave) {
    const int j = i >> lg;           // sub-vector
    const int G = i >> 3;            // group of 8 coordinates
    uint32_t bits = 0;
    for (int b = 0; b < cp.bits; ++b) bits |= uint32_t(codes[tile_byte_addr(rec, G, b, cp)]) << (8 * b);
    const uint32_t code = (bits >> (cp.w * (j - G * per))) & ((1u << cp.w) - 1u);
    const float c = (j < cp.lead) ? cbl[code & 7u] : cbs[code * g + (i & (g - 1))];
    v[px(i)] = sh * c;
  }
  wave_sync();
  const uint2 sm = lane_sign_masks(rp, lane);
  const uint32_t s1out = (rp.passes > 0) ? sm.x : 0u;
  const float *res = rotate_inverse(v, w, rp, sm.y, lane);
  const float *cr = (L >= 0) ? cen + int64_t(L) * D : nullptr;
  float *orow = out + rec * D;
#pragma unroll 4
  for (int i = lane, t = 0; i < D; i += kWave, ++t) {
    const float base = cr ? cr[i] : 0.f;
    orow[i] = gh * (base + flip(res[px(i)], s1out, t));
  }
}

// --------------------------------------------------------- pack / unpack
// Group G of a record is the `bits` canonical bytes [G bits, G bits + bits).
__global__ void k_pack(const uint8_t *__restrict__ canon, int64_t n, uint8_t *__restrict__ tiles,
                       CodecParams cp) {
  const int n_groups = cp.d_pad >> 3;
  const int64_t total = ((n + 15) >> 4) * 16 * n_groups;
  for (int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; t < total;
       t += int64_t(gridDim.x) * blockDim.x) {
    const int64_t rec = t / n_groups;
    const int G = int(t - rec * n_groups);
    for (int b = 0; b < cp.bits; ++b) {
      const int cb = G * cp.bits + b;
      tiles[tile_byte_addr(rec, G, b, cp)] =
          (rec < n && cb < cp.canon_bytes) ? canon[rec * cp.canon_bytes + cb] : uint8_t(0);
    }
  }
}

__global__ void k_unpack(const uint8_t *__restrict__ tiles, int64_t n, uint8_t *__restrict__ canon,
                         CodecParams cp) {
  const int n_groups = cp.d_pad >> 3;
  const int64_t total = n * n_groups;
  for (int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; t < total;
       t += int64_t(gridDim.x) * blockDim.x) {
    const int64_t rec = t / n_groups;
    const int G = int(t - rec * n_groups);
    for (int b = 0; b < cp.bits; ++b) {
      const int cb = G * cp.bits + b;
      if (cb < cp.canon_bytes) canon[rec * cp.canon_bytes + cb] = tiles[tile_byte_addr(rec, G, b, cp)];
    }
  }
}

// Packed records (canonical codes + scale suffix, or Lite codes alone) from
// the scan tile layout and the scales array.  Thread per (record, group of 8
// coordinates); group 0 also writes the suffix.
__global__ void k_pack_records(const uint8_t *__restrict__ tiles, const uint32_t *__restrict__ scales,
                               int64_t n, uint8_t *__restrict__ records, CodecParams cp) {
  const int n_groups = cp.d_pad >> 3;
  const int64_t total = n * n_groups;
  for (int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; t < total;
       t += int64_t(gridDim.x) * blockDim.x) {
    const int64_t rec = t / n_groups;
    const int G = int(t - rec * n_groups);
    uint8_t *dst = records + rec * cp.record_bytes;
    for (int b = 0; b < cp.bits; ++b) {
      const int cb = G * cp.bits + b;
      if (cb < cp.canon_bytes) dst[cb] = tiles[tile_byte_addr(rec, G, b, cp)];
    }
    if (G == 0 && cp.lead == 0) {
      const uint32_t sc = scales[rec];
      dst[cp.canon_bytes] = uint8_t(sc);
      dst[cp.canon_bytes + 1] = uint8_t(sc >> 8);
      if (cp.global) {
        dst[cp.canon_bytes + 2] = uint8_t(sc >> 16);
        dst[cp.canon_bytes + 3] = uint8_t(sc >> 24);
      }
    }
  }
}

static int lds_floats(int D) { return (padded_len((D + 31) / 32 * 32) + 3) / 4 * 4; }

// Forward rotation at D = 96 with both passes in registers (fwht64_r8):
// 8 lanes per row, 32 rows per workgroup, the transpose through one LDS
// buffer per row.  The same results as k_rotate bit for bit.
constexpr int kRot96Rows = 32;
__global__ void __launch_bounds__(256) k_rotate96(const float *__restrict__ x, float *y, int64_t n,
                                                  RotParams rp, int dstride) {
  extern __shared__ float lds[];
  const int sl = threadIdx.x & 7;
  const int slot = threadIdx.x >> 3;
  const int64_t row = int64_t(blockIdx.x) * kRot96Rows + slot;
  if (row >= n) return;   // a row's 8 lanes leave together; no barriers below
  float *v = lds + slot * dstride;
  const uint2 sm = sub_sign_masks<8>(rp, sl);
  const float *xr = x + row * 96;
  float e[12];
#pragma unroll
  for (int t = 0; t < 12; ++t) e[t] = flip_w<8>(xr[sl + 8 * t], sm.x, t);
  fwht64_r8(e, 0, sl, rp.inv_sqrt_b);
  fwht64_r8(e, 4, sl, rp.inv_sqrt_b);
#pragma unroll
  for (int t = 0; t < 12; ++t) v[px(sl + 8 * t)] = e[t];
  wave_sync();
#pragma unroll
  for (int t = 0; t < 12; ++t) e[t] = flip_w<8>(v[px(transpose_src(sl + 8 * t, rp))], sm.y, t);
  fwht64_r8(e, 0, sl, rp.inv_sqrt_b);
  fwht64_r8(e, 4, sl, rp.inv_sqrt_b);
  float *yr = y + row * 96;
#pragma unroll
  for (int t = 0; t < 12; ++t) yr[sl + 8 * t] = e[t];
}


}  // namespace rslm

using namespace rslm;

extern "C" {

int rslm_fwht(const rslm_plan *p, const float *x, float *y, int64_t n, int inverse, void *stream) {
  if (!p || (!x && n) || (!y && n) || n < 0 || (inverse != 0 && inverse != 1))
    return RSLM_ERR_INVALID_ARG;
  if (n == 0) return RSLM_OK;
  if ((n + 3) / 4 > 0x7fffffff) return RSLM_ERR_INVALID_ARG;
  if (launch_rotate_reg(p, x, y, n, inverse, as_stream(stream))) return check_launch();
  const int D = p->rot.D;
  const int dstride = lds_floats(D);
  if (!inverse && D == 96 && p->rot.B == 64 && p->rot.passes == 2) {
    const int64_t g96 = (n + kRot96Rows - 1) / kRot96Rows;
    hipLaunchKernelGGL(k_rotate96, dim3(unsigned(g96)), dim3(8 * kRot96Rows),
                       size_t(kRot96Rows) * dstride * sizeof(float), as_stream(stream), x, y, n,
                       p->rot, dstride);
    return check_launch();
  }
  int waves = 4;
  while (waves > 1 && size_t(waves) * 2 * dstride * 4 > 65536) waves >>= 1;
  const size_t shm = size_t(waves) * 2 * dstride * sizeof(float);
  const int64_t grid = (n + waves - 1) / waves;
  if (grid > 0x7fffffff) return RSLM_ERR_INVALID_ARG;
  hipLaunchKernelGGL(k_rotate, dim3(unsigned(grid)), dim3(64 * waves), shm, as_stream(stream), x,
                     y, n, p->rot, inverse, dstride);
  return check_launch();
}

static int encode_impl(const rslm_plan *p, const rslm_plan *p2, const float *x, int64_t n_rows,
                       const int64_t *src_row, const int32_t *rec_list, int64_t n_records,
                       const float *centroids, const float *centroids_rot, int32_t nlist,
                       uint8_t *codes, uint32_t *scales, float *resid_rot, uint8_t *codes2,
                       uint32_t *scales2, const float *sq8_lo, const float *sq8_hi,
                       hipStream_t s) {
  if (launch_encode_reg(p, p2, x, n_rows, src_row, rec_list, n_records, centroids,
                        centroids_rot, nlist, codes, scales, resid_rot, codes2, scales2, sq8_lo,
                        sq8_hi, s))
    return check_launch();
  const int D = p->rot.D;
  const int dstride = lds_floats(D);
  // vectors per wavefront: a butterfly round has D / 8 groups, so give a
  // vector at most that many lanes (1 to 8 vectors per wavefront; at D = 96,
  // 8 lanes: 0.063 ms per 65,536 vectors against 0.073 with 16 and 0.175
  // with 64)
  int vpw = 1;
  while (vpw < 8 && D * vpw <= 512) vpw *= 2;
  // two float buffers plus one byte per sub-vector (<= dstride bytes) per
  // vector, and another for an RSLM second stage
  const size_t per_vec = 2 * size_t(dstride) * 4 + size_t(dstride) * (p2 ? 2 : 1);
  int waves = 4;
  while (waves > 1 && size_t(waves) * vpw * per_vec > 65536) waves >>= 1;
  const size_t shm = size_t(waves) * vpw * per_vec;
  const int64_t per_wg = int64_t(waves) * vpw;
  const int64_t grid = (n_records + per_wg - 1) / per_wg;
  if (grid > 0x7fffffff) return RSLM_ERR_INVALID_ARG;
#define RSLM_ENCODE_VPW(V)                                                                       \
  hipLaunchKernelGGL((k_encode<V>), dim3(unsigned(grid)), dim3(64 * waves), shm, s, x, n_rows,      \
                     src_row, rec_list, n_records, centroids, centroids_rot, nlist, codes, scales, \
                     resid_rot, p->rot, p->codec, dstride, codes2, scales2,                        \
                     p2 ? p2->codec : p->codec, sq8_lo, sq8_hi)
  switch (vpw) {
    case 8: RSLM_ENCODE_VPW(8); break;
    case 4: RSLM_ENCODE_VPW(4); break;
    case 2: RSLM_ENCODE_VPW(2); break;
    default: RSLM_ENCODE_VPW(1); break;
  }
#undef RSLM_ENCODE_VPW
  return check_launch();
}

static int encode_args_ok(const rslm_plan *p, const float *x, int64_t n_rows,
                          const int64_t *src_row, const int32_t *rec_list, int64_t n_records,
                          const float *centroids, const float *centroids_rot, int32_t nlist,
                          uint8_t *codes, uint32_t *scales) {
  if (!p || n_records < 0 || n_rows < 0) return RSLM_ERR_INVALID_ARG;
  if (n_records == 0) return RSLM_OK;
  if (!x || !codes || !scales) return RSLM_ERR_INVALID_ARG;
  if (centroids && (!rec_list || !centroids_rot || nlist < 1)) return RSLM_ERR_INVALID_ARG;
  if (!src_row && n_records > n_rows) return RSLM_ERR_INVALID_ARG;
  if ((n_records + 3) / 4 > 0x7fffffff) return RSLM_ERR_INVALID_ARG;
  return RSLM_OK;
}

int rslm_encode(const rslm_plan *p, const float *x, int64_t n_rows, const int64_t *src_row,
                const int32_t *rec_list, int64_t n_records, const float *centroids,
                const float *centroids_rot, int32_t nlist, uint8_t *codes, uint32_t *scales,
                float *resid_rot, void *stream) {
  const int st = encode_args_ok(p, x, n_rows, src_row, rec_list, n_records, centroids,
                                centroids_rot, nlist, codes, scales);
  if (st || n_records == 0) return st;
  return encode_impl(p, nullptr, x, n_rows, src_row, rec_list, n_records, centroids,
                     centroids_rot, nlist, codes, scales, resid_rot, nullptr, nullptr, nullptr,
                     nullptr, as_stream(stream));
}

int rslm_encode_two_stage(const rslm_plan *p, const rslm_plan *p2, const float *x,
                          int64_t n_rows, const int64_t *src_row, const int32_t *rec_list,
                          int64_t n_records, const float *centroids, const float *centroids_rot,
                          int32_t nlist, uint8_t *codes, uint32_t *scales, uint8_t *codes2,
                          uint32_t *scales2, void *stream) {
  const int st = encode_args_ok(p, x, n_rows, src_row, rec_list, n_records, centroids,
                                centroids_rot, nlist, codes, scales);
  if (st) return st;
  if (!p2 || p2->rot.D != p->rot.D || p2->rot.passes != 0) return RSLM_ERR_INVALID_ARG;
  if (n_records == 0) return RSLM_OK;
  if (!codes2 || !scales2) return RSLM_ERR_INVALID_ARG;
  return encode_impl(p, p2, x, n_rows, src_row, rec_list, n_records, centroids, centroids_rot,
                     nlist, codes, scales, nullptr, codes2, scales2, nullptr, nullptr,
                     as_stream(stream));
}

int rslm_encode_sq8(const rslm_plan *p, const float *x, int64_t n_rows, const int64_t *src_row,
                    const int32_t *rec_list, int64_t n_records, const float *centroids,
                    const float *centroids_rot, int32_t nlist, uint8_t *codes, uint32_t *scales,
                    const float *sq8_lo, const float *sq8_hi, uint8_t *codes2, void *stream) {
  const int st = encode_args_ok(p, x, n_rows, src_row, rec_list, n_records, centroids,
                                centroids_rot, nlist, codes, scales);
  if (st || n_records == 0) return st;
  if (!sq8_lo || !sq8_hi || !codes2) return RSLM_ERR_INVALID_ARG;
  return encode_impl(p, nullptr, x, n_rows, src_row, rec_list, n_records, centroids,
                     centroids_rot, nlist, codes, scales, nullptr, codes2, nullptr, sq8_lo,
                     sq8_hi, as_stream(stream));
}

static int64_t pack_grid(int64_t total) {
  int64_t grid = (total + 255) / 256;
  return grid > 65536 ? 65536 : (grid < 1 ? 1 : grid);
}

int rslm_pack_codes(const rslm_plan *p, const uint8_t *canon, int64_t n, uint8_t *tiles,
                    void *stream) {
  if (!p || n < 0) return RSLM_ERR_INVALID_ARG;
  if (n == 0) return RSLM_OK;
  if (!canon || !tiles) return RSLM_ERR_INVALID_ARG;
  const int64_t total = (n + 15) / 16 * 16 * (p->codec.d_pad / 8);
  hipLaunchKernelGGL(k_pack, dim3(unsigned(pack_grid(total))), dim3(256), 0, as_stream(stream),
                     canon, n, tiles, p->codec);
  return check_launch();
}

int rslm_decode(const rslm_plan *p, const uint8_t *codes, const uint32_t *scales, int64_t n,
                const int32_t *rec_list, const float *centroids, int32_t nlist, float *out,
                void *stream) {
  if (!p || n < 0) return RSLM_ERR_INVALID_ARG;
  if (n == 0) return RSLM_OK;
  if (!codes || !scales || !out) return RSLM_ERR_INVALID_ARG;
  if (centroids && (!rec_list || nlist < 1)) return RSLM_ERR_INVALID_ARG;
  const int D = p->rot.D;
  const int dstride = lds_floats(D);
  int waves = 4;
  while (waves > 1 && size_t(waves) * 2 * dstride * 4 > 65536) waves >>= 1;
  const size_t shm = size_t(waves) * 2 * dstride * sizeof(float);
  const int64_t grid = (n + waves - 1) / waves;
  if (grid > 0x7fffffff) return RSLM_ERR_INVALID_ARG;
  hipLaunchKernelGGL(k_decode, dim3(unsigned(grid)), dim3(64 * waves), shm, as_stream(stream),
                     codes, scales, n, rec_list, centroids, nlist, out, p->rot, p->codec, dstride);
  return check_launch();
}

int rslm_pack_records(const rslm_plan *p, const uint8_t *tiles, const uint32_t *scales, int64_t n,
                      uint8_t *records, void *stream) {
  if (!p || n < 0) return RSLM_ERR_INVALID_ARG;
  if (n == 0) return RSLM_OK;
  if (!tiles || !records || (!scales && p->codec.lead == 0)) return RSLM_ERR_INVALID_ARG;
  const int64_t total = n * (p->codec.d_pad / 8);
  hipLaunchKernelGGL(k_pack_records, dim3(unsigned(pack_grid(total))), dim3(256), 0,
                     as_stream(stream), tiles, scales, n, records, p->codec);
  return check_launch();
}

int rslm_unpack_codes(const rslm_plan *p, const uint8_t *tiles, int64_t n, uint8_t *canon,
                      void *stream) {
  if (!p || n < 0) return RSLM_ERR_INVALID_ARG;
  if (n == 0) return RSLM_OK;
  if (!canon || !tiles) return RSLM_ERR_INVALID_ARG;
  const int64_t total = n * (p->codec.d_pad / 8);
  hipLaunchKernelGGL(k_unpack, dim3(unsigned(pack_grid(total))), dim3(256), 0, as_stream(stream),
                     tiles, n, canon, p->codec);
  return check_launch();
}

}  // extern "C"
