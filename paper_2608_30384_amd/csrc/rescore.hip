// Rescoring stage: the 8-bit SQ8 codec on the rotated second residual and
// the rescoring of a shortlist (paper, Section "Background and Related Work":
// low-bit scoring produces a shortlist that a higher-fidelity representation
// rescores; SQ8 as a per-dimension 256-level scalar quantiser; Section
// "Relative Quantization": <q, a + r~2> = <q, a> + <q, r~2> reuses the
// first-stage score <q, a>).
//
// Rescoring gathers one record per shortlisted candidate (random access, the
// paper's "LargePool" pattern); a workgroup per query decodes and scores its
// candidates (16 lanes per candidate, dword loads across coordinates) and
// sorts them in LDS.
#include "rslm_internal.h"
#include "select_dev.h"

namespace rslm {

__global__ void k_keys_init(uint32_t *lo, uint32_t *hi, int dim, int from_floats) {
  const int d = blockIdx.x * blockDim.x + threadIdx.x;
  if (d >= dim) return;
  if (from_floats) {
    lo[d] = order_key(__uint_as_float(lo[d]));
    hi[d] = order_key(__uint_as_float(hi[d]));
  } else {
    lo[d] = 0xffffffffu;
    hi[d] = 0u;
  }
}

__global__ void k_keys_to_float(uint32_t *lo, uint32_t *hi, int dim) {
  const int d = blockIdx.x * blockDim.x + threadIdx.x;
  if (d >= dim) return;
  lo[d] = __float_as_uint(key_to_float(lo[d]));
  hi[d] = __float_as_uint(key_to_float(hi[d]));
}

// grid.x covers dimensions (256 per block), grid.y splits the rows
__global__ void k_sq8_minmax(const float *__restrict__ v, int64_t n, int dim, int64_t rows_per,
                             uint32_t *lo, uint32_t *hi) {
  const int d = blockIdx.x * blockDim.x + threadIdx.x;
  if (d >= dim) return;
  const int64_t r0 = int64_t(blockIdx.y) * rows_per;
  const int64_t r1 = min(n, r0 + rows_per);
  if (r0 >= r1) return;
  float mn = 3.4e38f, mx = -3.4e38f;
  for (int64_t r = r0; r < r1; ++r) {
    const float x = v[r * dim + d];
    mn = fminf(mn, x);
    mx = fmaxf(mx, x);
  }
  atomicMin(&lo[d], order_key(mn));
  atomicMax(&hi[d], order_key(mx));
}

__global__ void k_sq8_encode(const float *__restrict__ v, int64_t n, int dim,
                             const float *__restrict__ lo, const float *__restrict__ hi,
                             const int32_t *__restrict__ dest, int64_t n_dest,
                             uint8_t *__restrict__ codes) {
  const int64_t total = n * dim;
  for (int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; t < total;
       t += int64_t(gridDim.x) * blockDim.x) {
    const int64_t r = t / dim;
    const int d = int(t - r * dim);
    const int64_t o = dest ? int64_t(dest[r]) : r;
    if (o < 0 || o >= n_dest) continue;
    codes[o * dim + d] = uint8_t(sq8_code(v[t], lo[d], hi[d]));
  }
}

constexpr int kRescoreThreads = 256;

// Sorts the n (key, id) entries of buf descending (LDS bitonic sort over the
// next power of two) and writes the first k_out of query q, padding with
// (-inf, -1).  Every thread of the workgroup calls it.
__device__ void sort_emit(uint64_t *buf, int n, int q, int k_out, float *__restrict__ out_s,
                          int32_t *__restrict__ out_i) {
  const int tid = threadIdx.x;
  if (n <= int(blockDim.x)) {   // one candidate per thread: order by rank counting
    rank_emit(buf, n, k_out, out_s + int64_t(q) * k_out, out_i + int64_t(q) * k_out);
    return;
  }
  int p2 = 1;
  while (p2 < n) p2 <<= 1;
  for (int i = n + tid; i < p2; i += blockDim.x) buf[i] = 0ull;
  __syncthreads();
  for (int size = 2; size <= p2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < p2 / 2; i += blockDim.x) {
        const int a0 = 2 * i - (i & (stride - 1));
        const int a1 = a0 + stride;
        const bool desc = ((a0 & size) == 0);
        const uint64_t x = buf[a0], y = buf[a1];
        if ((x < y) == desc) {
          buf[a0] = y;
          buf[a1] = x;
        }
      }
      __syncthreads();
    }
  }
  for (int j = tid; j < k_out; j += blockDim.x) {
    if (j < n) {
      out_s[int64_t(q) * k_out + j] = key_to_float(uint32_t(buf[j] >> 32));
      out_i[int64_t(q) * k_out + j] = int32_t(0xffffffffu - uint32_t(buf[j] & 0xffffffffu));
    } else {
      out_s[int64_t(q) * k_out + j] = -__builtin_inff();
      out_i[int64_t(q) * k_out + j] = -1;
    }
  }
}

__device__ __forceinline__ uint64_t score_key(float s, int32_t id) {
  return (uint64_t(order_key(s)) << 32) | uint64_t(0xffffffffu - uint32_t(id));
}

constexpr int kSq8Threads = 1024;   // 64 candidates in flight per workgroup

__global__ void __launch_bounds__(kSq8Threads) k_rescore_sq8(
    const uint8_t *__restrict__ codes, int64_t n_vec, int dim, const float *__restrict__ lo,
    const float *__restrict__ hi, const float *__restrict__ q_rot,
    const float *__restrict__ cand_s, const int32_t *__restrict__ cand_i, int k_in, int k_out,
    float *__restrict__ out_s, int32_t *__restrict__ out_i) {
  extern __shared__ float qs[];   // dim floats: q_d * step_d
  __shared__ uint64_t buf[kMaxK];
  __shared__ float red[kSq8Threads / 64];
  __shared__ uint32_t count;
  const int q = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float *qr = q_rot + int64_t(q) * dim;
  const bool wide = (dim & 15) == 0 && (reinterpret_cast<uintptr_t>(codes) & 15) == 0;
  // wide rows: float4 f of qs is stored at f ^ ((f >> 4) & 3), so that the
  // 16 lanes of a candidate, reading float4s 4 j + c (j = lane, c fixed),
  // touch 16 distinct 16-byte bank groups
  auto slot = [&](int d) { return wide ? (d ^ (((d >> 6) & 3) << 2)) : d; };
  float part = 0.f;
  for (int d = tid; d < dim; d += kSq8Threads) {
    const float step = (hi[d] - lo[d]) / 255.f;
    qs[slot(d)] = qr[d] * step;
    part += qr[d] * lo[d];
  }
  part = wave_sum(part);
  if (lane == 0) red[wave] = part;
  if (tid == 0) count = 0;
  __syncthreads();
  float qlo = 0.f;
  for (int w = 0; w < kSq8Threads / 64; ++w) qlo += red[w];
  // 16 lanes per candidate, four candidates per wavefront; lane j of a group
  // takes the 16-byte units j, j + 16, ... of the candidate's codes (dwords
  // when rows are not whole aligned 16-byte runs), all loads of a candidate
  // issued before its products.
  __syncthreads();   // qs complete
  const int grp = lane >> 4, gl = lane & 15;
  const int ngroups = (kSq8Threads / 64) * 4;
  for (int j0 = wave * 4; j0 < k_in; j0 += ngroups) {
    const int j = j0 + grp;
    int32_t id = -1;
    float s1 = 0.f;   // loaded with the id, not after the products
    if (j < k_in) {
      id = cand_i[int64_t(q) * k_in + j];
      s1 = cand_s[int64_t(q) * k_in + j];
    }
    const bool valid = id >= 0 && id < n_vec;
    float dot = 0.f;
    if (valid) {
      const uint8_t *cr = codes + int64_t(id) * dim;
      auto dot4 = [&](uint32_t w, int d) {
        const float4 qv = *reinterpret_cast<const float4 *>(qs + d);
        return qv.x * float(w & 0xffu) + qv.y * float((w >> 8) & 0xffu) +
               qv.z * float((w >> 16) & 0xffu) + qv.w * float(w >> 24);
      };
      if (wide) {
        const uint4 *cw = reinterpret_cast<const uint4 *>(cr);
        const int nd16 = dim >> 4;
#pragma unroll 4
        for (int d16 = gl; d16 < nd16; d16 += 16) {
          const uint4 w = cw[d16];
          dot += dot4(w.x, slot(16 * d16)) + dot4(w.y, slot(16 * d16 + 4)) +
                 dot4(w.z, slot(16 * d16 + 8)) + dot4(w.w, slot(16 * d16 + 12));
        }
      } else if ((dim & 3) == 0) {
        const uint32_t *cw = reinterpret_cast<const uint32_t *>(cr);
        const int nd4 = dim >> 2;
#pragma unroll 4
        for (int d4 = gl; d4 < nd4; d4 += 16) dot += dot4(cw[d4], 4 * d4);
      } else {
        for (int d = gl; d < dim; d += 16) dot += qs[d] * float(cr[d]);
      }
    }
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) dot += __shfl_xor(dot, off, 64);
    if (valid && gl == 0) {
      const float s2 = s1 + (qlo + dot);
      const uint32_t pos = atomicAdd(&count, 1u);
      buf[pos] = score_key(s2, id);
    }
  }
  __syncthreads();
  sort_emit(buf, int(count), q, k_out, out_s, out_i);
}

// RSLM rescoring records (canonical layout, w-bit codes of g-sub-vectors):
// score2 = g2^ (score1 + s2^ sum_j <q_rot[j g:(j+1) g], C2[code_j]>).  A
// workgroup per query holds the zero-padded rotated query and the codebook
// in LDS; 16 lanes per candidate, lane j of a group decoding the 8-code
// groups j, j + 16, ... (w bytes each: one dword for 4-bit codes).
template <int W, int G>
__global__ void __launch_bounds__(kRescoreThreads) k_rescore_rslm(
    const uint8_t *__restrict__ codes, const uint32_t *__restrict__ scales, int64_t n_vec,
    int dim, int n_sub, int canon_bytes, CodecParams cp, const float *__restrict__ q_rot, const float *__restrict__ cand_s,
    const int32_t *__restrict__ cand_i, int k_in, int k_out, float *__restrict__ out_s,
    int32_t *__restrict__ out_i) {
  extern __shared__ float qs[];   // n_groups * 8 * G floats, zero beyond dim
  __shared__ uint64_t buf[kMaxK];
  __shared__ float cbs[16 * G];
  __shared__ uint32_t count;
  const int q = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_groups = (n_sub + 7) / 8;
  const float *qr = q_rot + int64_t(q) * dim;
  for (int d = tid; d < n_groups * 8 * G; d += kRescoreThreads) qs[d] = (d < dim) ? qr[d] : 0.f;
  if (tid < 16 * G && tid < (1 << W) * G) cbs[tid] = cp.cb[tid];
  if (tid == 0) count = 0;
  __syncthreads();
  const int grp = lane >> 4, gl = lane & 15;
  const int ngroups = (kRescoreThreads / 64) * 4;
  const bool dword_ok = (W == 4) && (canon_bytes % 4 == 0) &&
                        (reinterpret_cast<uintptr_t>(codes) % 4 == 0);
  for (int j0 = wave * 4; j0 < k_in; j0 += ngroups) {
    const int j = j0 + grp;
    int32_t id = -1;
    if (j < k_in) id = cand_i[int64_t(q) * k_in + j];
    const bool valid = id >= 0 && id < n_vec;
    float dot = 0.f;
    if (valid) {
      const uint8_t *cr = codes + int64_t(id) * canon_bytes;
      for (int G8 = gl; G8 < n_groups; G8 += 16) {
        // the w bytes of 8 codes (bytes past the record read as 0)
        uint32_t bits;
        if (dword_ok) {
          bits = reinterpret_cast<const uint32_t *>(cr)[G8];
        } else {
          bits = 0u;
#pragma unroll
          for (int t = 0; t < W; ++t) {
            const int byte = W * G8 + t;
            if (byte < canon_bytes) bits |= uint32_t(cr[byte]) << (8 * t);
          }
        }
        const float *qv = qs + G8 * 8 * G;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const uint32_t code = (bits >> (W * c)) & ((1u << W) - 1u);
#pragma unroll
          for (int t = 0; t < G; ++t) dot = fmaf(qv[c * G + t], cbs[code * G + t], dot);
        }
      }
    }
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) dot += __shfl_xor(dot, off, 64);
    if (valid && gl == 0) {
      const uint32_t sc = scales[id];
      const float s2 = dec_ue4m12(sc >> 16) *
                       (cand_s[int64_t(q) * k_in + j] + dec_ue7m9(sc & 0xffffu) * dot);
      const uint32_t pos = atomicAdd(&count, 1u);
      buf[pos] = score_key(s2, id);
    }
  }
  __syncthreads();
  sort_emit(buf, int(count), q, k_out, out_s, out_i);
}

// OneToMany scoring of packed records: score = g^ s^ sum_j <q_rot[j g:(j+1) g],
// C[code_j]> for record ids[j] (or j).  A workgroup covers `per_block`
// consecutive entries of one query (grid.y); 16 lanes per record, lane j of a
// group decoding the 8-code groups j, j + 16, ... from one 4-byte load (any
// alignment; 3-bit records: three bytes).  LITE: the first cp.lead codes are
// 3-bit codes on the K = 8 codebook whose bit 3 carries the scales, gathered
// from the 16 lanes by an OR reduction.
struct __attribute__((packed, aligned(1))) U32Unaligned {
  uint32_t v;
};

template <int W, int G, bool LITE>
__global__ void __launch_bounds__(kRescoreThreads) k_score(
    const uint8_t *__restrict__ records, int64_t n_pool, const int64_t *__restrict__ ids,
    int64_t n, int64_t per_block, const float *__restrict__ q_rot, int dim, CodecParams cp,
    float *__restrict__ out) {
  extern __shared__ float qs[];   // n_groups * 8 * G floats, zero beyond dim
  __shared__ float cbs[16 * G], cbl[8];
  const int q = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_groups = (cp.n_sub + 7) / 8;
  const float *qr = q_rot + int64_t(q) * dim;
  for (int d = tid; d < n_groups * 8 * G; d += kRescoreThreads) qs[d] = (d < dim) ? qr[d] : 0.f;
  if (tid < 16 * G && tid < (1 << W) * G) cbs[tid] = cp.cb[tid];
  if (LITE && tid < 8) cbl[tid] = cp.cb_lead[tid];
  __syncthreads();
  const int grp = wave * 4 + (lane >> 4), gl = lane & 15;
  const int64_t j0 = int64_t(blockIdx.x) * per_block;
  const int64_t j1 = min(n, j0 + per_block);
  for (int64_t j = j0 + grp; j < j1; j += (kRescoreThreads / 16)) {
    const int64_t r = ids ? ids[j] : j;
    const bool valid = r >= 0 && r < n_pool;
    const uint8_t *rec = records + (valid ? r : 0) * int64_t(cp.record_bytes);
    float dot = 0.f;
    uint32_t sbits = 0u, gbits = 0u;
    for (int G8 = gl; valid && G8 < n_groups; G8 += 16) {
      uint32_t bits = 0u;
      if (W * G8 + 4 <= cp.record_bytes) {
        bits = reinterpret_cast<const U32Unaligned *>(rec + W * G8)->v;
      } else {
#pragma unroll
        for (int t = 0; t < W; ++t)
          if (W * G8 + t < cp.canon_bytes) bits |= uint32_t(rec[W * G8 + t]) << (8 * t);
      }
      if (W * G8 + W > cp.canon_bytes)   // the record's last group: only its code bytes
        bits &= (cp.canon_bytes - W * G8 >= 4) ? 0xffffffffu
                                              : ((1u << (8 * (cp.canon_bytes - W * G8))) - 1u);
      const float *qv = qs + G8 * 8 * G;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        uint32_t code = (bits >> (W * c)) & ((1u << W) - 1u);
        if (LITE && G8 * 8 + c < cp.lead) {
          const int jj = G8 * 8 + c;
          if (jj < 16) sbits |= (code >> 3) << jj;
          else gbits |= (code >> 3) << (jj - 16);
          dot = fmaf(qv[c], cbl[code & 7u], dot);
          continue;
        }
#pragma unroll
        for (int t = 0; t < G; ++t) dot = fmaf(qv[c * G + t], cbs[code * G + t], dot);
      }
    }
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) {
      dot += __shfl_xor(dot, off, 64);
      if (LITE) {
        sbits |= __shfl_xor(sbits, off, 64);
        gbits |= __shfl_xor(gbits, off, 64);
      }
    }
    if (gl == 0) {
      uint32_t su = 0u, gu = 0u;
      if (LITE) {
        su = sbits;
        gu = cp.global ? gbits : 0x7000u;
      } else if (valid) {
        const uint8_t *sf = rec + cp.canon_bytes;
        su = uint32_t(sf[0]) | (uint32_t(sf[1]) << 8);
        gu = cp.global ? (uint32_t(sf[2]) | (uint32_t(sf[3]) << 8)) : 0x7000u;
      }
      out[int64_t(q) * n + j] = valid ? dec_ue4m12(gu) * (dec_ue7m9(su) * dot) : -__builtin_inff();
    }
  }
}

// The same scoring with the query held in registers (D <= 1024): lane j of a
// record's 16 lanes always decodes the groups j + 16 k (k < 8 / G), so it
// loads its q values once; per code: a field extract, one LDS lookup of the
// 16-entry codebook (16 banks, broadcast-friendly) and G multiply-adds.
// Each 16-lane group scores two records per pass with all loads issued first.
template <int W, int G, bool LITE, int KMAX>
__global__ void __launch_bounds__(kRescoreThreads) k_score_reg(
    const uint8_t *__restrict__ records, int64_t n_pool, const int64_t *__restrict__ ids,
    int64_t n, int64_t per_block, const float *__restrict__ q_rot, int dim, CodecParams cp,
    float *__restrict__ out) {
  // KMAX: groups per lane (n_groups <= 16 KMAX)
  constexpr uint32_t kMask = (1u << W) - 1u;
  __shared__ float cbs[16 * G], cbl[16];
  const int q = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_groups = (cp.n_sub + 7) / 8;
  if (tid < 16 * G) cbs[tid] = (tid < (1 << W) * G) ? cp.cb[tid] : 0.f;
  if (LITE && tid < 16) cbl[tid] = cp.cb_lead[tid & 7];
  const int gl = lane & 15;
  const float *qr = q_rot + int64_t(q) * dim;
  float qv[KMAX][8 * G];
#pragma unroll
  for (int k = 0; k < KMAX; ++k)
#pragma unroll
    for (int t = 0; t < 8 * G; ++t) {
      const int d = (gl + 16 * k) * 8 * G + t;
      qv[k][t] = (d < dim) ? qr[d] : 0.f;
    }
  __syncthreads();
  const int grp = wave * 4 + (lane >> 4);
  const int64_t j0 = int64_t(blockIdx.x) * per_block;
  const int64_t j1 = min(n, j0 + per_block);
  constexpr int kGroups = kRescoreThreads / 16;
  for (int64_t jb = j0 + grp; jb < j1; jb += 2 * kGroups) {
    const uint8_t *rec[2];
    bool valid[2];
    uint32_t bits[2][KMAX];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t j = jb + u * kGroups;
      int64_t r = -1;
      if (j < j1) r = ids ? ids[j] : j;
      valid[u] = r >= 0 && r < n_pool;
      rec[u] = records + (valid[u] ? r : 0) * int64_t(cp.record_bytes);
#pragma unroll
      for (int k = 0; k < KMAX; ++k) {
        const int G8 = gl + 16 * k;
        uint32_t b = 0u;
        if (valid[u] && G8 < n_groups) {
          if (W * G8 + 4 <= cp.record_bytes) {
            b = reinterpret_cast<const U32Unaligned *>(rec[u] + W * G8)->v;
          } else {
#pragma unroll
            for (int t = 0; t < W; ++t)
              if (W * G8 + t < cp.canon_bytes) b |= uint32_t(rec[u][W * G8 + t]) << (8 * t);
          }
          if (W * G8 + W > cp.canon_bytes && cp.canon_bytes - W * G8 < 4)
            b &= (1u << (8 * (cp.canon_bytes - W * G8))) - 1u;
        }
        bits[u][k] = b;
      }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t j = jb + u * kGroups;
      float dot = 0.f;
      uint32_t sbits = 0u, gbits = 0u;
#pragma unroll
      for (int k = 0; k < KMAX; ++k) {
        uint32_t b = bits[u][k];
        if (LITE && k == 0 && gl < cp.lead / 8) {
          // leading coordinates: 3-bit codes on the K = 8 codebook, bit 3 a scale bit
          uint32_t top = 0u;
#pragma unroll
          for (int c = 0; c < 8; ++c) top |= ((b >> (4 * c + 3)) & 1u) << c;
          if (gl < 2) sbits = top << (8 * gl);
          else gbits = top << (8 * (gl - 2));
#pragma unroll
          for (int c = 0; c < 8; ++c) dot = fmaf(qv[k][c], cbl[(b >> (4 * c)) & 7u], dot);
          continue;
        }
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const uint32_t code = (b >> (W * c)) & kMask;
#pragma unroll
          for (int t = 0; t < G; ++t) dot = fmaf(qv[k][c * G + t], cbs[code * G + t], dot);
        }
      }
#pragma unroll
      for (int off = 8; off >= 1; off >>= 1) {
        dot += __shfl_xor(dot, off, 64);
        if (LITE) {
          sbits |= __shfl_xor(sbits, off, 64);
          gbits |= __shfl_xor(gbits, off, 64);
        }
      }
      if (gl == 0 && j < j1) {
        uint32_t su = 0u, gu = 0u;
        if (LITE) {
          su = sbits;
          gu = cp.global ? gbits : 0x7000u;
        } else if (valid[u]) {
          const uint8_t *sf = rec[u] + cp.canon_bytes;
          su = uint32_t(sf[0]) | (uint32_t(sf[1]) << 8);
          gu = cp.global ? (uint32_t(sf[2]) | (uint32_t(sf[3]) << 8)) : 0x7000u;
        }
        out[int64_t(q) * n + j] =
            valid[u] ? dec_ue4m12(gu) * (dec_ue7m9(su) * dot) : -__builtin_inff();
      }
    }
  }
}

}  // namespace rslm

using namespace rslm;

extern "C" {

int rslm_sq8_fit(const float *v, int64_t n, int32_t dim, float *lo, float *hi, int accumulate,
                 void *stream) {
  if (n < 0 || dim < 1 || !lo || !hi || (n > 0 && !v)) return RSLM_ERR_INVALID_ARG;
  hipStream_t s = as_stream(stream);
  uint32_t *klo = reinterpret_cast<uint32_t *>(lo), *khi = reinterpret_cast<uint32_t *>(hi);
  const dim3 gd((dim + 255) / 256);
  hipLaunchKernelGGL(k_keys_init, gd, dim3(256), 0, s, klo, khi, dim, accumulate ? 1 : 0);
  int st = check_launch();
  if (st) return st;
  if (n > 0) {
    int64_t splits = (n + 4095) / 4096;
    if (splits > 4096) splits = 4096;
    const int64_t rows_per = (n + splits - 1) / splits;
    hipLaunchKernelGGL(k_sq8_minmax, dim3(gd.x, unsigned(splits)), dim3(256), 0, s, v, n, dim,
                       rows_per, klo, khi);
    if ((st = check_launch())) return st;
  }
  hipLaunchKernelGGL(k_keys_to_float, gd, dim3(256), 0, s, klo, khi, dim);
  return check_launch();
}

int rslm_sq8_encode(const float *v, int64_t n, int32_t dim, const float *lo, const float *hi,
                    const int32_t *dest_row, int64_t n_dest, uint8_t *codes, void *stream) {
  if (n < 0 || dim < 1 || n_dest < 0) return RSLM_ERR_INVALID_ARG;
  if (n == 0) return RSLM_OK;
  if (!v || !lo || !hi || !codes) return RSLM_ERR_INVALID_ARG;
  if (!dest_row && n > n_dest) return RSLM_ERR_INVALID_ARG;
  int64_t grid = (n * dim + 255) / 256;
  if (grid > 1 << 20) grid = 1 << 20;
  hipLaunchKernelGGL(k_sq8_encode, dim3(unsigned(grid)), dim3(256), 0, as_stream(stream), v, n,
                     dim, lo, hi, dest_row, n_dest, codes);
  return check_launch();
}

int rslm_rescore(const rslm_rescore_codec *c, const float *q_rot, int32_t Q,
                 const float *cand_scores, const int32_t *cand_ids, int32_t k_in, int32_t k_out,
                 float *out_scores, int32_t *out_ids, void *stream) {
  if (!c || Q < 0 || k_in < 1 || k_in > kMaxK || k_out < 1 || k_out > k_in)
    return RSLM_ERR_INVALID_ARG;
  if (c->kind != RSLM_RESCORE_SQ8 && c->kind != RSLM_RESCORE_RSLM) return RSLM_ERR_UNSUPPORTED;
  if (c->dim < 1 || c->dim > kMaxDim || c->n_vectors < 0) return RSLM_ERR_INVALID_ARG;
  if (c->kind == RSLM_RESCORE_RSLM &&
      (!c->plan || c->plan->rot.D != c->dim || c->plan->rot.passes != 0))
    return RSLM_ERR_INVALID_ARG;
  if (c->kind == RSLM_RESCORE_RSLM && c->plan->codec.lead > 0) return RSLM_ERR_UNSUPPORTED;
  if (Q == 0) return RSLM_OK;
  if (!c->codes || !q_rot || !cand_scores || !cand_ids || !out_scores || !out_ids)
    return RSLM_ERR_INVALID_ARG;
  hipStream_t s = as_stream(stream);
  if (c->kind == RSLM_RESCORE_SQ8) {
    if (!c->lo || !c->hi) return RSLM_ERR_INVALID_ARG;
    hipLaunchKernelGGL(k_rescore_sq8, dim3(unsigned(Q)), dim3(kSq8Threads),
                       size_t(c->dim) * sizeof(float), s, c->codes, c->n_vectors, c->dim, c->lo,
                       c->hi, q_rot, cand_scores, cand_ids, k_in, k_out, out_scores, out_ids);
    return check_launch();
  }
  if (!c->scales) return RSLM_ERR_INVALID_ARG;
  const CodecParams &cp = c->plan->codec;
  const int n_groups = (cp.n_sub + 7) / 8;
  const size_t shm = size_t(n_groups) * 8 * cp.g * sizeof(float);
#define RSLM_RESCORE_CALL(W, G)                                                               \
  hipLaunchKernelGGL((k_rescore_rslm<W, G>), dim3(unsigned(Q)), dim3(kRescoreThreads), shm, s, \
                     c->codes, c->scales, c->n_vectors, c->dim, cp.n_sub, cp.canon_bytes, cp,  \
                     q_rot, cand_scores, cand_ids, k_in, k_out, out_scores, out_ids)
  switch (cp.bits) {
    case 1: RSLM_RESCORE_CALL(4, 4); break;
    case 2: RSLM_RESCORE_CALL(4, 2); break;
    case 3: RSLM_RESCORE_CALL(3, 1); break;
    default: RSLM_RESCORE_CALL(4, 1); break;
  }
#undef RSLM_RESCORE_CALL
  return check_launch();
}

int rslm_score(const rslm_plan *p, const uint8_t *records, int64_t n_pool, const int64_t *ids,
               int64_t n, const float *q_rot, int32_t Q, float *out, void *stream) {
  if (!p || n_pool < 0 || n < 0 || Q < 0) return RSLM_ERR_INVALID_ARG;
  if (Q > 65535) return RSLM_ERR_INVALID_ARG;
  if (!ids && n > n_pool) return RSLM_ERR_INVALID_ARG;
  if (n == 0 || Q == 0) return RSLM_OK;
  if (!records || !q_rot || !out) return RSLM_ERR_INVALID_ARG;
  const CodecParams &cp = p->codec;
  const int n_groups = (cp.n_sub + 7) / 8;
  const size_t shm = size_t(n_groups) * 8 * cp.g * sizeof(float);
  // workgroups of 256 records (16 per pass of the 16-lane groups)
  const int64_t per_block = 256;
  const int64_t blocks = (n + per_block - 1) / per_block;
  if (blocks > 0x7fffffff) return RSLM_ERR_INVALID_ARG;
  const dim3 grid(static_cast<unsigned>(blocks), static_cast<unsigned>(Q));
  hipStream_t s = as_stream(stream);
  // query in registers when every lane's groups fit (at most 8 / g groups of
  // 8 codes per lane): the instantiated group counts 1, 2, 4, 6, 8
  const int need = (n_groups + 15) / 16;
  int ngl = 0;
  for (int v : {1, 2, 4, 6, 8})
    if (v >= need) {
      ngl = v;
      break;
    }
  if (ngl * cp.g > 8) ngl = 0;
#define RSLM_SCORE_REG(W, G, LT, NG)                                                                \
  hipLaunchKernelGGL((k_score_reg<W, G, LT, NG>), grid, dim3(kRescoreThreads), 0, s, records,       \
                     n_pool, ids, n, per_block, q_rot, cp.D, cp, out)
#define RSLM_SCORE_CALL(W, G, LT)                                                                   \
  switch (ngl * int(8 / G >= ngl)) {                                                               \
    case 1: RSLM_SCORE_REG(W, G, LT, 1); break;                                                    \
    case 2: if (8 / G >= 2) RSLM_SCORE_REG(W, G, LT, (8 / G >= 2 ? 2 : 1)); break;                 \
    case 4: if (8 / G >= 4) RSLM_SCORE_REG(W, G, LT, (8 / G >= 4 ? 4 : 1)); break;                 \
    case 6: if (8 / G >= 6) RSLM_SCORE_REG(W, G, LT, (8 / G >= 6 ? 6 : 1)); break;                 \
    case 8: if (8 / G >= 8) RSLM_SCORE_REG(W, G, LT, (8 / G >= 8 ? 8 : 1)); break;                 \
    default:                                                                                       \
      hipLaunchKernelGGL((k_score<W, G, LT>), grid, dim3(kRescoreThreads), shm, s, records, n_pool, \
                         ids, n, per_block, q_rot, cp.D, cp, out);                                 \
  }
  if (cp.lead > 0) {
    RSLM_SCORE_CALL(4, 1, true);
  } else {
    switch (cp.bits) {
      case 1: RSLM_SCORE_CALL(4, 4, false); break;
      case 2: RSLM_SCORE_CALL(4, 2, false); break;
      case 3: RSLM_SCORE_CALL(3, 1, false); break;
      default: RSLM_SCORE_CALL(4, 1, false); break;
    }
  }
#undef RSLM_SCORE_CALL
#undef RSLM_SCORE_REG
  return check_launch();
}

}  // extern "C"
