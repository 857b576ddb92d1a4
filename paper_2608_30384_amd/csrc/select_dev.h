// Block-wide exact top-k of a float array in global memory, ordered by
// (value desc, id asc), with ids produced on demand by a functor (so ids are
// only looked up for survivors).
//
// Method: MSB radix select on order-preserving 32-bit keys.  Each pass
// histograms the next digit of the keys that still share the boundary
// prefix; as soon as the elements at or above the boundary bin fit in the
// LDS buffer they are collected with their ids and bitonic-sorted on the
// 64-bit composite (key << 32 | ~id).  If more than the buffer's capacity
// share one exact key, the smallest ids among them are chosen by a second
// radix select over the ids.  Every pass is a full read of the array.
#pragma once

#include "rslm_internal.h"

namespace rslm {

constexpr int kSelCap = 2048;       // LDS sort buffer entries
constexpr int kSelThreads = 256;

// The histogram is only live during the radix passes and the sort buffer
// only during sampling and collection, so they share storage.
struct SelectSmem {
  union {
    uint32_t hist[4096];
    uint64_t buf[kSelCap];
  };
  uint32_t bcast[8];
  uint32_t wsum[16];   // per-wavefront totals of find_boundary (<= 1,024 threads)
  uint32_t count;
};

// Find, in hist[0..nb), the highest bin bb with above + sum(hist[bb..]) >= k.
// Writes bb and the count strictly above it (plus `above`) to sm.bcast[0..1].
// Thread t sums the bins [t per, (t + 1) per); a suffix scan over the threads
// (within each wavefront by shuffles, then over the wavefronts' totals)
// gives every thread the count above its bins, and the one thread whose
// bins hold the boundary walks them.  nb and blockDim.x are powers of two.
__device__ __forceinline__ void find_boundary(SelectSmem &sm, int nb, uint32_t above, uint32_t k) {
  __syncthreads();
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int nt = blockDim.x;
  const int per = nb >= nt ? nb / nt : 1;
  const int lo = t * per;
  const bool active = lo < nb;
  uint32_t sum = 0;
  if (active)
    for (int b = lo; b < lo + per; ++b) sum += sm.hist[b];
  uint32_t incl = sum;   // inclusive suffix scan (higher threads hold higher bins)
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t v = __shfl_down(incl, off, 64);
    if (lane + off < 64) incl += v;
  }
  if (lane == 0) sm.wsum[wave] = incl;
  if (t == 0) {
    sm.bcast[0] = 0u;
    sm.bcast[1] = above;
  }
  __syncthreads();
  uint32_t after = 0;
  for (int w = wave + 1; w < (nt + 63) / 64; ++w) after += sm.wsum[w];
  incl += after + above;
  const uint32_t excl = incl - sum;
  if (active && excl < k && incl >= k) {
    uint32_t acc = excl;
    int bb = lo;
    for (int b = lo + per - 1; b >= lo; --b) {
      if (acc + sm.hist[b] >= k) {
        bb = b;
        break;
      }
      acc += sm.hist[b];
    }
    sm.bcast[0] = uint32_t(bb);
    sm.bcast[1] = acc;  // count strictly above bin bb
  }
  __syncthreads();
}

// Bitonic sort of buf[0..n) descending (buf holds at least the next power
// of two >= n entries).
__device__ __forceinline__ void sort_desc_buf(uint64_t *buf, int n) {
  int p2 = 1;
  while (p2 < n) p2 <<= 1;
  for (int i = n + threadIdx.x; i < p2; i += blockDim.x) buf[i] = 0ull;
  __syncthreads();
  for (int size = 2; size <= p2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < p2 / 2; i += blockDim.x) {
        const int lo = 2 * i - (i & (stride - 1));
        const int hi = lo + stride;
        const bool desc = ((lo & size) == 0);
        const uint64_t a = buf[lo], b = buf[hi];
        if ((a < b) == desc) {
          buf[lo] = b;
          buf[hi] = a;
        }
      }
      __syncthreads();
    }
  }
}

__device__ __forceinline__ void sort_desc(SelectSmem &sm, int n) { sort_desc_buf(sm.buf, n); }

__device__ __forceinline__ uint64_t composite(uint32_t key, int32_t id) {
  return (uint64_t(key) << 32) | uint64_t(0xffffffffu - uint32_t(id));
}

// Calls f(key, i) for every element; each thread first loads U keys with
// branch-free (clamped) loads so that U global loads are in flight at once.
template <int U, class F>
__device__ __forceinline__ void for_each_key(const float *__restrict__ vals, int n, F f) {
  const int nt = blockDim.x;
  for (int base = threadIdx.x; base < n; base += nt * U) {
    uint32_t key[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = base + u * nt;
      key[u] = order_key(vals[i < n ? i : n - 1]);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = base + u * nt;
      if (i < n) f(key[u], i);
    }
  }
}

// Sorts the collected survivors and writes the k best (padding when fewer).
// The k best of buf[0..cnt) (cnt <= blockDim.x, composites as above) in
// (score desc, id asc) order, (-inf, -1) padded: one entry per thread, whose
// rank is the number of entries ahead of it (equal composites ordered by
// slot).  One pass instead of a sort's barrier-separated stages.
__device__ __forceinline__ void rank_emit(const uint64_t *buf, int cnt, int k,
                                          float *__restrict__ out_s, int32_t *__restrict__ out_i) {
  const int t = threadIdx.x;
  if (t < cnt) {
    const uint64_t e = buf[t];
    int r = 0;
    for (int j = 0; j < cnt; ++j) {
      const uint64_t v = buf[j];
      r += (v > e) || (v == e && j < t);
    }
    if (r < k) {
      out_s[r] = key_to_float(uint32_t(e >> 32));
      out_i[r] = int32_t(0xffffffffu - uint32_t(e & 0xffffffffu));
    }
  }
  for (int j = cnt + t; j < k; j += blockDim.x) {
    out_s[j] = -__builtin_inff();
    out_i[j] = -1;
  }
}

__device__ __forceinline__ void emit_sorted(SelectSmem &sm, int cnt, int k, float *__restrict__ out_s,
                                            int32_t *__restrict__ out_i) {
  if (cnt <= int(blockDim.x)) {
    __syncthreads();   // the entries written by other threads are visible
    rank_emit(sm.buf, cnt, k, out_s, out_i);
    return;
  }
  sort_desc(sm, cnt);
  for (int j = threadIdx.x; j < k; j += blockDim.x) {
    if (j < cnt) {
      const uint64_t c = sm.buf[j];
      out_s[j] = key_to_float(uint32_t(c >> 32));
      out_i[j] = int32_t(0xffffffffu - uint32_t(c & 0xffffffffu));
    } else {
      out_s[j] = -__builtin_inff();
      out_i[j] = -1;
    }
  }
}

// Threshold from a strided sample: the key that about 8 k elements of the
// array exceed.  Collecting every element at or above it is exact whenever
// at least k and at most kSelCap elements qualify; the caller checks.
__device__ __forceinline__ uint32_t sample_threshold(const float *__restrict__ vals, int n, int k,
                                                     SelectSmem &sm, int target = 0) {
  constexpr int S = 1024;
  for (int i = threadIdx.x; i < S; i += blockDim.x) {
    const int idx = int((int64_t(i) * n) / S);
    sm.buf[i] = uint64_t(order_key(vals[idx]));
  }
  __syncthreads();
  sort_desc(sm, S);
  if (target <= 0) target = 8 * k;
  int64_t r = (int64_t(target) * S + n - 1) / n;
  if (r < 1) r = 1;
  if (r > S) r = S;
  const uint32_t t = uint32_t(sm.buf[r - 1]);
  __syncthreads();
  return t;
}

template <class IdFn>
__device__ void block_topk(const float *__restrict__ vals, int n, int k, IdFn idfn,
                           float *__restrict__ out_s, int32_t *__restrict__ out_i,
                           SelectSmem &sm) {
  const int tid = threadIdx.x, nt = blockDim.x;
  if (n > kSelCap && int64_t(32) * k <= n) {
    // fast path: one pass collecting the elements above a sampled threshold
    const uint32_t thr = sample_threshold(vals, n, k, sm);
    if (tid == 0) sm.count = 0;
    __syncthreads();
    for_each_key<8>(vals, n, [&](uint32_t key, int i) {
      if (key >= thr) {
        const uint32_t pos = atomicAdd(&sm.count, 1u);
        if (pos < uint32_t(kSelCap)) sm.buf[pos] = composite(key, idfn(i));
      }
    });
    __syncthreads();
    const uint32_t cnt = sm.count;
    __syncthreads();
    if (cnt >= uint32_t(k) && cnt <= uint32_t(kSelCap)) {
      emit_sorted(sm, int(cnt), k, out_s, out_i);
      return;
    }
    // otherwise fall through to the exact radix selection
  }
  uint32_t lo_key = 0;         // collect keys >= lo_key (when not tie mode)
  bool tie_mode = false;
  uint32_t tie_key = 0, id_limit = 0;
  if (n > kSelCap) {
    uint32_t prefix = 0, above = 0;
    int pbits = 0;
    const int digits[3] = {12, 12, 8};
    bool fits = false;
    for (int di = 0; di < 3 && !fits; ++di) {
      const int d = digits[di];
      const int nb = 1 << d;
      const int shift = 32 - pbits - d;
      for (int b = tid; b < nb; b += nt) sm.hist[b] = 0;
      __syncthreads();
      for_each_key<8>(vals, n, [&](uint32_t key, int) {
        if (pbits == 0 || (key >> (32 - pbits)) == prefix)
          atomicAdd(&sm.hist[(key >> shift) & (nb - 1)], 1u);
      });
      find_boundary(sm, nb, above, uint32_t(k));
      const uint32_t bb = sm.bcast[0];
      const uint32_t cnt_b = sm.hist[bb];
      above = sm.bcast[1];
      prefix = (prefix << d) | bb;
      pbits += d;
      if (above + cnt_b <= uint32_t(kSelCap)) fits = true;
      __syncthreads();
    }
    if (fits) {
      lo_key = prefix << (32 - pbits);
    } else {
      // > capacity elements share the exact key `prefix`: pick the smallest
      // ids among them by a radix select over the 31-bit id.
      tie_mode = true;
      tie_key = prefix;
      const uint32_t need = uint32_t(k) - above;
      uint32_t ip = 0, iabove = 0;   // here "above" counts smaller ids
      int ibits = 1;                 // ids are < 2^31: top bit is 0
      const int idig[3] = {11, 10, 10};
      for (int di = 0; di < 3; ++di) {
        const int d = idig[di];
        const int nb = 1 << d;
        const int shift = 32 - ibits - d;
        for (int b = tid; b < nb; b += nt) sm.hist[b] = 0;
        __syncthreads();
        for_each_key<8>(vals, n, [&](uint32_t key, int i) {
          if (key != tie_key) return;
          // reverse the order so that "highest bin" means smallest id
          const uint32_t rid = 0x7fffffffu - uint32_t(idfn(i));
          if ((rid >> (32 - ibits)) == ip) atomicAdd(&sm.hist[(rid >> shift) & (nb - 1)], 1u);
        });
        find_boundary(sm, nb, iabove, need);
        const uint32_t bb = sm.bcast[0];
        iabove = sm.bcast[1];
        ip = (ip << d) | bb;
        ibits += d;
        __syncthreads();
      }
      id_limit = 0x7fffffffu - ip;   // collect ties with id <= id_limit
    }
  }
  // collect
  if (tid == 0) sm.count = 0;
  __syncthreads();
  for_each_key<8>(vals, n, [&](uint32_t key, int i) {
    bool take;
    int32_t id = 0;
    if (n <= kSelCap) {
      take = true;
    } else if (!tie_mode) {
      take = key >= lo_key;
    } else if (key > tie_key) {
      take = true;
    } else if (key == tie_key) {
      id = idfn(i);
      take = uint32_t(id) <= id_limit;
    } else {
      take = false;
    }
    if (take) {
      if (!(tie_mode && key == tie_key)) id = idfn(i);
      const uint32_t pos = atomicAdd(&sm.count, 1u);
      if (pos < uint32_t(kSelCap)) sm.buf[pos] = composite(key, id);
    }
  });
  __syncthreads();
  int cnt = int(sm.count);
  if (cnt > kSelCap) cnt = kSelCap;  // cannot happen: the selection above bounds it
  emit_sorted(sm, cnt, k, out_s, out_i);
}

}  // namespace rslm
