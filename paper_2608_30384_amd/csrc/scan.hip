// Second-stage IVF scan with per-query top-k.
//
// Scoring (paper, Section "Relative Quantization", local/global scaling, and
// Section "Performance Impact and Memory Savings", scoring in the rotated
// space): for query q and candidate x of probed list p
//   score = g^_x (<q, c_p> + s^_x sum_j <q_rot[j g:(j+1) g], C[code_{x,j}]>).
//
// GPU design.  All (query, list) pairs of a batch are grouped by list, so a
// list is streamed from HBM once per group of up to 8 queries instead of once
// per query.  For such a group the residual term is a dense contraction
// [8 queries x D] . [D x candidates] once the codes are decoded to their
// centroid values, so it runs on the matrix cores: v_mfma_f32_16x16x32_f16
// with the 16 A rows = 8 queries x (hi, lo) float16 halves of the rotated
// query (hi + lo carries ~22 significant bits), and B = 16 candidates x 32
// coordinates of decoded centroids.  Centroids are float16-exact, so the
// products are exact and accumulate in float32.  Codes are decoded through
// an LDS table indexed by a whole code symbol (a byte = two 4-bit codes for
// 4-bit codecs), replicated once per lane so the 64 lanes of a read always
// hit 64 different banks.  The code layout in HBM ("tiles" of 16 records)
// is arranged so that each lane's share of a tile is contiguous in 16-byte
// units and a wavefront's load is 1 KiB contiguous.
//
// Scheduling.  A work item is (list, group of <= 8 queries, chunk of the
// list); lists are cut into equal chunks of at most 2,048 candidates and the
// items are ordered by decreasing size.  A persistent grid (two 256-thread
// workgroups per CU) takes items from atomic counters, so the launch ends on
// the smallest items.  The counters are per XCD: blocks of consecutive items
// (the query groups that stream the same chunk of a list are consecutive)
// go to one XCD's queue, so those groups read the chunk through the same L2;
// a workgroup whose queue is empty takes items from the others.  Within an item each wavefront scores every fourth
// tile with the next tile's codes in flight; all loads are range-checked
// buffer loads, so no load is conditional and the compiler's wait counts
// stay exact.
//
// Above 32 chunks (D > 1,024) the A operands of all chunks no longer fit in
// registers: an item is scored in passes over equal chunk ranges, each pass
// adding its part of the residual dot to the candidate's score slot and the
// last one applying the scales (Rslm4Lite: read again from chunk 0's code
// word).
//
// Scores of every candidate are written to a per-query region of the
// workspace; a second kernel selects each query's top-k exactly (radix
// select, then a bitonic sort of the survivors) and maps positions to ids.
#include "rslm_internal.h"
#include "select_dev.h"

#include <hip/hip_ext.h>

#include <type_traits>

namespace rslm {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kChunkCands = 2048;   // candidates per work item
constexpr int kGroupQ = 8;          // queries per work item (16 MFMA rows / 2)
constexpr int kScanThreads = 256;
constexpr int kScaleRegs = kChunkCands / 256;   // scale words per lane: 4 tiles of a wave each
// Work queues: one per XCD (accelerator complex die, each with its own L2).
// Queue x holds the blocks of kQueueBlock consecutive items (in the global
// order) whose block number is x modulo kQueues; its counter sits in its
// own 64-byte line of the workspace.
constexpr int kQueues = 8;
constexpr int kQueueShift = 4;
constexpr int kQueueBlock = 1 << kQueueShift;
constexpr int kQueueStride = 16;   // int32 words between two queue counters
static_assert(kChunkCands / 16 <= 4 * 4 * kScaleRegs, "scale registers of a wave's tiles");

static size_t align256(size_t b) { return (b + 255) / 256 * 256; }

struct ScanWs {
  _Float16 *qh, *ql;
  float *qinv;
  int32_t *counts, *cursor, *pair_off, *item_off;
  int32_t *pairs, *prefix, *totals;
  int4 *items;            // two int4 per work item (see k_plan_items)
  int32_t *work;          // per-XCD queue counters of the scan (dynamic schedule)
  float *scores;
  int64_t stride;
  size_t bytes;
};

static ScanWs scan_ws_layout(void *base, int Q, int nprobe, int nlist, int d_pad,
                             int max_list, int k) {
  ScanWs w{};
  char *p = static_cast<char *>(base);
  size_t off = 0;
  auto take = [&](size_t b) {
    char *r = p ? p + off : nullptr;
    off += align256(b);
    return r;
  };
  w.qh = reinterpret_cast<_Float16 *>(take(size_t(Q) * d_pad * 2));
  w.ql = reinterpret_cast<_Float16 *>(take(size_t(Q) * d_pad * 2));
  w.qinv = reinterpret_cast<float *>(take(size_t(Q) * 4));
  w.counts = reinterpret_cast<int32_t *>(take(size_t(nlist) * 4));
  w.cursor = reinterpret_cast<int32_t *>(take(size_t(nlist) * 4));
  w.pair_off = reinterpret_cast<int32_t *>(take(size_t(nlist + 1) * 4));
  w.item_off = reinterpret_cast<int32_t *>(take(size_t(nlist + 1) * 4));
  w.pairs = reinterpret_cast<int32_t *>(take(size_t(Q) * nprobe * 4));
  w.prefix = reinterpret_cast<int32_t *>(take(size_t(Q) * nprobe * 4));
  w.totals = reinterpret_cast<int32_t *>(take(size_t(Q) * 4));
  w.work = reinterpret_cast<int32_t *>(take(kQueues * kQueueStride * 4));
  {
    // work items <= (groups of <= 8 queries) x (chunks of the longest list);
    // groups <= npairs / 8 + (number of probed lists)
    const int64_t npairs = int64_t(Q) * nprobe;
    const int64_t groups = npairs / kGroupQ + std::min<int64_t>(nlist, npairs);
    const int64_t chunks = std::max<int64_t>(1, (int64_t(max_list) + kChunkCands - 1) / kChunkCands);
    w.items = reinterpret_cast<int4 *>(take(size_t(groups * chunks) * 2 * sizeof(int4)));
  }
  w.stride = (int64_t(nprobe) * max_list + 63) / 64 * 64;
  w.scores = reinterpret_cast<float *>(take(size_t(Q) * size_t(w.stride) * 4));
  (void)k;
  w.bytes = off;
  return w;
}

// ------------------------------------------------------------- query prep
// q_rot (Q x D) -> per-query power-of-two scale so that max |q| * scale lies
// in [2^14, 2^15), then float16 hi = rne(q * scale), lo = rne(q * scale - hi).
// One wavefront per query.
__device__ __forceinline__ void prep_query(const float *__restrict__ q, int row, int D, int d_pad,
                                           _Float16 *__restrict__ qh, _Float16 *__restrict__ ql,
                                           float *__restrict__ qinv) {
  const int lane = threadIdx.x & 63;
  const float *qr = q + int64_t(row) * D;
  float m = 0.f;
  for (int i = lane; i < D; i += 64) m = fmaxf(m, fabsf(qr[i]));
  m = wave_max(m);
  float scale = 1.f;
  if (m > 0.f) {
    const int e = ilogbf(m) + 1;  // m in [2^(e-1), 2^e)
    scale = ldexpf(1.f, 15 - e);
  }
  for (int i = lane; i < d_pad; i += 64) {
    const float v = (i < D) ? qr[i] * scale : 0.f;
    const _Float16 h = static_cast<_Float16>(v);
    const _Float16 l = static_cast<_Float16>(v - static_cast<float>(h));
    qh[int64_t(row) * d_pad + i] = h;
    ql[int64_t(row) * d_pad + i] = l;
  }
  if (lane == 0) qinv[row] = 1.f / scale;
}

// ------------------------------------------------------------- planning
// Two kernels.  The first prepares the queries and, per query, the exclusive
// prefix of its probed list sizes (where its scores go); its last workgroup
// counts the (query, list) pairs per list, scans the counts into pair_off and
// places each list's work items in an order by decreasing item size.  The
// second groups the pairs by list and writes the work item descriptors.

// One wavefront per query: exclusive prefix over its probes of the (clamped)
// probed list sizes.
__device__ __forceinline__ void query_prefix(const int32_t *__restrict__ probe_ids, int q,
                                             int nprobe, int nlist,
                                             const int32_t *__restrict__ sizes, int max_list,
                                             int32_t *__restrict__ prefix,
                                             int32_t *__restrict__ totals) {
  const int lane = threadIdx.x & 63;
  int carry = 0;
  for (int p0 = 0; p0 < nprobe; p0 += 64) {
    const int p = p0 + lane;
    int sz = 0;
    if (p < nprobe) {
      const int L = probe_ids[int64_t(q) * nprobe + p];
      if (L >= 0 && L < nlist) sz = max(0, min(sizes[L], max_list));
    }
    int incl = sz;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int t = __shfl_up(incl, off, 64);
      if (lane >= off) incl += t;
    }
    if (p < nprobe) prefix[int64_t(q) * nprobe + p] = carry + incl - sz;
    carry += __shfl(incl, 63, 64);
  }
  if (lane == 0) totals[q] = carry;
}

// Candidates per work item of a list of sz > 0 candidates: the list is split
// into the fewest chunks of at most kChunkCands, of equal size rounded up to
// whole tiles, so the items of a list have (almost) equal work.
__device__ __forceinline__ int item_cands(int sz) {
  const int nch = (sz + kChunkCands - 1) / kChunkCands;
  return ((sz + nch - 1) / nch + 15) & ~15;
}
constexpr int kSizeClasses = kChunkCands / 16;   // item size class = cands / 16 - 1
static_assert(kSizeClasses == 128, "the class-start scan takes two classes per lane");
constexpr int kPlanThreads = 1024;
constexpr int kPlanQueries = kPlanThreads / 64;   // queries per preparing workgroup
constexpr int kPlanRange = 16384;                 // lists counted per pass in LDS
static_assert(kPlanRange / kPlanThreads == 16, "per-thread list batch");

// Work items of a list with cp pairs and `size` candidates (groups of <= 8
// queries x chunks) and their size class.
__device__ __forceinline__ int list_items(int cp, int size, int max_list, int &cls) {
  const int sz = max(0, min(size, max_list));
  if (cp <= 0 || sz <= 0) return 0;
  const int ic = item_cands(sz);
  cls = ic / 16 - 1;
  return ((cp + kGroupQ - 1) / kGroupQ) * ((sz + ic - 1) / ic);
}

struct PlanSmem {
  int32_t cnt[kPlanRange];
  int32_t part[kPlanThreads / 64];   // per-wavefront totals
  int32_t hist[kSizeClasses], start[kSizeClasses];
};

// The planning workgroup: pair counts per list (LDS histogram, lists in
// passes of kPlanRange), their exclusive scan (pair_off), cursor = 0, and
// each list's first work item in an order by decreasing item size (counting
// sort over size classes; the order within a class is immaterial: every item
// writes its own scores).  Also resets the scan's queue counters.  Until the
// class starts are known, item_off[L] holds the list's item count.
__device__ void plan_lists(PlanSmem &sm, const int32_t *__restrict__ probe_ids, int npairs,
                           const int32_t *__restrict__ sizes, int nlist, int max_list,
                           int32_t *__restrict__ counts, int32_t *__restrict__ pair_off,
                           int32_t *__restrict__ item_off, int32_t *__restrict__ cursor,
                           int32_t *__restrict__ work) {
  const int t = threadIdx.x;
  if (t < kSizeClasses) sm.hist[t] = 0;
  int carry = 0;   // uniform: pairs of the lists before this pass
  for (int L0 = 0; L0 < nlist; L0 += kPlanRange) {
    const int nr = min(kPlanRange, nlist - L0);
    for (int i = t; i < nr; i += kPlanThreads) sm.cnt[i] = 0;
    __syncthreads();
    // batches of 16 pairs per thread: all loads issued before the atomics
    for (int base = 0; base < npairs; base += 16 * kPlanThreads) {
      int Ls[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int i = base + u * kPlanThreads + t;
        Ls[u] = i < npairs ? probe_ids[i] : -1;
      }
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (Ls[u] >= L0 && Ls[u] < L0 + nr) atomicAdd(&sm.cnt[Ls[u] - L0], 1);
    }
    __syncthreads();
    // thread t owns the consecutive lists [a, b) of the pass (at most
    // kPlanRange / kPlanThreads = 16); their sizes are loaded first
    const int per = (nr + kPlanThreads - 1) / kPlanThreads;
    const int a = min(nr, t * per), b = min(nr, a + per);
    int szv[kPlanRange / kPlanThreads];
#pragma unroll
    for (int u = 0; u < kPlanRange / kPlanThreads; ++u) szv[u] = a + u < b ? sizes[L0 + a + u] : 0;
    int sum = 0;
#pragma unroll
    for (int u = 0; u < kPlanRange / kPlanThreads; ++u) {
      if (a + u >= b) break;
      const int cp = sm.cnt[a + u];
      sum += cp;
      int cls = 0;
      const int ni = list_items(cp, szv[u], max_list, cls);
      if (ni > 0) atomicAdd(&sm.hist[cls], ni);
      item_off[L0 + a + u] = ni;
    }
    // exclusive prefix of the threads' sums: an inclusive scan within each
    // wavefront by shuffles, then the totals of the wavefronts before it
    const int lane = t & 63, wv = t >> 6;
    int incl = sum;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int v = __shfl_up(incl, off, 64);
      if (lane >= off) incl += v;
    }
    if (lane == 63) sm.part[wv] = incl;
    __syncthreads();
    int before = 0, total = 0;
    for (int w = 0; w < kPlanThreads / 64; ++w) {
      const int v = sm.part[w];
      before += w < wv ? v : 0;
      total += v;
    }
    int run = carry + before + incl - sum;
    for (int i = a; i < b; ++i) {
      const int cp = sm.cnt[i];
      counts[L0 + i] = cp;
      cursor[L0 + i] = 0;
      pair_off[L0 + i] = run;
      run += cp;
    }
    carry += total;
    __syncthreads();
  }
  if (t < 64) {
    // class starts in decreasing class order: lane t takes classes 127 - 2t
    // and 126 - 2t, an inclusive scan of their sums over the wavefront
    const int c0 = kSizeClasses - 1 - 2 * t;
    const int h0 = sm.hist[c0], h1 = sm.hist[c0 - 1];
    int incl = h0 + h1;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int v = __shfl_up(incl, off, 64);
      if (t >= off) incl += v;
    }
    sm.start[c0] = incl - h0 - h1;
    sm.start[c0 - 1] = incl - h1;
    if (t == 63) {
      pair_off[nlist] = carry;
      item_off[nlist] = incl;
    }
  }
  if (t < kQueues) work[t * kQueueStride] = 0;
  __syncthreads();   // item_off[L] written above is read back by this workgroup
  for (int base = 0; base < nlist; base += 16 * kPlanThreads) {   // loads first
    int niv[16], szv[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int L = base + u * kPlanThreads + t;
      niv[u] = L < nlist ? item_off[L] : 0;
      szv[u] = L < nlist ? sizes[L] : 0;
    }
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int L = base + u * kPlanThreads + t;
      if (L >= nlist) break;
      // a list with items has 0 < size; its class depends on the size only
      const int cls = item_cands(max(1, min(szv[u], max_list))) / 16 - 1;
      item_off[L] = niv[u] > 0 ? atomicAdd(&sm.start[cls], niv[u]) : 0;
    }
  }
}

// Block 0 plans the lists (the longest chain, so it is dispatched first);
// blocks [1, n_qblocks + 1) prepare kPlanQueries queries each (prep + prefix).
__global__ void __launch_bounds__(kPlanThreads) k_plan_a(
    const float *__restrict__ q_rot, int Q, int D, int d_pad, _Float16 *__restrict__ qh,
    _Float16 *__restrict__ ql, float *__restrict__ qinv, const int32_t *__restrict__ probe_ids,
    int nprobe, int nlist, const int32_t *__restrict__ sizes, int max_list,
    int32_t *__restrict__ prefix, int32_t *__restrict__ totals, int32_t *__restrict__ counts,
    int32_t *__restrict__ pair_off, int32_t *__restrict__ item_off, int32_t *__restrict__ cursor,
    int32_t *__restrict__ work) {
  __shared__ PlanSmem sm;
  if (blockIdx.x == 0) {
    plan_lists(sm, probe_ids, Q * nprobe, sizes, nlist, max_list, counts, pair_off, item_off,
               cursor, work);
    return;
  }
  const int q = (blockIdx.x - 1) * kPlanQueries + (threadIdx.x >> 6);
  if (q >= Q) return;
  prep_query(q_rot, q, D, d_pad, qh, ql, qinv);
  query_prefix(probe_ids, q, nprobe, nlist, sizes, max_list, prefix, totals);
}

// Threads [0, npairs): pair i joins its list's group (pairs[] grouped by
// list, slots from a per-list cursor).  Wavefront L (< nlist) writes the
// descriptors of list L's work items from item_off[L] on, one item per lane,
// chunk-major: the groups that stream the same chunk are consecutive items,
// so they land in the same XCD queue and their reads share that L2.
// Item = (group of <= 8 consecutive pairs of the list, chunk of
// item_cands(size) candidates):
//   d0 = {list, first candidate, candidate count, first pair (in pairs[])}
//   d1 = {queries in the group, first record (low, high word), 0}
constexpr int kPlanBThreads = 256;

__global__ void __launch_bounds__(kPlanBThreads) k_plan_b(
    const int32_t *__restrict__ probe_ids, int npairs, int nlist,
    const int32_t *__restrict__ counts, const int32_t *__restrict__ sizes,
    const int64_t *__restrict__ list_offsets, int max_list, const int32_t *__restrict__ pair_off,
    const int32_t *__restrict__ item_off, int32_t *__restrict__ cursor,
    int32_t *__restrict__ pairs, int4 *__restrict__ items) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < npairs) {
    const int L = probe_ids[i];
    if (L >= 0 && L < nlist) pairs[pair_off[L] + atomicAdd(&cursor[L], 1)] = i;
  }
  const int L = i >> 6, lane = i & 63;
  if (L >= nlist) return;
  const int c = counts[L];
  const int sz = max(0, min(sizes[L], max_list));
  if (c <= 0 || sz <= 0) return;
  const int ic = item_cands(sz);
  const int nch = (sz + ic - 1) / ic;
  const int ngr = (c + kGroupQ - 1) / kGroupQ;
  const int it0 = item_off[L];
  const int64_t lo = list_offsets[L];
  for (int t = lane; t < ngr * nch; t += 64) {
    const int ch = t / ngr, g = t - ch * ngr;
    const int cand0 = ch * ic;
    const int64_t rec0 = lo + cand0;
    const int64_t it = it0 + t;
    items[2 * it] = make_int4(L, cand0, min(sz - cand0, ic), pair_off[L] + g * kGroupQ);
    items[2 * it + 1] = make_int4(min(kGroupQ, c - g * kGroupQ), int(uint32_t(rec0)),
                                  int(uint32_t(uint64_t(rec0) >> 32)), 0);
  }
}

// ------------------------------------------------------------- scan kernel
// Index of the XCD (0..7) this wavefront runs on, from the hardware register.
__device__ __forceinline__ int xcd_id() {
  uint32_t v;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
  return int(v & uint32_t(kQueues - 1));
}

// Global item of ticket j of queue x (blocks of kQueueBlock items dealt
// round-robin over the queues); increasing in j.
__device__ __forceinline__ int64_t queue_item(int x, uint32_t j) {
  return (int64_t(j >> kQueueShift) << (kQueueShift + 3)) | (int64_t(x) << kQueueShift) |
         int64_t(j & uint32_t(kQueueBlock - 1));
}
static_assert(kQueues == 8, "queue_item deals blocks over 8 queues");
struct ScanArgs {
  const int64_t *list_offsets;
  const int32_t *list_sizes;
  const uint8_t *codes;
  const uint32_t *scales;
  const uint32_t *dtab;       // compact decode table
  const _Float16 *qh, *ql;
  const float *qinv;
  const float *probe_dots;
  const int32_t *item_off, *pairs, *prefix;
  const int4 *items;
  int32_t *work;
  float *scores;
  int64_t stride;
  int nlist, nprobe, d_pad, n_chunks, tile_bytes, lane_units, max_list;
  int n_pass;             // passes over ranges of NC chunks (NC * n_pass = n_chunks)
  int lead;               // Rslm4Lite: leading coordinates on the K = 8 codebook (16 or 32)
  int global;             // Rslm4Lite: the global scale is embedded too
  float cb_lead[8];       // Rslm4Lite: the K = 8 codebook
};

// LDS decode table of a scan instantiation.  The plan ships a compact
// table: per symbol (a byte = two 4-bit codes; 6 bits = two 3-bit codes; a
// nibble = one 2-D or 4-D centroid for 2 and 1 bits) its float16 centroid
// values.  In LDS every entry is replicated once per lane of an LDS pass, so
// the lanes of a read always hit distinct banks: 64 copies for 32-bit reads.
// From 24 chunks up (where registers already limit the scan to two
// workgroups per CU) 2- and 1-bit codes are decoded by whole bytes: a byte
// of 2-bit codes is four coordinates (a 64-bit read, 32 copies), a byte of
// 1-bit codes eight (a 128-bit read, 16 copies), built in the kernel from the
// compact nibble table.  Entry e of copy l sits at byte e * 256 + l * 4 *
// kWords, so an address is one v_perm (except the nibble tables of 1-bit
// codes: 64 copies of two words, an entry stride of 512 bytes).
template <int BITS, int NC> struct DecodeTab {
  static constexpr bool kByte = BITS <= 2 && NC >= 24;
  static constexpr int kCompactWords = BITS == 1 ? 2 : 1;   // words per compact entry
  static constexpr int kCompactEntries = BITS == 4 ? 256 : BITS == 3 ? 64 : 16;
  static constexpr int kEntries = kByte ? 256 : kCompactEntries;
  static constexpr int kWords = kByte ? 2 * kCompactWords : kCompactWords;
  static constexpr int kCopies = kByte ? 64 / kWords : 64;
  static_assert(!kByte || kCopies * kWords * 4 == 256, "byte tables: entry stride of 256 bytes");
};

__device__ __forceinline__ uint32_t lds_word(const uint32_t *tab, uint32_t byte_addr) {
  return *reinterpret_cast<const uint32_t *>(reinterpret_cast<const char *>(tab) + byte_addr);
}
__device__ __forceinline__ uint2 lds_dword2(const uint32_t *tab, uint32_t byte_addr) {
  return *reinterpret_cast<const uint2 *>(reinterpret_cast<const char *>(tab) + byte_addr);
}
__device__ __forceinline__ uint4 lds_dword4(const uint32_t *tab, uint32_t byte_addr) {
  return *reinterpret_cast<const uint4 *>(reinterpret_cast<const char *>(tab) + byte_addr);
}

// Bits of chunk c (8 coordinates of this lane) from the lane's stream words.
template <int BITS>
__device__ __forceinline__ uint32_t chunk_bits(const uint32_t *sw, int c) {
  if (BITS == 4) return sw[c];
  if (BITS == 2) return (sw[c >> 1] >> (16 * (c & 1))) & 0xffffu;
  if (BITS == 1) return (sw[c >> 2] >> (8 * (c & 3))) & 0xffu;
  // BITS == 3: 24 bits at bit offset 24 c
  const int bo = 24 * c;
  const int wi = bo >> 5, sh = bo & 31;
  uint64_t v = sw[wi];
  if (sh > 8) v |= uint64_t(sw[wi + 1]) << 32;
  return uint32_t(v >> sh) & 0xffffffu;
}

// 4 and 3 bits: eight coordinates from their bits (one chunk of a lane).
template <int BITS>
__device__ __forceinline__ half8 decode8(const uint32_t *tab, uint32_t bits, uint32_t lane4) {
  union {
    uint32_t u[4];
    half8 h;
  } r;
  if constexpr (BITS == 4) {
    // symbol = byte i; LDS byte address = byte * 256 + lane * 4 (one v_perm)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      r.u[i] = lds_word(tab, __builtin_amdgcn_perm(bits, lane4, 0x0c0c0400u | ((4u + i) << 8)));
  } else {
    static_assert(BITS == 3, "1 and 2 bits decode in decode_chunk");
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t sym = (bits >> (6 * i)) & 63u;
      r.u[i] = lds_word(tab, (sym << 8) | lane4);
    }
  }
  return r.h;
}

// Decode chunk c of this lane's stream words sw.  1 and 2 bits read the
// codes straight from the stream word: with byte tables each address is one
// v_perm of a code byte; with nibble tables, for 1 bit each address is one
// bit-field extract and one shift-or (entry of nibble v at v * 512 + lane *
// 8), for 2 bits the low and high nibbles of a whole word are split into
// bytes once for the two chunks it holds, and each address is one v_perm.
template <int BITS, int NC, int W>
__device__ __forceinline__ half8 decode_chunk(const uint32_t *tab, const uint32_t (&sw)[W], int c,
                                              uint32_t lane4) {
  union {
    uint32_t u[4];
    half8 h;
  } r;
  if constexpr (DecodeTab<BITS, NC>::kByte && BITS == 2) {
    // bytes 2 (c & 1) and 2 (c & 1) + 1 of the word: coordinates 0-3, 4-7
    const uint32_t w = sw[c >> 1];
    const uint32_t lo = (lane4 & 124u) << 1;   // copy lane % 32, 8 bytes each
    const uint32_t b0 = 4u + 2u * uint32_t(c & 1);
    const uint2 e0 = lds_dword2(tab, __builtin_amdgcn_perm(w, lo, 0x0c0c0400u | (b0 << 8)));
    const uint2 e1 = lds_dword2(tab, __builtin_amdgcn_perm(w, lo, 0x0c0c0400u | ((b0 + 1u) << 8)));
    r.u[0] = e0.x;
    r.u[1] = e0.y;
    r.u[2] = e1.x;
    r.u[3] = e1.y;
    return r.h;
  } else if constexpr (DecodeTab<BITS, NC>::kByte && BITS == 1) {
    // byte c & 3 of the word: all eight coordinates
    const uint32_t w = sw[c >> 2];
    const uint32_t lo = (lane4 & 60u) << 2;   // copy lane % 16, 16 bytes each
    const uint4 e = lds_dword4(
        tab, __builtin_amdgcn_perm(w, lo, 0x0c0c0400u | ((4u + uint32_t(c & 3)) << 8)));
    r.u[0] = e.x;
    r.u[1] = e.y;
    r.u[2] = e.z;
    r.u[3] = e.w;
    return r.h;
  } else if constexpr (BITS == 2) {
    const uint32_t w = sw[c >> 1];
    const uint32_t t = w & 0x0f0f0f0fu, u = (w >> 4) & 0x0f0f0f0fu;
    const uint32_t b0 = 4u + 2u * uint32_t(c & 1);   // selector of the chunk's first byte
    r.u[0] = lds_word(tab, __builtin_amdgcn_perm(t, lane4, 0x0c0c0400u | (b0 << 8)));
    r.u[1] = lds_word(tab, __builtin_amdgcn_perm(u, lane4, 0x0c0c0400u | (b0 << 8)));
    r.u[2] = lds_word(tab, __builtin_amdgcn_perm(t, lane4, 0x0c0c0400u | ((b0 + 1u) << 8)));
    r.u[3] = lds_word(tab, __builtin_amdgcn_perm(u, lane4, 0x0c0c0400u | ((b0 + 1u) << 8)));
    return r.h;
  } else if constexpr (BITS == 1) {
    const uint32_t w = sw[c >> 2];
    const int s = 8 * (c & 3);
    const uint32_t lane8 = lane4 << 1;
    const uint32_t a0 = (((w >> s) & 0xfu) << 9) | lane8;
    const uint32_t a1 = (((w >> (s + 4)) & 0xfu) << 9) | lane8;
    const uint2 e0 = lds_dword2(tab, a0), e1 = lds_dword2(tab, a1);
    r.u[0] = e0.x;
    r.u[1] = e0.y;
    r.u[2] = e1.x;
    r.u[3] = e1.y;
    return r.h;
  } else {
    return decode8<BITS>(tab, chunk_bits<BITS>(sw, c), lane4);
  }
}

// Buffer resources (gfx9 format: 48-bit base, stride 0, byte range, data
// format word).  A raw buffer access past the range returns zeros (loads) or
// is dropped (stores) without touching memory, so prefetches of tiles beyond
// a work item need no branch.  Unconditional loads let the compiler count
// outstanding loads exactly, which keeps the prefetched tiles in flight.
constexpr int kRsrcWord3 = 0x00020000;
// s_waitcnt immediate (gfx9 encoding) waiting for vmcnt = 0 only
// (expcnt = 7 and lgkmcnt = 15 are "do not wait").
constexpr int kWaitVmcnt0 = 0x0F70;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, int(bytes),
                                           kRsrcWord3);
}

// Codes of local tile lt of a work item: this lane's 16-byte units.  The
// resource is rebuilt per tile in scalar registers (base advanced by lt
// tiles, range one tile, or zero past the item), so the per-lane offsets are
// loop invariant and the tile loop does no vector address arithmetic.
template <int W>
__device__ __forceinline__ void load_tile(uint32_t (&w)[W], const uint8_t *tiles, int lt,
                                          int n_tiles, uint32_t tile_bytes, uint32_t voff) {
  const __amdgpu_buffer_rsrc_t r =
      make_rsrc(tiles + int64_t(lt) * tile_bytes, lt < n_tiles ? tile_bytes : 0u);
#pragma unroll
  for (int u = 0; u < W / 4; ++u) {
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff + u * 1024u, 0, 0);
    w[4 * u + 0] = v.x;
    w[4 * u + 1] = v.y;
    w[4 * u + 2] = v.z;
    w[4 * u + 3] = v.w;
  }
}

// Decode one tile (16 candidates) and multiply it with the item's queries;
// lane (kq, m) ends with rows 4 kq + {0,1,2,3} of candidate column m, i.e.
// query slots 2 kq (hi, lo) and 2 kq + 1 (hi, lo).
// Rslm4Lite, chunk 0 of a lead lane: the nibbles' low three bits index the
// K = 8 codebook (a 256-entry table by byte symbol, not replicated: only this
// chunk of these lanes reads it), bit 3 is a scale bit.
__device__ __forceinline__ half8 decode8_lite(const uint32_t *ltab, uint32_t bits) {
  union {
    uint32_t u[4];
    half8 h;
  } r;
#pragma unroll
  for (int i = 0; i < 4; ++i) r.u[i] = ltab[(bits >> (8 * i)) & 0xffu];
  return r.h;
}

// The top bit of each nibble of a 32-bit word, packed: bit i = bit 4 i + 3.
__device__ __forceinline__ uint32_t nibble_tops(uint32_t w) {
  uint32_t t = 0u;
#pragma unroll
  for (int i = 0; i < 8; ++i) t |= ((w >> (4 * i + 3)) & 1u) << i;
  return t;
}

// MODE: 0 one pass over all chunks (score written); above 32 chunks the
// chunks are scored in passes and the raw residual dot of a candidate is
// kept in its score slot between them: 1 first pass (dot stored), 2 middle
// pass (added), 3 last pass (added, then the score written).
// Rslm4Lite: the scale word of candidate m from the chunk-0 code words of
// the four lanes holding it (bit 3 of each nibble: s^ in kq 0, 1, g^ in kq
// 2, 3).
__device__ __forceinline__ uint32_t lite_scales(uint32_t chunk0, int m, int global) {
  const uint32_t t = nibble_tops(chunk0);
  const uint32_t t0 = __shfl(int(t), m, 64), t1 = __shfl(int(t), 16 + m, 64);
  const uint32_t t2 = __shfl(int(t), 32 + m, 64), t3 = __shfl(int(t), 48 + m, 64);
  return (t0 | (t1 << 8)) | ((global ? (t2 | (t3 << 8)) : 0x7000u) << 16);
}

template <int BITS, int NC, int W, bool LITE = false, int MODE = 0>
__device__ __forceinline__ void score_tile(const uint32_t (&tw)[W], uint32_t sc,
                                           const half8 (&av)[NC], const uint32_t *dtab,
                                           uint32_t lane4, int lt, int n_cand, int m,
                                           const bool (&ok)[2],
                                           const float (&qc)[2], const float (&qi)[2],
                                           float *const (&out)[2],
                                           const uint32_t *ltab = nullptr, bool lead_lane = false,
                                           int global = 0) {
  // Decoding runs two chunks ahead of the matrix multiply so that the LDS
  // latency of chunk c + 2 overlaps the MFMAs of chunks c and c + 1; even and
  // odd chunks accumulate separately to halve the dependent MFMA chain.
  floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
  float prev[2] = {0.f, 0.f};     // dot of the earlier passes, loaded before the MFMAs
  if constexpr (MODE >= 2) {
    const int c = lt * 16 + m;
    if (c < n_cand) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
        if (ok[i]) prev[i] = out[i][c];
    }
  }
  half8 b[3];
  if (LITE && MODE <= 1) {
    // scales from the code stream: lane (kq, m) holds 8 scale bits of
    // candidate m in chunk 0 (kq 0, 1: s^; kq 2, 3: g^); in passes the last
    // one gets them from the caller, which reads chunk 0's word again
    if (MODE == 0) sc = lite_scales(chunk_bits<BITS>(tw, 0), m, global);
    b[0] = lead_lane ? decode8_lite(ltab, chunk_bits<BITS>(tw, 0))
                     : decode_chunk<BITS, NC>(dtab, tw, 0, lane4);
  } else {
    b[0] = decode_chunk<BITS, NC>(dtab, tw, 0, lane4);
  }
  if (NC > 1) b[1] = decode_chunk<BITS, NC>(dtab, tw, NC > 1 ? 1 : 0, lane4);
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    if (c + 2 < NC)
      b[(c + 2) % 3] = decode_chunk<BITS, NC>(dtab, tw, c + 2 < NC ? c + 2 : 0, lane4);
    if (c & 1) acc1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(av[c], b[c % 3], acc1, 0, 0, 0);
    else acc0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(av[c], b[c % 3], acc0, 0, 0, 0);
  }
  const floatx4 acc = acc0 + acc1;
  const int cand = lt * 16 + m;   // item-local candidate index
  if (cand < n_cand) {
    if (MODE == 0) {
      const float sh = dec_ue7m9(sc & 0xffffu);
      const float gh = dec_ue4m12(sc >> 16);
      if (ok[0]) out[0][cand] = gh * (qc[0] + sh * ((acc[0] + acc[1]) * qi[0]));
      if (ok[1]) out[1][cand] = gh * (qc[1] + sh * ((acc[2] + acc[3]) * qi[1]));
    } else {
      float d[2] = {acc[0] + acc[1], acc[2] + acc[3]};
      if (MODE >= 2) {
        d[0] += prev[0];
        d[1] += prev[1];
      }
      const float sh = dec_ue7m9(sc & 0xffffu);
      const float gh = dec_ue4m12(sc >> 16);
#pragma unroll
      for (int i = 0; i < 2; ++i)
        if (ok[i]) out[i][cand] = (MODE == 3) ? gh * (qc[i] + sh * (d[i] * qi[i])) : d[i];
    }
  }
}

// MP: the multi-pass variant (items scored in a.n_pass passes of NC chunks).
template <int BITS, int NC, bool LITE = false, bool MP = false>
__global__ void __launch_bounds__(kScanThreads, 2) k_scan(ScanArgs a) {
  using T = DecodeTab<BITS, NC>;
  __shared__ uint32_t dtab[T::kEntries * T::kCopies * T::kWords];
  __shared__ uint32_t ltab[LITE ? 256 : 1];
  if (LITE) {   // Rslm4Lite chunk-0 table: byte -> half2(C8[lo & 7], C8[hi & 7])
    const int e = threadIdx.x;   // kScanThreads == 256 entries
    const _Float16 lo = static_cast<_Float16>(a.cb_lead[e & 7]);
    const _Float16 hi = static_cast<_Float16>(a.cb_lead[(e >> 4) & 7]);
    uint16_t lb, hb;
    __builtin_memcpy(&lb, &lo, 2);
    __builtin_memcpy(&hb, &hi, 2);
    ltab[e] = uint32_t(lb) | (uint32_t(hb) << 16);
  }
  constexpr int kWordsPerLane = ((NC * BITS + 15) / 16) * 4;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar loop control
  const int nwaves = kScanThreads / 64;
  const uint32_t lane4 = uint32_t(lane) * 4u;

  // replicate the table: entry e of copy l at word (e * kCopies + l) *
  // kWords; a byte entry is the compact entries of its low and high nibbles.
  // Unrolled so that a batch of the (cached) table loads is in flight at
  // once: one load and its wait per iteration made the fill a chain of 64
  // dependent loads per thread at every launch.
#pragma unroll 16
  for (int idx = tid; idx < T::kEntries * T::kCopies; idx += kScanThreads) {
    const int e = idx / T::kCopies;
    if constexpr (T::kByte) {
      constexpr int cw = T::kCompactWords;
#pragma unroll
      for (int w = 0; w < cw; ++w) {
        dtab[idx * T::kWords + w] = a.dtab[(e & 15) * cw + w];
        dtab[idx * T::kWords + cw + w] = a.dtab[(e >> 4) * cw + w];
      }
    } else {
#pragma unroll
      for (int w = 0; w < T::kWords; ++w) dtab[idx * T::kWords + w] = a.dtab[e * T::kWords + w];
    }
  }
  __syncthreads();

  const int n_items = __builtin_amdgcn_readfirstlane(a.item_off[a.nlist]);
  const int m = lane & 15;           // A row / B column of this lane
  const int kq = lane >> 4;          // k-quarter: coordinates 8 kq .. 8 kq + 7 of a chunk
  // Dynamic schedule: a workgroup takes items (largest first) from the queue
  // of its XCD, and once that is empty from the other queues in turn (a
  // queue whose ticket maps past the last item stays empty).  Thread 0 keeps
  // the queue state.  The ticket for the next item is drawn when an item
  // starts and published in LDS after its tiles are scored (by then the
  // atomic has returned), in one of two slots: a slot is rewritten only two
  // barriers after it was read.
  __shared__ int s_ticket[2];
  int q_cur = xcd_id(), q_tried = 0;
  // atomicInc (not add): left alone by the compiler's wave-aggregation
  // rewrite, which would wait for the returned value where it is issued
  auto draw = [&](int x) {
    return uint32_t(atomicInc(reinterpret_cast<unsigned *>(a.work + x * kQueueStride), 0x7fffffffu));
  };
  // item of ticket j of the current queue, moving on to the next queues
  // while the current one is empty; n_items when every queue is
  auto resolve = [&](uint32_t j) {
    int64_t it = queue_item(q_cur, j);
    while (it >= n_items && ++q_tried < kQueues) {
      q_cur = (q_cur + 1) & (kQueues - 1);
      it = queue_item(q_cur, draw(q_cur));
    }
    return int(it < n_items ? it : n_items);
  };
  if (tid == 0) s_ticket[0] = resolve(draw(q_cur));
  __syncthreads();
  int k_it = 0;
  for (int item = __builtin_amdgcn_readfirstlane(s_ticket[0]); item < n_items;
       ++k_it, item = __builtin_amdgcn_readfirstlane(s_ticket[k_it & 1])) {
    uint32_t next_ticket = 0;
    if (tid == 0) next_ticket = draw(q_cur);
    // The descriptor is the same for the whole wavefront: readfirstlane keeps
    // every item-level quantity (and so the buffer resources and the tile
    // loop) in scalar registers.
    const int4 d0 = a.items[2 * int64_t(item)];
    const int4 d1 = a.items[2 * int64_t(item) + 1];
    const int cand0 = __builtin_amdgcn_readfirstlane(d0.y);
    const int n_cand = __builtin_amdgcn_readfirstlane(d0.z);
    const int pbase = __builtin_amdgcn_readfirstlane(d0.w);
    const int G = __builtin_amdgcn_readfirstlane(d1.x);
    const int64_t rec0 = int64_t((uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(d1.z))) << 32) |
                                 uint32_t(__builtin_amdgcn_readfirstlane(d1.y)));

    const int n_tiles = (n_cand + 15) / 16;
    // lists start on a tile boundary and cand0 is a multiple of 16
    const uint8_t *tiles = a.codes + (rec0 >> 4) * a.tile_bytes;
    const uint32_t tb = uint32_t(a.tile_bytes);
    // Scale words.  Up to 24 chunks: every tile this wave scores (tile lt =
    // wave + 4 j, j < 32) has its scales loaded before any code tile, lane
    // (kq, m) holding candidate m of tiles j = kq + 4 r; issued first, they
    // never make the tile loop wait for code tiles still in flight.  With 32
    // chunks the registers are short: each tile's scale word is loaded with
    // its codes instead and shares their wait.
    // (Rslm4Lite: the scales are in the code stream; no scales array read.)
    constexpr bool kPreload = NC < 32;
    const __amdgpu_buffer_rsrc_t rs =
        make_rsrc(LITE ? static_cast<const void *>(a.codes) : static_cast<const void *>(a.scales + rec0),
                  LITE ? 0u : uint32_t(n_cand) * 4u);
    uint32_t sreg[kPreload ? kScaleRegs : 1];
#pragma unroll
    for (int r = 0; r < (kPreload ? kScaleRegs : 1); ++r)
      sreg[r] = (LITE || !kPreload) ? 0u : __builtin_amdgcn_raw_buffer_load_b32(
                                rs, uint32_t((wave + nwaves * (kq + 4 * r)) * 16 + m) * 4u, 0, 0);
    auto load_scale = [&](int t) {
      return (LITE || kPreload) ? 0u
                                : __builtin_amdgcn_raw_buffer_load_b32(rs, uint32_t(t * 16 + m) * 4u, 0, 0);
    };
    // single pass: the wave's first code tile is issued here, ahead of the
    // dependent query loads below, so that it arrives while they do
    uint32_t bufA[MP ? 1 : kWordsPerLane];
    uint32_t scA = 0u;
    const uint32_t voff = uint32_t(lane) * 16u;
    if constexpr (!MP) {
      load_tile(bufA, tiles, wave, n_tiles, tb, voff);
      scA = load_scale(wave);
    }

    // The item's queries, in two dependent rounds of unconditional loads:
    // the pairs of this lane's A row slot (m / 2) and of its two output slots
    // (2 kq, 2 kq + 1), then the query rows and epilogue terms.  Slots at or
    // past G read the item's last pair instead: their A rows only feed MFMA
    // output rows that are never stored (ok[] below).
    const int prA = a.pairs[pbase + min(m >> 1, G - 1)];
    int prs[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) prs[i] = a.pairs[pbase + min(2 * kq + i, G - 1)];
    const int qA = prA / a.nprobe;
    // A operands: row m = 2 * slot + part (part 0 = hi, 1 = lo)
    const _Float16 *asrc = ((m & 1) ? a.ql : a.qh) + int64_t(qA) * a.d_pad + 8 * kq;
    half8 av[NC];
    if constexpr (!MP) {
#pragma unroll
      for (int c = 0; c < NC; ++c) av[c] = *reinterpret_cast<const half8 *>(asrc + 32 * c);
    }
    // multi-pass: the A operands of chunks [c0, c0 + NC), loaded per pass
    auto load_a = [&](int c0) {
#pragma unroll
      for (int c = 0; c < NC; ++c) av[c] = *reinterpret_cast<const half8 *>(asrc + 32 * (c0 + c));
    };
    // epilogue parameters of the two query slots this lane outputs
    float qc[2], qi[2];
    int64_t obase[2];
    bool ok[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = prs[i] / a.nprobe;
      ok[i] = 2 * kq + i < G;
      qc[i] = a.probe_dots[prs[i]];
      qi[i] = a.qinv[q];
      obase[i] = int64_t(q) * a.stride + a.prefix[prs[i]];
    }
    float *out[2] = {a.scores + obase[0] + cand0, a.scores + obase[1] + cand0};
    const bool lead_lane = LITE && kq < a.lead / 8;
    auto scale_of = [&](int j) {   // j is uniform across the wave
      const int r = j >> 2;
      uint32_t v = sreg[0];
#pragma unroll
      for (int t = 1; t < (kPreload ? kScaleRegs : 1); ++t) v = r == t ? sreg[t] : v;
      return uint32_t(__shfl(int(v), 16 * (j & 3) + m, 64));
    };
    if constexpr (!MP) {
      // Software pipeline, depth 1: the codes of the wave's next tile are in
      // flight while the current tile is decoded and multiplied (the first
      // tile, bufA, was issued above).  Tiles past the item read as zeros
      // from the buffer range check and are not scored.
      uint32_t bufB[kWordsPerLane];
      uint32_t scB = 0u;
      int lt = wave, j = 0;
      while (lt < n_tiles) {
        load_tile(bufB, tiles, lt + nwaves, n_tiles, tb, voff);
        scB = load_scale(lt + nwaves);
        score_tile<BITS, NC, kWordsPerLane, LITE>(bufA, LITE ? 0u : kPreload ? scale_of(j) : scA, av,
                                                  dtab, lane4, lt, n_cand, m, ok, qc, qi, out, ltab,
                                                  lead_lane, a.global);
        lt += nwaves;
        ++j;
        if (lt >= n_tiles) break;
        load_tile(bufA, tiles, lt + nwaves, n_tiles, tb, voff);
        scA = load_scale(lt + nwaves);
        score_tile<BITS, NC, kWordsPerLane, LITE>(bufB, LITE ? 0u : kPreload ? scale_of(j) : scB, av,
                                                  dtab, lane4, lt, n_cand, m, ok, qc, qi, out, ltab,
                                                  lead_lane, a.global);
        lt += nwaves;
        ++j;
      }
    } else {
      // Software pipeline, depth 1: the codes of the wave's next tile are in
      // flight while the current tile is decoded and multiplied.  Tiles past
      // the item read as zeros from the buffer range check and are not scored.
      // voff: this lane's first 16-byte unit of the pass's chunks.
      auto run_tiles = [&](auto mode_tag, uint32_t voff) {
        constexpr int MODE = decltype(mode_tag)::value;
        // Rslm4Lite, last pass: the first code word of the lane's stream
        // (chunk 0, which holds the scale bits), read with each tile
        constexpr bool kWord0 = LITE && MODE == 3;
        auto load_word0 = [&](int t) {
          return kWord0 ? __builtin_amdgcn_raw_buffer_load_b32(
                              make_rsrc(tiles + int64_t(t) * tb, t < n_tiles ? tb : 0u),
                              uint32_t(lane) * 16u, 0, 0)
                        : 0u;
        };
        auto sc_of = [&](uint32_t word0, uint32_t sc_reg, int jj) {
          if (LITE) return kWord0 ? lite_scales(word0, m, a.global) : 0u;
          return kPreload ? scale_of(jj) : sc_reg;
        };
        uint32_t bufA[kWordsPerLane], bufB[kWordsPerLane];
        uint32_t scA, scB = 0u, w0A, w0B = 0u;
        int lt = wave, j = 0;
        load_tile(bufA, tiles, lt, n_tiles, tb, voff);
        scA = load_scale(lt);
        w0A = load_word0(lt);
        while (lt < n_tiles) {
          load_tile(bufB, tiles, lt + nwaves, n_tiles, tb, voff);
          scB = load_scale(lt + nwaves);
          w0B = load_word0(lt + nwaves);
          score_tile<BITS, NC, kWordsPerLane, LITE, MODE>(bufA, sc_of(w0A, scA, j), av, dtab, lane4,
                                                          lt, n_cand, m, ok, qc, qi, out, ltab,
                                                          lead_lane, a.global);
          lt += nwaves;
          ++j;
          if (lt >= n_tiles) break;
          load_tile(bufA, tiles, lt + nwaves, n_tiles, tb, voff);
          scA = load_scale(lt + nwaves);
          w0A = load_word0(lt + nwaves);
          score_tile<BITS, NC, kWordsPerLane, LITE, MODE>(bufB, sc_of(w0B, scB, j), av, dtab, lane4,
                                                          lt, n_cand, m, ok, qc, qi, out, ltab,
                                                          lead_lane, a.global);
          lt += nwaves;
          ++j;
        }
      };
      const uint32_t voff0 = uint32_t(lane) * 16u;
      static_assert(NC >= 16 && (NC * BITS) % 16 == 0, "multi-pass configuration");
      // passes over chunk ranges of NC chunks: NC * BITS bytes of a lane's
      // stream, a whole number of 16-byte units (the plan's chunk counts
      // above 32 are multiples of such ranges; the host picks NC)
      constexpr uint32_t kPassUnits = uint32_t(NC * BITS / 16);
      for (int pass = 0; pass < a.n_pass; ++pass) {
        load_a(pass * NC);
        const uint32_t voff = voff0 + uint32_t(pass) * kPassUnits * 1024u;
        if (pass == 0) run_tiles(std::integral_constant<int, 1>{}, voff);
        else if (pass + 1 < a.n_pass) run_tiles(std::integral_constant<int, 2>{}, voff);
        else run_tiles(std::integral_constant<int, 3>{}, voff);
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        // this lane's dot stores of the pass before the next pass's loads
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      }
    }
    // Retire the last (out-of-range, zero-traffic) prefetch before the next
    // item, so the tile loop always starts with a known set of loads in
    // flight and the compiler keeps its waits partial.
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    if (tid == 0) s_ticket[(k_it + 1) & 1] = resolve(next_ticket);
    __syncthreads();
  }
}

// ------------------------------------------------------------- top-k
struct ScanId {
  const int32_t *prefix;       // nprobe entries of this query
  const int32_t *probe_ids;    // nprobe entries of this query
  const int64_t *list_offsets;
  const int32_t *ids;
  int nprobe;
  __device__ int32_t operator()(int i) const {
    int lo = 0, hi = nprobe;  // last p with prefix[p] <= i
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (prefix[mid] <= i) lo = mid;
      else hi = mid;
    }
    const int L = probe_ids[lo];
    return ids[list_offsets[L] + (i - prefix[lo])];
  }
};

// ------------------------------------------------------------- top-k
// One 1,024-thread workgroup per query streams the query's score region once.
// Candidates are kept in LDS as (key << 32 | position) for every score whose
// key is at or above a running threshold T.  T is the lower edge of a radix
// bin that holds the k-th largest key among the candidates kept so far, so T
// never exceeds the k-th largest key of the whole region: every element of
// the exact top-k (ties at its k-th key included) is kept.  When more than
// kStreamSoft candidates are held, T is raised by radix selection over them
// and the buffer is compacted.  At the end the survivors (usually a few
// hundred) get their ids and are sorted by (score desc, id asc).  If the
// buffer ever overflows (runs of equal keys wider than it), the exact block
// selection runs over the whole region instead.
constexpr int kStreamThreads = 1024;
constexpr int kStreamCap = 4096;
constexpr int kStreamSoft = 2048;

struct StreamSmem {
  uint64_t buf[2][kStreamCap];
  uint32_t hist[4096];
  uint32_t bcast[4 + kStreamThreads / 64];   // results, then per-wavefront totals
  uint32_t count[2];
  uint32_t overflow;
  int32_t spre[kMaxNprobe], sprobe[kMaxNprobe];
};

// The highest bin bb of hist[0..nb) with above + sum(hist[bb..nb)) >= k, and
// the count strictly above it, into bcast[0..1].  Every thread must call it.
// Thread t sums the bins [t per, (t + 1) per); a suffix scan over the threads
// (within each wavefront by shuffles, then over the wavefronts' totals)
// gives every thread the count above its bins, and the one thread whose
// bins hold the boundary walks them (at most four).
__device__ __forceinline__ void stream_boundary(StreamSmem &sm, int nb, uint32_t above,
                                                uint32_t k) {
  __syncthreads();
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int nt = blockDim.x;
  const int per = nb >= nt ? nb / nt : 1;       // nb and nt are powers of two
  const int lo = t * per;
  const bool active = lo < nb;
  uint32_t sum = 0;
  if (active)
    for (int b = lo; b < lo + per; ++b) sum += sm.hist[b];
  // inclusive suffix scan within the wavefront (higher threads hold higher bins)
  uint32_t incl = sum;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t v = __shfl_down(incl, off, 64);
    if (lane + off < 64) incl += v;
  }
  uint32_t *wsum = sm.bcast + 4;   // per-wavefront totals (kStreamThreads / 64 of them)
  if (lane == 0) wsum[wave] = incl;
  if (t == 0) {
    sm.bcast[0] = 0u;
    sm.bcast[1] = above;
  }
  __syncthreads();
  uint32_t after = 0;   // counts of the wavefronts above this one
  for (int w = wave + 1; w < nt / 64; ++w) after += wsum[w];
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
    sm.bcast[1] = acc;
  }
  __syncthreads();
}

// Raises the threshold over the cnt >= k candidates of buffer `cur`: radix
// passes of up to 12 bits, starting below the leading bits every candidate
// shares, narrow the bin holding the k-th largest key until at most `target`
// candidates are at or above its lower edge; returns that edge (never above
// the k-th largest key).
__device__ uint32_t stream_threshold(StreamSmem &sm, int cur, int cnt, int k, int target) {
  const int tid = threadIdx.x, nt = blockDim.x, lane = tid & 63, wave = tid >> 6;
  // the leading bits all candidates share: the first digit starts below them
  uint32_t kmin = 0xffffffffu, kmax = 0u;
  for (int i = tid; i < cnt; i += nt) {
    const uint32_t key = uint32_t(sm.buf[cur][i] >> 32);
    kmin = min(kmin, key);
    kmax = max(kmax, key);
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    kmin = min(kmin, uint32_t(__shfl_xor(int(kmin), off, 64)));
    kmax = max(kmax, uint32_t(__shfl_xor(int(kmax), off, 64)));
  }
  __syncthreads();   // hist is free: the previous use of it is complete
  if (lane == 0) {
    sm.hist[2 * wave] = kmin;
    sm.hist[2 * wave + 1] = kmax;
  }
  __syncthreads();
  for (int w = 0; w < nt / 64; ++w) {
    kmin = min(kmin, sm.hist[2 * w]);
    kmax = max(kmax, sm.hist[2 * w + 1]);
  }
  const uint32_t diff = kmin ^ kmax;
  if (diff == 0u) return kmin;   // every candidate has the same key
  int pbits = __clz(diff);
  uint32_t prefix = pbits ? kmax >> (32 - pbits) : 0u;
  uint32_t above = 0, edge = 0;
  while (pbits < 32) {
    const int d = min(12, 32 - pbits), nb = 1 << d, shift = 32 - pbits - d;
    __syncthreads();   // the reads of hist above (or of the previous pass) are done
    for (int b = tid; b < nb; b += nt) sm.hist[b] = 0;
    __syncthreads();
    for (int i = tid; i < cnt; i += nt) {
      const uint32_t key = uint32_t(sm.buf[cur][i] >> 32);
      if (pbits == 0 || (key >> (32 - pbits)) == prefix)
        atomicAdd(&sm.hist[(key >> shift) & (nb - 1)], 1u);
    }
    stream_boundary(sm, nb, above, uint32_t(k));
    const uint32_t bb = sm.bcast[0];
    const uint32_t in_bin = sm.hist[bb];
    above = sm.bcast[1];
    prefix = (prefix << d) | bb;
    pbits += d;
    edge = prefix << (32 - pbits);
    if (above + in_bin <= uint32_t(target)) break;
  }
  __syncthreads();
  return edge;
}

// Moves the candidates of buffer `cur` with key >= T to the other buffer;
// returns their number.
__device__ int stream_compact(StreamSmem &sm, int cur, int cnt, uint32_t T) {
  const int tid = threadIdx.x, nt = blockDim.x;
  if (tid == 0) sm.count[cur ^ 1] = 0;
  __syncthreads();
  for (int i = tid; i < cnt; i += nt) {
    const uint64_t e = sm.buf[cur][i];
    if (uint32_t(e >> 32) >= T) sm.buf[cur ^ 1][atomicAdd(&sm.count[cur ^ 1], 1u)] = e;
  }
  __syncthreads();
  return int(sm.count[cur ^ 1]);
}

__global__ void __launch_bounds__(kStreamThreads) k_topk_stream(
    const float *__restrict__ scores, int64_t stride, const int32_t *__restrict__ totals,
    const int32_t *__restrict__ prefix, const int32_t *__restrict__ probe_ids, int nprobe,
    const int64_t *__restrict__ list_offsets, const int32_t *__restrict__ ids, int k,
    float *__restrict__ out_s, int32_t *__restrict__ out_i) {
  __shared__ StreamSmem sm;
  const int tid = threadIdx.x, nt = blockDim.x;
  const int q = blockIdx.x;
  const int n = __builtin_amdgcn_readfirstlane(totals[q]);
  const float *row = scores + int64_t(q) * stride;   // stride: a multiple of 64
  for (int p = tid; p < nprobe; p += nt) {
    sm.spre[p] = prefix[int64_t(q) * nprobe + p];
    sm.sprobe[p] = probe_ids[int64_t(q) * nprobe + p];
  }
  if (tid == 0) sm.overflow = 0;
  // the first kStreamCap scores are all candidates
  const int n0 = min(n, kStreamCap);
  for (int i = tid; i < n0; i += nt) sm.buf[0][i] = (uint64_t(order_key(row[i])) << 32) | uint32_t(i);
  __syncthreads();
  int cur = 0, cnt = n0;
  uint32_t T = 0;
  // candidates kept after a threshold raise: a tight target raises T early,
  // so that later rounds add few candidates and rarely trigger another raise
  const int keep = min(kStreamSoft / 2, max(256, 2 * k));
  if (n > n0) {
    // the rest, 16 scores per thread per round (four 16-byte loads); the
    // next round's loads are issued before the current round is filtered
    constexpr int kRound = kStreamThreads * 16;
    // range-checked loads (unconditional, zeros past the region): the range
    // is n rounded up to whole 16-byte groups, inside the region's stride
    // (n <= 2^30 - 4, so at most 2^32 - 16 bytes: a 32-bit range)
    const uint32_t rbytes = uint32_t((int64_t(n) + 3) & ~int64_t(3)) * 4u;
    const __amdgpu_buffer_rsrc_t rr = make_rsrc(row, rbytes);
    auto load_round = [&](float4 (&v)[4], int base) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const u32x4 w = __builtin_amdgcn_raw_buffer_load_b128(rr, uint32_t(base + (u * nt + tid) * 4) * 4u, 0, 0);
        v[u] = make_float4(__uint_as_float(w.x), __uint_as_float(w.y), __uint_as_float(w.z),
                           __uint_as_float(w.w));
      }
    };
    // filter one round held in v; false when the buffer overflowed
    auto filter_round = [&](const float4 (&v)[4], int base) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = base + (u * nt + tid) * 4;
        const float e[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const uint32_t key = order_key(e[c]);
          if (i + c < n && key >= T) {
            const uint32_t pos = atomicAdd(&sm.count[cur], 1u);
            if (pos < uint32_t(kStreamCap)) sm.buf[cur][pos] = (uint64_t(key) << 32) | uint32_t(i + c);
            else sm.overflow = 1;
          }
        }
      }
      __syncthreads();
      if (sm.overflow) return false;
      cnt = int(sm.count[cur]);
      if (cnt > kStreamSoft) {
        T = stream_threshold(sm, cur, cnt, k, keep);
        cnt = stream_compact(sm, cur, cnt, T);
        cur ^= 1;
      }
      return true;
    };
    float4 va[4], vb[4];
    T = stream_threshold(sm, cur, cnt, k, keep);
    cnt = stream_compact(sm, cur, cnt, T);
    cur ^= 1;
    load_round(va, n0);
    for (int base = n0; base < n;) {
      load_round(vb, base + kRound);
      if (!filter_round(va, base)) break;
      base += kRound;
      if (base >= n) break;
      load_round(va, base + kRound);
      if (!filter_round(vb, base)) break;
      base += kRound;
    }
    // retire the last (zero-traffic) prefetch
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  }
  const ScanId f{sm.spre, sm.sprobe, list_offsets, ids, nprobe};
  // final narrowing, then ids and the exact order of the survivors
  const int target = max(256, 2 * k);
  if (!sm.overflow && cnt > target && cnt >= k) {
    T = stream_threshold(sm, cur, cnt, k, target);
    cnt = stream_compact(sm, cur, cnt, T);
    cur ^= 1;
  }
  if (!sm.overflow && cnt <= kStreamCap) {
    uint64_t *out = sm.buf[cur ^ 1];
    for (int i = tid; i < cnt; i += nt) {
      const uint64_t e = sm.buf[cur][i];
      out[i] = composite(uint32_t(e >> 32), f(int(e & 0xffffffffu)));
    }
    __syncthreads();
    float *os = out_s + int64_t(q) * k;
    int32_t *oi = out_i + int64_t(q) * k;
    if (cnt <= nt) {
      rank_emit(out, cnt, k, os, oi);
      return;
    }
    sort_desc_buf(out, cnt);
    for (int j = tid; j < k; j += nt) {
      if (j < cnt) {
        os[j] = key_to_float(uint32_t(out[j] >> 32));
        oi[j] = int32_t(0xffffffffu - uint32_t(out[j] & 0xffffffffu));
      } else {
        os[j] = -__builtin_inff();
        oi[j] = -1;
      }
    }
    return;
  }
  // exact selection over the whole region (SelectSmem fits in one buffer)
  __syncthreads();
  static_assert(sizeof(SelectSmem) <= sizeof(uint64_t) * kStreamCap, "select scratch");
  SelectSmem &ss = *reinterpret_cast<SelectSmem *>(sm.buf[0]);
  block_topk(row, n, k, f, out_s + int64_t(q) * k, out_i + int64_t(q) * k, ss);
}

// Profiling hook: events that take the start and end times of the scan
// kernel's (0) and the top-k kernel's (1) own dispatch in later
// rslm_scan_topk calls made by the same host thread (the setting is per
// thread, so calls from other threads are never timed by it).  The events
// ride on the kernels' dispatch packets (hipExtLaunchKernelGGL), so timing
// adds no packets, and no gaps, to the stream.
static thread_local void *g_timer[2][2] = {{nullptr, nullptr}, {nullptr, nullptr}};

static hipEvent_t timer_event(int which, int end) {
  return reinterpret_cast<hipEvent_t>(g_timer[which][end]);
}

static int cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  (void)hipGetDevice(&dev);
  if (dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

template <int BITS, bool LITE = false>
static void launch_scan_bits(int nc, bool multi, dim3 grid, hipStream_t s, const ScanArgs &a) {
  const hipEvent_t e0 = timer_event(0, 0), e1 = timer_event(0, 1);
#define RSLM_SCAN_NC(NCV) \
  hipExtLaunchKernelGGL((k_scan<BITS, NCV, LITE>), grid, dim3(kScanThreads), 0, s, e0, e1, 0, a)
#define RSLM_SCAN_MP(NCV)                                                                    \
  hipExtLaunchKernelGGL((k_scan<BITS, NCV, LITE, true>), grid, dim3(kScanThreads), 0, s, e0, e1, \
                        0, a)
  if (multi) {
    // pass ranges of 24 or 16 chunks starting on 16-byte units (ranges of
    // 32 would spill registers in the pass loop)
    if (nc == 16) RSLM_SCAN_MP(16);
    else if constexpr (BITS % 2 == 0) RSLM_SCAN_MP(24);
    return;
  }
  switch (nc) {
    case 1: RSLM_SCAN_NC(1); break;
    case 2: RSLM_SCAN_NC(2); break;
    case 3: RSLM_SCAN_NC(3); break;
    case 4: RSLM_SCAN_NC(4); break;
    case 6: RSLM_SCAN_NC(6); break;
    case 8: RSLM_SCAN_NC(8); break;
    case 12: RSLM_SCAN_NC(12); break;
    case 16: RSLM_SCAN_NC(16); break;
    case 24: RSLM_SCAN_NC(24); break;
    default: RSLM_SCAN_NC(32); break;
  }
#undef RSLM_SCAN_MP
#undef RSLM_SCAN_NC
}

}  // namespace rslm

using namespace rslm;

extern "C" {

size_t rslm_scan_topk_workspace(const rslm_plan *p, const rslm_index *idx, int32_t Q,
                                int32_t nprobe, int32_t k) {
  if (!p || !idx || Q < 0 || nprobe < 1 || idx->nlist < 1 || idx->max_list_size < 0 || k < 1)
    return 0;
  return scan_ws_layout(nullptr, Q, nprobe, idx->nlist, p->codec.d_pad, idx->max_list_size, k)
      .bytes;
}

int rslm_scan_topk(const rslm_plan *p, const rslm_index *idx, const float *q_rot, int32_t Q,
                   const int32_t *probe_ids, const float *probe_dots, int32_t nprobe, int32_t k,
                   float *out_scores, int32_t *out_ids, void *ws, size_t ws_bytes,
                   void *stream) {
  if (!p || !idx || Q < 0 || nprobe < 1 || nprobe > kMaxNprobe || k < 1 || k > kMaxK)
    return RSLM_ERR_INVALID_ARG;
  if (idx->nlist < 1 || idx->nlist > 65536 || nprobe > idx->nlist || idx->max_list_size < 0)
    return RSLM_ERR_INVALID_ARG;
  // a query's score region is read through 32-bit byte offsets
  // a query's score region is read with 32-bit byte ranges of whole 16-byte
  // groups: at most 2^30 - 4 scores
  if (int64_t(nprobe) * idx->max_list_size > (int64_t(1) << 30) - 4) return RSLM_ERR_INVALID_ARG;
  if (Q == 0) return RSLM_OK;
  if (Q > 65535) return RSLM_ERR_INVALID_ARG;   // gridDim.y of the top-k kernel
  if (!q_rot || !probe_ids || !probe_dots || !out_scores || !out_ids || !idx->list_offsets ||
      !idx->list_sizes || !idx->ids || !idx->codes || (!idx->scales && p->codec.lead == 0))
    return RSLM_ERR_INVALID_ARG;
  // the tile loads are 16-byte buffer loads; scales, ids and sizes are
  // read as 4-byte words, offsets as 8-byte words
  if ((reinterpret_cast<uintptr_t>(idx->codes) & 15) || (reinterpret_cast<uintptr_t>(idx->scales) & 3) ||
      (reinterpret_cast<uintptr_t>(idx->ids) & 3) || (reinterpret_cast<uintptr_t>(idx->list_sizes) & 3) ||
      (reinterpret_cast<uintptr_t>(idx->list_offsets) & 7) || (reinterpret_cast<uintptr_t>(q_rot) & 3) ||
      (reinterpret_cast<uintptr_t>(probe_ids) & 3) || (reinterpret_cast<uintptr_t>(probe_dots) & 3) ||
      (reinterpret_cast<uintptr_t>(out_scores) & 3) || (reinterpret_cast<uintptr_t>(out_ids) & 3))
    return RSLM_ERR_INVALID_ARG;
  // above 32 chunks: passes over equal ranges of 24 or 16 chunks that start
  // on a 16-byte unit of a lane's stream (the plan's chunk counts above 32
  // are multiples of 16, 24 or 32)
  int nc_pass = p->codec.n_chunks, n_pass = 1;
  if (nc_pass > 32) {
    n_pass = 0;
    for (int per : {24, 16})
      if (p->codec.n_chunks % per == 0 && (per * p->codec.bits) % 16 == 0) {
        nc_pass = per;
        n_pass = p->codec.n_chunks / per;
        break;
      }
    if (n_pass == 0) return RSLM_ERR_UNSUPPORTED;
  }
  const size_t need = rslm_scan_topk_workspace(p, idx, Q, nprobe, k);
  if (!ws || ws_bytes < need) return RSLM_ERR_WORKSPACE;
  const int nlist = idx->nlist;
  const int d_pad = p->codec.d_pad;
  ScanWs w = scan_ws_layout(ws, Q, nprobe, nlist, d_pad, idx->max_list_size, k);
  hipStream_t s = as_stream(stream);
  const int npairs = Q * nprobe;
  int st;
  hipLaunchKernelGGL(k_plan_a, dim3((Q + kPlanQueries - 1) / kPlanQueries + 1), dim3(kPlanThreads),
                     0, s, q_rot, Q,
                     p->rot.D, d_pad, w.qh, w.ql, w.qinv, probe_ids, nprobe, nlist,
                     idx->list_sizes, idx->max_list_size, w.prefix, w.totals, w.counts,
                     w.pair_off, w.item_off, w.cursor, w.work);
  if ((st = check_launch())) return st;
  const int64_t planb_threads = std::max<int64_t>(npairs, int64_t(nlist) * 64);
  hipLaunchKernelGGL(k_plan_b, dim3(unsigned((planb_threads + kPlanBThreads - 1) / kPlanBThreads)),
                     dim3(kPlanBThreads), 0, s, probe_ids, npairs, nlist, w.counts,
                     idx->list_sizes, idx->list_offsets, idx->max_list_size, w.pair_off,
                     w.item_off, w.cursor, w.pairs, w.items);
  if ((st = check_launch())) return st;

  ScanArgs a;
  a.list_offsets = idx->list_offsets;
  a.list_sizes = idx->list_sizes;
  a.codes = idx->codes;
  a.scales = idx->scales;
  a.dtab = p->d_dtab;
  a.qh = w.qh;
  a.ql = w.ql;
  a.qinv = w.qinv;
  a.probe_dots = probe_dots;
  a.item_off = w.item_off;
  a.items = w.items;
  a.work = w.work;
  a.pairs = w.pairs;
  a.prefix = w.prefix;
  a.scores = w.scores;
  a.stride = w.stride;
  a.nlist = nlist;
  a.nprobe = nprobe;
  a.d_pad = d_pad;
  a.n_chunks = p->codec.n_chunks;
  a.n_pass = n_pass;
  a.tile_bytes = p->codec.tile_bytes;
  a.lane_units = p->codec.lane_bytes / 16;
  a.max_list = idx->max_list_size;
  a.lead = p->codec.lead;
  a.global = p->codec.global;
  for (int i = 0; i < 8; ++i) a.cb_lead[i] = p->codec.cb_lead[i];
  // two workgroups per CU where the decode table takes 64 KiB of LDS (4 bits;
  // byte tables of 2 and 1 bits from 24 chunks up)
  const bool big_table = p->codec.bits == 4 || (p->codec.bits <= 2 && nc_pass >= 24);
  const int wg_per_cu = big_table ? 2 : 4;
  const dim3 grid(unsigned(cu_count() * wg_per_cu));
  switch (p->codec.bits) {
    case 4:
      if (a.lead > 0) launch_scan_bits<4, true>(nc_pass, n_pass > 1, grid, s, a);
      else launch_scan_bits<4>(nc_pass, n_pass > 1, grid, s, a);
      break;
    case 3: launch_scan_bits<3>(nc_pass, n_pass > 1, grid, s, a); break;
    case 2: launch_scan_bits<2>(nc_pass, n_pass > 1, grid, s, a); break;
    default: launch_scan_bits<1>(nc_pass, n_pass > 1, grid, s, a); break;
  }
  if ((st = check_launch())) return st;
  hipExtLaunchKernelGGL(k_topk_stream, dim3(unsigned(Q)), dim3(kStreamThreads), 0, s,
                        timer_event(1, 0), timer_event(1, 1), 0, w.scores, w.stride, w.totals,
                        w.prefix, probe_ids, nprobe, idx->list_offsets, idx->ids, k, out_scores,
                        out_ids);
  return check_launch();
}

int rslm_set_timer(int which, void *ev_begin, void *ev_end) {
  if (which < 0 || which > 1 || (!ev_begin) != (!ev_end)) return RSLM_ERR_INVALID_ARG;
  g_timer[which][0] = ev_begin;
  g_timer[which][1] = ev_end;
  return RSLM_OK;
}

}  // extern "C"
