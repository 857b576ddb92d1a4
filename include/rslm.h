/*
 * rslm.h -- C ABI of librslm, an MI355X (gfx950) implementation of the RSLM
 * (Rotated Scaled Lloyd-Max) IVF second-stage scan and bulk encoder.
 *
 * Method: "RSLM: Training-Free Vector Quantization for Approximate Nearest
 * Neighbor Search" (arXiv 2608.30384).  Each entry point cites the section of
 * the paper that defines the operation.
 *
 * Conventions shared by every call
 *   - Array arguments are DEVICE pointers owned by the caller, row-major and
 *     contiguous, unless a comment says "host".  The library never frees or
 *     retains caller memory; only rslm_plan_create allocates (the plan's own
 *     device tables, released by rslm_plan_destroy).
 *   - Scratch memory is a caller-provided workspace ("ws", "ws_bytes") whose
 *     size comes from the matching *_workspace function.
 *   - "stream" is a hipStream_t passed as void* (NULL = the null stream).
 *     Every call is asynchronous on that stream; results are ready after the
 *     caller synchronises the stream.
 *   - Every call returns an rslm_status.  Arguments are validated before any
 *     launch; on a non-zero status nothing was launched and outputs are
 *     untouched.  RSLM_ERR_HIP means a launch failed (the HIP error is
 *     retrievable with rslm_last_hip_error).  Faults during kernel execution
 *     surface at the caller's next synchronisation.
 *   - Calls on distinct streams are thread-safe; a plan may be shared.
 *   - Vector ids are int32 (collections of up to 2^31 - 1 vectors).
 */
#ifndef RSLM_H
#define RSLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum rslm_status {
  RSLM_OK = 0,
  RSLM_ERR_INVALID_ARG = 1,   /* null pointer, size or enum out of range */
  RSLM_ERR_UNSUPPORTED = 2,   /* valid request the library does not implement */
  RSLM_ERR_HIP = 3,           /* a HIP launch or runtime call failed */
  RSLM_ERR_WORKSPACE = 4,     /* ws_bytes smaller than the *_workspace size */
  RSLM_ERR_NO_DEVICE = 5      /* no usable gfx950 device is current */
} rslm_status;

/* Human-readable name of a status code (static string, never NULL). */
const char *rslm_status_string(int status);
/* The hipError_t recorded by the last RSLM_ERR_HIP on this thread. */
int rslm_last_hip_error(void);
/* Library version, "major.minor.patch" (static string). */
const char *rslm_version(void);

/* ------------------------------------------------------------------------
 * Codec plan.  Section "Rslm codec family": the block-wise cascaded FWHT
 * ("Pre-Quantization Transformations"), the fixed Lloyd-Max codebooks
 * ("Quantization Using Lloyd-Max Codebook", table tab:rslm_codecs), the
 * norm-correcting scale ("Norm Correction", "Scale Encoding") and the
 * local/global relative modes ("Relative Quantization").
 * ------------------------------------------------------------------------ */
typedef struct rslm_plan rslm_plan;

typedef struct rslm_plan_desc {
  int32_t dim;            /* D, 1 <= D <= 4096 */
  int32_t bits;           /* 1, 2, 3 or 4 bits per dimension: (g, K) = (4,16),
                             (2,16), (1,8), (1,16) */
  int32_t passes;         /* rotation passes: 0 (none), 1, 2, or -1 for the
                             paper's rule (1 iff bits == 4 and D <= 256) */
  int32_t scale_mode;     /* 0 local (second scale fixed to 1.0),
                             1 global (second scale ||x|| / ||a + r~||) */
  const int8_t *signs;    /* host, 256 entries, each +1 or -1 (S1) */
  const int32_t *perm;    /* host, 128 entries, a permutation of 0..127 (P) */
  const float *codebook;  /* host, K*g floats, centroid k at [k*g, k*g+g);
                             every value exactly representable in float16;
                             for g == 1 strictly ascending */
  int32_t lite;           /* 1: Rslm4Lite (bits == 4, dim >= 64; Section
                             "Codecs Description"): the first 16 coordinates
                             (32 with the global scale) use the K = 8
                             codebook_lead and bit 3 of their codes holds
                             the scales, bit j of UE7M9 s^ in coordinate j
                             (j < 16), bit j - 16 of UE4M12 g^ in coordinate
                             j (16 <= j < 32); 0: standard codec */
  const float *codebook_lead;  /* host, 8 ascending float16-exact floats
                                  (lite only, else ignored) */
} rslm_plan_desc;

typedef struct rslm_plan_info {
  int32_t dim, bits, passes, scale_mode;
  int32_t K, g;            /* centroids and sub-vector size */
  int32_t block;           /* FWHT block size B */
  int32_t n_full_blocks;   /* floor(D / B); an overlap block follows iff D % B */
  int32_t d_pad;           /* D rounded up to a multiple of 32 (scan layout) */
  int32_t canon_bytes;     /* canonical code bytes per record */
  int32_t tile_records;    /* records per scan tile (16) */
  int32_t tile_bytes;      /* bytes of one tile of packed codes */
  double emax;             /* E_max(D) = E[max_i |Z_i|], Z_i ~ N(0,1) i.i.d. */
  int32_t lite;            /* 1 for Rslm4Lite */
  int32_t record_bytes;    /* packed record (rslm_pack_records): canon_bytes
                              + 2 (local) or + 4 (global); Lite: canon_bytes */
} rslm_plan_info;

/* Creates a plan on the current HIP device; copies the host tables.
 * Status INVALID_ARG for out-of-range fields or tables, NO_DEVICE when the
 * current device is not gfx950. */
int rslm_plan_create(const rslm_plan_desc *desc, rslm_plan **out);
int rslm_plan_destroy(rslm_plan *plan);
int rslm_plan_get_info(const rslm_plan *plan, rslm_plan_info *info);

/* ------------------------------------------------------------------------
 * rslm_fwht -- the cascaded rotation R (Sections "Fast Walsh Hadamard
 * Transform", "Sign Flips and Dimension Permutation", "Cascaded Rotation
 * Pipeline"); used for Precompute-Query (Section "Performance Impact and
 * Memory Savings": rotate a query once, score in the rotated space).
 *   x, y   : n x D float32 (y may equal x).
 *   inverse: 0 -> y = R x;  1 -> y = R^T x (blocks in reverse order).
 * ------------------------------------------------------------------------ */
int rslm_fwht(const rslm_plan *plan, const float *x, float *y, int64_t n,
              int inverse, void *stream);

/* ------------------------------------------------------------------------
 * rslm_encode -- bulk RSLM encoding of records (Sections "Quantization Using
 * Lloyd-Max Codebook", "Norm Correction", "Scale Encoding", "Relative
 * Quantization"; the IVF residual of Section "End-to-End Comparison": the
 * residual is taken against the record's partition centre).
 * For record r (0 <= r < n_records):
 *   row  = src_row ? src_row[r] : r        (row of x; < 0 marks a padding
 *                                            record, which is skipped)
 *   c    = centroids ? centroids[rec_list[r]] : 0
 *   z    = R (x[row] - c);  u = z * E_max(D) / max|z|
 *   code = nearest centroid per g-sub-vector (lower index on ties)
 *   s^   = UE7M9(||x - c|| / ||C[code]||)
 *   g^   = UE4M12(||x|| / ||c + R^T s^ C[code]||) (global) or 1.0 (local)
 * Outputs:
 *   codes     : scan tile layout, ceil(n_records/16) * tile_bytes bytes
 *               (record r is in tile r/16; see rslm_pack_codes)
 *   scales    : n_records uint32, lo16 = s^ (UE7M9), hi16 = g^ (UE4M12)
 *   resid_rot : n_rows x D float32 or NULL: row `row` of record r receives
 *               the rotated second residual R x - g^ (R c + s^ C[code]) for a
 *               rescoring codec (rows not referenced are left untouched)
 * centroids_rot (nlist x D, = R c) is required when centroids is given.
 * x has n_rows rows (bounds for src_row); centroids has nlist rows.
 * ------------------------------------------------------------------------ */
int rslm_encode(const rslm_plan *plan, const float *x, int64_t n_rows,
                const int64_t *src_row, const int32_t *rec_list,
                int64_t n_records, const float *centroids,
                const float *centroids_rot, int32_t nlist, uint8_t *codes,
                uint32_t *scales, float *resid_rot, void *stream);

/* ------------------------------------------------------------------------
 * rslm_encode_two_stage -- rslm_encode plus, in the same pass, the rescoring
 * codec of Section "Relative Quantization" applied to the first stage's
 * error (two-stage relative coding, the RelApprox(Global)-Rslm rescoring
 * records of table tab:recall_eval_relative).  With the first-stage
 * approximation a = g^ (c + R^T s^ C[code]) of record r (row `row`):
 *   r2    = R x - R a                  (rotated space; no further rotation:
 *                                        the rotation is a fixed table)
 *   u2    = r2 * E_max(D) / max|r2|
 *   code2 = nearest centroid of plan2's codebook per g2-sub-vector
 *   s2^   = UE7M9(||r2|| / ||C2[code2]||)
 *   g2^   = UE4M12(||x|| / ||R a + s2^ C2[code2]||) if plan2 is global,
 *           else 1.0 (code 0x7000)
 * A zero r2 gives codes2 = 0 and s2^ = 0.
 *   plan2   : same dim as plan, passes == 0.
 *   codes2  : n_rows x canon_bytes(plan2) uint8, canonical layout (see
 *             rslm_pack_codes), row `row` written for record r.
 *   scales2 : n_rows uint32, lo16 = s2^ (UE7M9), hi16 = g2^ (UE4M12).
 * Every other argument and output is as in rslm_encode (no rotated residual
 * is produced).  Rows not referenced by a record are left untouched.
 * ------------------------------------------------------------------------ */
int rslm_encode_two_stage(const rslm_plan *plan, const rslm_plan *plan2, const float *x,
                          int64_t n_rows, const int64_t *src_row, const int32_t *rec_list,
                          int64_t n_records, const float *centroids,
                          const float *centroids_rot, int32_t nlist, uint8_t *codes,
                          uint32_t *scales, uint8_t *codes2, uint32_t *scales2,
                          void *stream);

/* ------------------------------------------------------------------------
 * rslm_grid2_lists -- host utility (no device work, no GPU needed): the
 * candidate lists with which the encoder finds the nearest centroid of a
 * 2-D codebook (the second stage of rslm_encode_two_stage) without scoring
 * all K: a RSLM_GRID2 x RSLM_GRID2 grid of cells over [-emax, emax]^2, the
 * cell of u being (gx, gy), g_d = floor(clamp(u_d s + o, 0, RSLM_GRID2 - 1)),
 * whose list holds every code that can be nearest to some point of the cell
 * (lowest code on ties), so that scanning it in order with a strict
 * comparison of |C_k|^2 / 2 - <u, C_k> gives the nearest code.  Plans of
 * 2-D codebooks build the same lists.
 *   codebook     : K x 2 floats (host), 1 <= K <= 16, finite.
 *   emax         : > 0, E_max of the plan's dimension (float).
 *   out          : RSLM_GRID2 * RSLM_GRID2 uint16 (host); cell (gx, gy) at
 *                  gx * RSLM_GRID2 + gy, four 4-bit codes from the lowest
 *                  bits up, ascending, the last one repeated.
 *   scale_offset : 2 floats (host) receiving s and o.
 * RSLM_ERR_INVALID_ARG for a bad argument, RSLM_ERR_UNSUPPORTED if some cell
 * needs more than four codes (the encoder then scores all K).
 * ------------------------------------------------------------------------ */
#define RSLM_GRID2 32
int rslm_grid2_lists(const float *codebook, int32_t K, float emax, uint16_t *out,
                     float *scale_offset);

/* ------------------------------------------------------------------------
 * rslm_encode_sq8 -- rslm_encode with the rotated second residual
 * r2 = R x - g^ (R c + s^ C[code]) written directly as SQ8 codes with given
 * ranges (the RelApprox-SQ8 rescoring records; Sections "Background and
 * Related Work" and "Relative Quantization"): for d < D,
 *   codes2[row][d] = clamp(rne((r2_d - sq8_lo[d]) / step_d), 0, 255),
 *   step_d = (sq8_hi[d] - sq8_lo[d]) / 255 (a zero step gives 0),
 * exactly what rslm_sq8_encode computes from the float residual.  Used to
 * encode vectors added to a collection whose ranges were fitted already.
 *   sq8_lo, sq8_hi : D float32 (device); codes2 : n_rows x D uint8, row
 *   `row` written for record r.  Everything else as in rslm_encode.
 * ------------------------------------------------------------------------ */
int rslm_encode_sq8(const rslm_plan *plan, const float *x, int64_t n_rows,
                    const int64_t *src_row, const int32_t *rec_list, int64_t n_records,
                    const float *centroids, const float *centroids_rot, int32_t nlist,
                    uint8_t *codes, uint32_t *scales, const float *sq8_lo,
                    const float *sq8_hi, uint8_t *codes2, void *stream);

/* ------------------------------------------------------------------------
 * rslm_decode -- Decompress (Section "Performance Impact and Memory
 * Savings": Compress / Decompress; Section "Relative Quantization"): the
 * reconstruction of record r (tile layout codes and scales as rslm_encode
 * wrote them)
 *   x~_r = g^ (c + R^T s^ C[code])      (g^ = 1.0 for a local plan)
 * with c = centroids[rec_list[r]] when centroids is given, else 0; R^T runs
 * the blocks in reverse order.  out: n x D float32.
 * ------------------------------------------------------------------------ */
int rslm_decode(const rslm_plan *plan, const uint8_t *codes, const uint32_t *scales, int64_t n,
                const int32_t *rec_list, const float *centroids, int32_t nlist, float *out,
                void *stream);

/* Canonical <-> scan layout of packed codes (Section "Codecs Description":
 * codes are a packed bit stream, code j of a record at bits [w j, w j + w),
 * w = log2 K, little-endian).  canon: n x canon_bytes; tiles: ceil(n/16) *
 * tile_bytes.  Padding records of the last tile are zero-filled. */
int rslm_pack_codes(const rslm_plan *plan, const uint8_t *canon, int64_t n,
                    uint8_t *tiles, void *stream);
int rslm_unpack_codes(const rslm_plan *plan, const uint8_t *tiles, int64_t n,
                      uint8_t *canon, void *stream);

/* ------------------------------------------------------------------------
 * Packed records (Section "Codecs Description", table tab:rslm_codecs: the
 * codes followed by the scale factor): record r = canonical codes
 * (canon_bytes) then UE7M9 s^ as a little-endian uint16, then for a global
 * plan UE4M12 g^ likewise; a Lite plan's record is its canonical codes alone
 * (scales embedded), ceil(D / 2) bytes.  record_bytes in rslm_plan_info.
 *   rslm_pack_records: tiles (rslm_encode's layout) + scales (n uint32; may
 *   be NULL for Lite) -> records, n x record_bytes.
 * ------------------------------------------------------------------------ */
int rslm_pack_records(const rslm_plan *plan, const uint8_t *tiles, const uint32_t *scales,
                      int64_t n, uint8_t *records, void *stream);

/* ------------------------------------------------------------------------
 * rslm_score -- OneToMany scoring (Section "Performance Impact and Memory
 * Savings": a rotated query against many encoded vectors, contiguous or
 * gathered from a large pool): for query q < Q and entry j < n,
 *   r = ids ? ids[j] : j
 *   out[q * n + j] = g^_r s^_r sum_i <q_rot[q][i g:(i+1) g], C[code_{r,i}]>
 * (g^ = 1 for a local plan), records as above, n_pool records in `records`;
 * an id outside [0, n_pool) gives -inf.  q_rot: Q x D (rslm_fwht);
 * ids: n int64 or NULL (then n <= n_pool); Q <= 65535.
 * ------------------------------------------------------------------------ */
int rslm_score(const rslm_plan *plan, const uint8_t *records, int64_t n_pool,
               const int64_t *ids, int64_t n, const float *q_rot, int32_t Q, float *out,
               void *stream);

/* ------------------------------------------------------------------------
 * ivf_assign_probe -- IVF routing (Section "End-to-End Comparison", Setup):
 *   IVF_ASSIGN_L2: out_ids[i] = argmin_p ||x_i - c_p||^2 (lowest p on ties),
 *                  out_scores[i] = that squared distance (may be NULL);
 *                  nprobe must be 1.
 *   IVF_PROBE_IP : the nprobe partitions with the largest <x_i, c_p>,
 *                  ordered by (dot desc, p asc): out_ids / out_scores are
 *                  n x nprobe (out_scores = the dots).
 *   x: n x dim, centroids: nlist x dim (float32).  nlist <= 65536,
 *   nprobe <= min(nlist, 1024).
 * ------------------------------------------------------------------------ */
#define IVF_ASSIGN_L2 0
#define IVF_PROBE_IP 1
size_t ivf_assign_probe_workspace(int64_t n, int32_t dim, int32_t nlist,
                                  int32_t nprobe, int mode);
int ivf_assign_probe(const float *x, int64_t n, int32_t dim,
                     const float *centroids, int32_t nlist, int32_t nprobe,
                     int mode, int32_t *out_ids, float *out_scores, void *ws,
                     size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * ivf_assign_probe_noalloc -- ivf_assign_probe for callers that cannot
 * allocate memory or hand in a workspace: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  The same kernels
 * and results as ivf_assign_probe; the scratch is a fixed device array of
 * ivf_assign_probe_noalloc_limit() bytes (64 MiB + 256 KiB) that the library
 * holds once per GPU it runs on until the process ends.  This call allocates
 * nothing (no hipMalloc / hipFree, no allocating library routine); the
 * caller passes inputs and outputs as for ivf_assign_probe.
 *   Sizes whose workspace (ivf_assign_probe_workspace) exceeds the limit --
 *   probing needs n * nlist * 4 bytes plus 4 * nlist rounded to 256 -- return
 *   RSLM_ERR_WORKSPACE before any launch.
 *   Every call on one GPU shares that GPU's scratch: calls that overlap in
 *   time on one GPU (different streams, threads or processes' graphs) race
 *   and must be serialised by the caller.  Nothing in the scratch needs to
 *   start at zero; its contents after a call are unspecified.
 * ------------------------------------------------------------------------ */
int ivf_assign_probe_noalloc(const float *x, int64_t n, int32_t dim,
                             const float *centroids, int32_t nlist, int32_t nprobe,
                             int mode, int32_t *out_ids, float *out_scores, void *stream);
size_t ivf_assign_probe_noalloc_limit(void);

/* ------------------------------------------------------------------------
 * ivf_kmeans_update -- the centre update of one Lloyd iteration of the
 * Euclidean k-means that partitions the collection (Section "End-to-End
 * Comparison", Setup): given each point's centre (IVF_ASSIGN_L2),
 *   centroids[p] = mean of the rows x_i with assign[i] == p,
 * evaluated as float64 sums rounded once to float32; a centre with no points
 * keeps its value.  Assignments outside [0, nlist) are ignored.
 *   x: n x dim float32; assign: n int32; centroids: nlist x dim float32,
 *   read and written in place.  n < 2^31, nlist <= 65536, dim <= 2^20; all
 *   arrays 4-byte aligned, else RSLM_ERR_INVALID_ARG.
 * ------------------------------------------------------------------------ */
size_t ivf_kmeans_update_workspace(int64_t n, int32_t nlist);
int ivf_kmeans_update(const float *x, int64_t n, int32_t dim, const int32_t *assign,
                      int32_t nlist, float *centroids, void *ws, size_t ws_bytes,
                      void *stream);

/* ------------------------------------------------------------------------
 * IVF index of RSLM records (caller-owned device arrays).  List L holds
 * list_sizes[L] records starting at record list_offsets[L] (a multiple of
 * 16, the tile size); record r has id ids[r], packed codes in tile r/16 and
 * scales[r].
 * ------------------------------------------------------------------------ */
typedef struct rslm_index {
  int32_t nlist;
  int32_t max_list_size;        /* host value: max_L list_sizes[L] */
  const int64_t *list_offsets;  /* nlist */
  const int32_t *list_sizes;    /* nlist */
  const int32_t *ids;           /* per record */
  const uint8_t *codes;         /* scan tile layout */
  const uint32_t *scales;       /* per record: lo16 s^ | hi16 g^ (unused, may be
                                   NULL, for Rslm4Lite plans) */
} rslm_index;

/* ------------------------------------------------------------------------
 * rslm_scan_topk -- second-stage scan and per-query top-k (Sections
 * "Relative Quantization" and "End-to-End Comparison"): for every query q
 * and every candidate x of its probed lists (probe_ids, from IVF_PROBE_IP),
 *   score = g^_x (<q, c_p> + s^_x sum_j <q_rot[j g:(j+1) g], C[code_x,j]>)
 * with <q, c_p> = probe_dots; then the k best by (score desc, id asc),
 * padded with (-inf, -1).
 *   q_rot: Q x D rotated queries (rslm_fwht); probe_ids / probe_dots:
 *   Q x nprobe; out_scores / out_ids: Q x k.  1 <= k <= 1024, Q <= 65535,
 *   nprobe * index->max_list_size <= 2^30 - 4 (a query's scores are read
 *   with 32-bit byte ranges), else RSLM_ERR_INVALID_ARG.  Alignment:
 *   index->codes 16 bytes, list_offsets 8 bytes, every other array 4 bytes,
 *   else RSLM_ERR_INVALID_ARG.  Any plan dimension (above D = 1,024 the
 *   coordinates are scored in passes over equal chunk ranges).  With a Lite
 *   plan the scales are read from the codes (the index's scales array is not
 *   used and may be NULL).
 * ------------------------------------------------------------------------ */
size_t rslm_scan_topk_workspace(const rslm_plan *plan, const rslm_index *index,
                                int32_t Q, int32_t nprobe, int32_t k);
int rslm_scan_topk(const rslm_plan *plan, const rslm_index *index,
                   const float *q_rot, int32_t Q, const int32_t *probe_ids,
                   const float *probe_dots, int32_t nprobe, int32_t k,
                   float *out_scores, int32_t *out_ids, void *ws,
                   size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * rslm_workspace_size -- the workspace (bytes) of one call, by call:
 *   RSLM_WS_SCAN_TOPK      = rslm_scan_topk_workspace(plan, index, n (= Q),
 *                            nprobe, k)
 *   RSLM_WS_ASSIGN_L2      = ivf_assign_probe_workspace(n, dim, nlist, 1,
 *                            IVF_ASSIGN_L2)
 *   RSLM_WS_PROBE_IP       = ivf_assign_probe_workspace(n, dim, nlist,
 *                            nprobe, IVF_PROBE_IP)
 *   RSLM_WS_KMEANS_UPDATE  = ivf_kmeans_update_workspace(n, nlist)
 * Arguments a call does not use are ignored (plan and index may be NULL
 * except for RSLM_WS_SCAN_TOPK).  Returns 0 for an unknown call or out-of-
 * range arguments.  Host arithmetic only; no device is touched.  The calls
 * not listed need no workspace.
 * ------------------------------------------------------------------------ */
#define RSLM_WS_SCAN_TOPK 0
#define RSLM_WS_ASSIGN_L2 1
#define RSLM_WS_PROBE_IP 2
#define RSLM_WS_KMEANS_UPDATE 3
size_t rslm_workspace_size(int call, const rslm_plan *plan, const rslm_index *index, int64_t n,
                           int32_t dim, int32_t nlist, int32_t nprobe, int32_t k);

/* ------------------------------------------------------------------------
 * 8-bit rescoring codec: SQ8 (Section "Background and Related Work": scalar
 * quantisation to 2^8 levels with a per-dimension range) applied to the
 * rotated second residual, used relatively with local scaling ("RelApprox-
 * SQ8", tab:recall_eval_relative).
 *   rslm_sq8_fit   : lo[d] / hi[d] = min / max over the n rows of v (n x dim);
 *                    accumulate != 0 folds into the existing lo / hi.
 *   rslm_sq8_encode: codes[dest_row[i] or i] = clamp(rne((v - lo) / step),
 *                    0, 255), step = (hi - lo) / 255 (a zero step gives 0),
 *                    evaluated as (v - lo) * (255 / (hi - lo)) with a 1-ulp
 *                    reciprocal (results differ from exact division only for
 *                    values within ~1e-5 of a rounding midpoint).
 * ------------------------------------------------------------------------ */
int rslm_sq8_fit(const float *v, int64_t n, int32_t dim, float *lo, float *hi,
                 int accumulate, void *stream);
int rslm_sq8_encode(const float *v, int64_t n, int32_t dim, const float *lo,
                    const float *hi, const int32_t *dest_row, int64_t n_dest,
                    uint8_t *codes, void *stream);

/* ------------------------------------------------------------------------
 * rslm_rescore -- second stage of two-stage retrieval (Sections "Background
 * and Related Work" and "Relative Quantization"): for each shortlisted
 * candidate, with score1 = <q, a> its first-stage score,
 *   RSLM_RESCORE_SQ8 : score2 = score1 + <q_rot, r~2>, r~2 the SQ8 decode
 *                      (local relative scaling);
 *   RSLM_RESCORE_RSLM: score2 = g2^ (score1 + s2^ sum_j <q_rot[j g2:(j+1) g2],
 *                      C2[code2_j]>) (g2^ = 1.0 for a local plan);
 * then the k_out best by (score2 desc, id asc).
 *   SQ8 : codes is n_vectors x dim uint8 indexed by id, lo / hi the ranges.
 *   RSLM: codes is n_vectors x canon_bytes(plan) (rslm_encode_two_stage's
 *         codes2), scales n_vectors uint32, plan the rescoring codec
 *         (passes == 0, dim == dim).
 *   cand_ids < 0 are empty slots; ids >= n_vectors are skipped as well.
 *   cand_scores / cand_ids: Q x k_in; out_*: Q x k_out; k_out <= k_in <= 1024.
 * ------------------------------------------------------------------------ */
#define RSLM_RESCORE_SQ8 0
#define RSLM_RESCORE_RSLM 1
typedef struct rslm_rescore_codec {
  int32_t kind;
  int32_t dim;
  int64_t n_vectors;
  const uint8_t *codes;
  const float *lo;            /* SQ8 only */
  const float *hi;            /* SQ8 only */
  const uint32_t *scales;     /* RSLM only: lo16 s2^ | hi16 g2^ */
  const rslm_plan *plan;      /* RSLM only */
} rslm_rescore_codec;

int rslm_rescore(const rslm_rescore_codec *codec, const float *q_rot,
                 int32_t Q, const float *cand_scores, const int32_t *cand_ids,
                 int32_t k_in, int32_t k_out, float *out_scores,
                 int32_t *out_ids, void *stream);

/* ------------------------------------------------------------------------
 * Profiling hook (not part of the method): in later rslm_scan_topk calls
 * made by the calling host thread, ev_begin / ev_end (hipEvent_t passed as
 * void*, created by the caller with timing enabled) take the start and end
 * times of one of their kernels' dispatch (the events are attached to the
 * kernel launch itself, so timing adds nothing to the stream):
 *   RSLM_TIMER_SCAN: the scan kernel;  RSLM_TIMER_TOPK: the top-k kernel.
 * Both NULL disables.  The setting belongs to the calling thread (thread-
 * local), so calls from other threads are unaffected and never timed by it.
 * ------------------------------------------------------------------------ */
#define RSLM_TIMER_SCAN 0
#define RSLM_TIMER_TOPK 1
int rslm_set_timer(int which, void *ev_begin, void *ev_end);

/* ------------------------------------------------------------------------
 * Measurement utility (not part of the method): a plain streaming read of
 * `bytes` bytes of device memory at buf (16-byte aligned, bytes a multiple of
 * 16) by `grid` workgroups of 256 threads, each writing the XOR of the words
 * it read to out[blockIdx] (out: grid uint32); nontemporal != 0 uses
 * non-temporal loads.  Timing it gives the read bandwidth the device
 * sustains, the reference for the scan's bandwidth.
 * ------------------------------------------------------------------------ */
int rslm_calibrate_read(const void *buf, int64_t bytes, uint32_t *out, int32_t grid,
                        int nontemporal, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* RSLM_H */
