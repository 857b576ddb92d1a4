// Plan objects, status handling and the E_max constant.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <new>

#include "rslm_internal.h"

namespace rslm {

static thread_local int g_last_hip = 0;

// Uniform bucket grid over sorted 1-D decision thresholds (quant_bucket):
// the smallest of 128, 256 or 512 buckets over +-1.0625 max |t| that puts
// every threshold in a bucket of its own; none (qn = 0) if even 512 do not.
static void quant_grid(const float *thr, int n, float &qs, float &qo, int &qn) {
  qs = qo = 0.0f;
  qn = 0;
  if (n < 1) return;
  float R = 0.0f;
  for (int k = 0; k < n; ++k) R = std::max(R, std::fabs(thr[k]));
  if (!(R > 0.0f) || !std::isfinite(R)) R = 1.0f;
  for (int cand = 128; cand <= 512; cand *= 2) {
    const float s = float(cand) / (2.125f * R), o = float(cand / 2);
    bool ok = true;
    for (int k = 1; k < n && ok; ++k)
      ok = quant_bucket(thr[k], s, o, cand) > quant_bucket(thr[k - 1], s, o, cand);
    if (ok) {
      qs = s;
      qo = o;
      qn = cand;
      return;
    }
  }
}

// |C_k|^2 / 2 of a g-dimensional centroid, in float as the encoders use it.
static float half_norm2(const float *c, int g) {
  float h = 0.0f;
  for (int t = 0; t < g; ++t) h += c[t] * c[t];
  return 0.5f * h;
}

// Candidate lists of the 2-D nearest-centroid grid (CodecParams::g2tab).
// Code k is left out of a cell only if one other code j is nearer by more
// than kMargin everywhere in the cell widened by kWiden (the device rounds
// u, the cell index and the distance in float32, far below both margins):
// with d_k(u) = |C_k|^2 / 2 - <u, C_k>, j beats k on a box when
// (h_k - h_j) - max_u <u, C_k - C_j> > kMargin, the maximum taken at the
// box's corner in the direction of C_k - C_j (an unbounded side, the outer
// cells extend to infinity, only if that component is zero or points away).
// The nearest code of any point is then in its cell's list, and the device,
// scanning the list in ascending order with a strict comparison, picks the
// same code (lowest on ties) as a search over all K.  False if a cell needs
// more than four codes.
static bool grid2_lists(const float *cb, const float *cbh, int K, float g2s, float g2o,
                        uint16_t *tab) {
  constexpr double kWiden = 1e-4, kMargin = 1e-4;
  const double inf = std::numeric_limits<double>::infinity();
  for (int i = 0; i < kGrid2; ++i)
    for (int j = 0; j < kGrid2; ++j) {
      double lo[2] = {(i - double(g2o)) / g2s - kWiden, (j - double(g2o)) / g2s - kWiden};
      double hi[2] = {(i + 1 - double(g2o)) / g2s + kWiden, (j + 1 - double(g2o)) / g2s + kWiden};
      if (i == 0) lo[0] = -inf;
      if (i == kGrid2 - 1) hi[0] = inf;
      if (j == 0) lo[1] = -inf;
      if (j == kGrid2 - 1) hi[1] = inf;
      int list[16], n = 0;
      for (int k = 0; k < K; ++k) {
        bool beaten = false;
        for (int o = 0; o < K && !beaten; ++o) {
          if (o == k) continue;
          double m = 0.0;   // max over the box of <u, C_k - C_o>
          for (int d = 0; d < 2; ++d) {
            const double a = double(cb[2 * k + d]) - double(cb[2 * o + d]);
            if (a > 0) m += a * hi[d];
            else if (a < 0) m += a * lo[d];
          }
          beaten = (double(cbh[k]) - double(cbh[o])) - m > kMargin;
        }
        if (!beaten) list[n++] = k;
      }
      if (n < 1 || n > 4) return false;
      uint32_t e = 0;
      for (int t = 0; t < 4; ++t) e |= uint32_t(list[t < n ? t : n - 1]) << (4 * t);
      tab[i * kGrid2 + j] = uint16_t(e);   // cell (gx = i, gy = j)
    }
  return true;
}

int set_hip_error(hipError_t e) {
  g_last_hip = int(e);
  return RSLM_ERR_HIP;
}

int check_launch() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? RSLM_OK : set_hip_error(e);
}

bool device_ok() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return false;
  return std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
}

// E_max(D) = E[max_{i<=D} |Z_i|] for i.i.d. standard normal Z_i
//          = integral_0^inf P(max |Z_i| > t) dt = integral_0^inf 1 - (1 - erfc(t/sqrt2))^D dt.
// Composite Simpson on [0, 16] (the tail beyond is below D * 1e-57).
static double emax_of(int D) {
  const int n = 1 << 18;
  const double a = 0.0, b = 16.0, h = (b - a) / n;
  auto f = [D](double t) {
    double q = std::erfc(t / std::sqrt(2.0));          // P(|Z| > t)
    return -std::expm1(double(D) * std::log1p(-q));    // 1 - (1 - q)^D
  };
  double s = f(a) + f(b);
  for (int i = 1; i < n; ++i) s += f(a + i * h) * ((i & 1) ? 4.0 : 2.0);
  return s * h / 3.0;
}

static bool f16_exact(float v) {
  _Float16 h = static_cast<_Float16>(v);
  return static_cast<float>(h) == v;
}

static uint16_t f16_bits(float v) {
  _Float16 h = static_cast<_Float16>(v);
  uint16_t b;
  std::memcpy(&b, &h, 2);
  return b;
}

}  // namespace rslm

using namespace rslm;

extern "C" {

const char *rslm_status_string(int s) {
  switch (s) {
    case RSLM_OK: return "ok";
    case RSLM_ERR_INVALID_ARG: return "invalid argument";
    case RSLM_ERR_UNSUPPORTED: return "unsupported";
    case RSLM_ERR_HIP: return "HIP error";
    case RSLM_ERR_WORKSPACE: return "workspace too small";
    case RSLM_ERR_NO_DEVICE: return "no gfx950 device";
    default: return "unknown status";
  }
}

int rslm_last_hip_error(void) { return g_last_hip; }

const char *rslm_version(void) { return "0.1.0"; }

size_t rslm_workspace_size(int call, const rslm_plan *plan, const rslm_index *index, int64_t n,
                           int32_t dim, int32_t nlist, int32_t nprobe, int32_t k) {
  switch (call) {
    case RSLM_WS_SCAN_TOPK:
      if (n < 0 || n > 0x7fffffff) return 0;
      return rslm_scan_topk_workspace(plan, index, int32_t(n), nprobe, k);
    case RSLM_WS_ASSIGN_L2: return ivf_assign_probe_workspace(n, dim, nlist, 1, IVF_ASSIGN_L2);
    case RSLM_WS_PROBE_IP: return ivf_assign_probe_workspace(n, dim, nlist, nprobe, IVF_PROBE_IP);
    case RSLM_WS_KMEANS_UPDATE: return ivf_kmeans_update_workspace(n, nlist);
    default: return 0;
  }
}

int rslm_plan_create(const rslm_plan_desc *d, rslm_plan **out) {
  if (!d || !out || !d->signs || !d->perm || !d->codebook) return RSLM_ERR_INVALID_ARG;
  if (d->dim < 1 || d->dim > kMaxDim) return RSLM_ERR_INVALID_ARG;
  if (d->bits < 1 || d->bits > 4) return RSLM_ERR_INVALID_ARG;
  if (d->passes < -1 || d->passes > 2) return RSLM_ERR_INVALID_ARG;
  if (d->scale_mode != 0 && d->scale_mode != 1) return RSLM_ERR_INVALID_ARG;
  for (int i = 0; i < 256; ++i)
    if (d->signs[i] != 1 && d->signs[i] != -1) return RSLM_ERR_INVALID_ARG;
  {
    bool seen[128] = {};
    for (int i = 0; i < 128; ++i) {
      int p = d->perm[i];
      if (p < 0 || p >= 128 || seen[p]) return RSLM_ERR_INVALID_ARG;
      seen[p] = true;
    }
  }
  const int D = d->dim, bits = d->bits;
  static const int kK[5] = {0, 16, 16, 8, 16};
  static const int kG[5] = {0, 4, 2, 1, 1};
  const int K = kK[bits], g = kG[bits];
  for (int i = 0; i < K * g; ++i) {
    float v = d->codebook[i];
    if (!std::isfinite(v) || !f16_exact(v)) return RSLM_ERR_INVALID_ARG;
  }
  if (g == 1)
    for (int k = 0; k + 1 < K; ++k)
      if (!(d->codebook[k] < d->codebook[k + 1])) return RSLM_ERR_INVALID_ARG;
  if (d->lite != 0 && d->lite != 1) return RSLM_ERR_INVALID_ARG;
  if (d->lite) {
    if (bits != 4 || D < 64 || !d->codebook_lead) return RSLM_ERR_INVALID_ARG;
    for (int k = 0; k < 8; ++k) {
      const float v = d->codebook_lead[k];
      if (!std::isfinite(v) || !f16_exact(v)) return RSLM_ERR_INVALID_ARG;
      if (k > 0 && !(d->codebook_lead[k - 1] < v)) return RSLM_ERR_INVALID_ARG;
    }
  }
  if (!device_ok()) return RSLM_ERR_NO_DEVICE;

  rslm_plan *p = new (std::nothrow) rslm_plan();
  if (!p) return RSLM_ERR_HIP;
  (void)hipGetDevice(&p->device);
  std::memcpy(p->signs, d->signs, 256);
  std::memcpy(p->perm, d->perm, 128 * sizeof(int32_t));

  // --- rotation parameters (block size, full blocks, overlap block, passes)
  RotParams &r = p->rot;
  r.D = D;
  r.B = (D >= 128) ? 128 : (1 << (31 - __builtin_clz(unsigned(D))));
  r.logB = 31 - __builtin_clz(unsigned(r.B));
  r.n_full = D / r.B;
  r.overlap = (D % r.B) != 0;
  r.passes = (d->passes >= 0) ? d->passes : ((bits == 4 && D <= 256) ? 1 : 2);
  r.inv_sqrt_b = float(1.0 / std::sqrt(double(r.B)));

  // --- codec parameters
  CodecParams &c = p->codec;
  c.D = D;
  c.bits = bits;
  c.K = K;
  c.g = g;
  c.w = (K == 16) ? 4 : 3;
  c.n_sub = (D + g - 1) / g;
  // The scan kernel is instantiated for these chunk counts (32 coordinates
  // each); the padded dimension is rounded up to the next one so that the
  // kernel's chunk loop is fully static.  Padding coordinates carry code 0
  // and meet zero query coordinates.
  // Above 32 chunks the scan runs in passes over equal chunk ranges of 16,
  // 24 or 32 chunks whose codes start on a 16-byte unit of a lane's stream
  // (chunks x bits a multiple of 16); the count is the smallest such total.
  {
    static const int kInst[] = {1, 2, 3, 4, 6, 8, 12, 16, 24, 32};
    int nc = (D + 31) / 32;
    if (nc <= 32) {
      for (int v : kInst)
        if (v >= nc) {
          nc = v;
          break;
        }
    } else {
      int best = 0;
      for (int per : {32, 24, 16}) {
        if ((per * bits) % 16) continue;
        const int total = (nc + per - 1) / per * per;
        if (!best || total < best) best = total;
      }
      nc = best;
    }
    c.n_chunks = nc;
    c.d_pad = nc * 32;
  }
  c.lane_bytes = (c.n_chunks * bits + 15) / 16 * 16;
  c.tile_bytes = 64 * c.lane_bytes;
  c.canon_bytes = (c.n_sub * c.w + 7) / 8;
  c.global = d->scale_mode;
  p->emax = emax_of(D);
  c.emax = float(p->emax);
  for (int i = 0; i < 64; ++i) c.cb[i] = (i < K * g) ? d->codebook[i] : 0.0f;
  for (int k = 0; k < 16; ++k) c.cbh[k] = (k < K) ? half_norm2(d->codebook + k * g, g) : 3.0e38f;
  for (int k = 0; k < 16; ++k)
    c.thr[k] = (g == 1 && k + 1 < K) ? 0.5f * (d->codebook[k] + d->codebook[k + 1]) : 0.0f;
  c.lead = d->lite ? (d->scale_mode ? 32 : 16) : 0;
  c.record_bytes = c.canon_bytes + (d->lite ? 0 : (d->scale_mode ? 4 : 2));
  for (int k = 0; k < 8; ++k) c.cb_lead[k] = d->lite ? d->codebook_lead[k] : 0.0f;
  for (int k = 0; k < 16; ++k)
    c.thr_lead[k] = (d->lite && k < 7) ? 0.5f * (d->codebook_lead[k] + d->codebook_lead[k + 1])
                                       : __builtin_inff();
  quant_grid(c.thr, g == 1 ? K - 1 : 0, c.qs, c.qo, c.qn);
  quant_grid(c.thr_lead, d->lite ? 7 : 0, c.qs_lead, c.qo_lead, c.qn_lead);
  // 2-D codebooks: nearest-centroid grid over [-emax, emax]^2 (|u| <= emax)
  uint16_t g2[kGrid2 * kGrid2];
  c.g2s = float(kGrid2) / (2.0f * c.emax);
  c.g2o = float(kGrid2 / 2);
  c.g2tab = nullptr;
  const bool has_g2 = g == 2 && grid2_lists(c.cb, c.cbh, K, c.g2s, c.g2o, g2);

  // --- device tables: signs, intra-block permutation, compact decode table
  float s1f[256];
  for (int i = 0; i < 256; ++i) s1f[i] = float(d->signs[i]);
  int16_t pi[128];
  for (int k = 0; k < r.B; ++k) {
    if (r.B == 128) {
      pi[k] = int16_t(d->perm[k]);
    } else {
      int v = 0;
      for (int t = 0; t < r.logB; ++t)
        if ((k >> t) & 1) v |= 1 << (r.logB - 1 - t);
      pi[k] = int16_t(v);
    }
  }
  // Decode table: symbol -> the float16 centroid values it stands for.
  //   bits 4: symbol = a byte (two 1-D codes), entry = half2(C[lo], C[hi])
  //   bits 3: symbol = 6 bits (two 3-bit codes), entry = half2
  //   bits 2: symbol = a nibble (one 2-D centroid), entry = half2
  //   bits 1: symbol = a nibble (one 4-D centroid), entry = half4
  uint32_t tab[512];
  int entries = 0, words = 1;
  auto h = [&](int k, int j) { return uint32_t(f16_bits(d->codebook[k * g + j])); };
  if (bits == 4) {
    entries = 256;
    for (int s = 0; s < 256; ++s) tab[s] = h(s & 15, 0) | (h(s >> 4, 0) << 16);
  } else if (bits == 3) {
    entries = 64;
    for (int s = 0; s < 64; ++s) tab[s] = h(s & 7, 0) | (h(s >> 3, 0) << 16);
  } else if (bits == 2) {
    entries = 16;
    for (int s = 0; s < 16; ++s) tab[s] = h(s, 0) | (h(s, 1) << 16);
  } else {
    entries = 16;
    words = 2;
    for (int s = 0; s < 16; ++s) {
      tab[2 * s] = h(s, 0) | (h(s, 1) << 16);
      tab[2 * s + 1] = h(s, 2) | (h(s, 3) << 16);
    }
  }
  p->dtab_entries = entries;
  p->dtab_words = words;

  // source index of every output of the strided transpose, x'[k M + b] = x[b B + P(k)]
  // for the first M B outputs, identity on the tail
  int16_t *tsrc = new (std::nothrow) int16_t[D];
  if (!tsrc) {
    rslm_plan_destroy(p);
    return RSLM_ERR_HIP;
  }
  {
    const int M = r.n_full, MB = r.n_full * r.B;
    for (int o = 0; o < D; ++o) tsrc[o] = int16_t(o < MB ? (o % M) * r.B + pi[o / M] : o);
  }
  hipError_t e;
  if ((e = hipMalloc(&p->d_tsrc, sizeof(int16_t) * D)) != hipSuccess ||
      (e = hipMemcpy(p->d_tsrc, tsrc, sizeof(int16_t) * D, hipMemcpyHostToDevice)) != hipSuccess) {
    delete[] tsrc;
    rslm_plan_destroy(p);
    return set_hip_error(e);
  }
  delete[] tsrc;
  if ((e = hipMalloc(&p->d_s1, sizeof(s1f))) != hipSuccess ||
      (e = hipMalloc(&p->d_pi, sizeof(pi))) != hipSuccess ||
      (e = hipMalloc(&p->d_dtab, sizeof(uint32_t) * entries * words)) != hipSuccess) {
    rslm_plan_destroy(p);
    return set_hip_error(e);
  }
  if ((e = hipMemcpy(p->d_s1, s1f, sizeof(s1f), hipMemcpyHostToDevice)) != hipSuccess ||
      (e = hipMemcpy(p->d_pi, pi, sizeof(pi), hipMemcpyHostToDevice)) != hipSuccess ||
      (e = hipMemcpy(p->d_dtab, tab, sizeof(uint32_t) * entries * words,
                     hipMemcpyHostToDevice)) != hipSuccess) {
    rslm_plan_destroy(p);
    return set_hip_error(e);
  }
  if (has_g2) {
    if ((e = hipMalloc(&p->d_g2tab, sizeof(g2))) != hipSuccess ||
        (e = hipMemcpy(p->d_g2tab, g2, sizeof(g2), hipMemcpyHostToDevice)) != hipSuccess) {
      rslm_plan_destroy(p);
      return set_hip_error(e);
    }
    c.g2tab = p->d_g2tab;
  }
  r.s1 = p->d_s1;
  r.pi = p->d_pi;
  r.tsrc = p->d_tsrc;
  for (int w = 0; w < 8; ++w) {
    uint32_t m = 0;
    for (int b = 0; b < 32; ++b)
      if (d->signs[w * 32 + b] < 0) m |= 1u << b;
    r.s1mask[w] = m;
  }
  *out = p;
  return RSLM_OK;
}

int rslm_grid2_lists(const float *codebook, int32_t K, float emax, uint16_t *out,
                     float *scale_offset) {
  if (!codebook || !out || !scale_offset || K < 1 || K > 16 || !(emax > 0.0f) ||
      !std::isfinite(emax))
    return RSLM_ERR_INVALID_ARG;
  float cb[32], cbh[16];
  for (int k = 0; k < K; ++k) {
    cb[2 * k] = codebook[2 * k];
    cb[2 * k + 1] = codebook[2 * k + 1];
    if (!std::isfinite(cb[2 * k]) || !std::isfinite(cb[2 * k + 1])) return RSLM_ERR_INVALID_ARG;
    cbh[k] = half_norm2(cb + 2 * k, 2);
  }
  const float s = float(kGrid2) / (2.0f * emax), o = float(kGrid2 / 2);
  uint16_t tab[kGrid2 * kGrid2];
  if (!grid2_lists(cb, cbh, K, s, o, tab)) return RSLM_ERR_UNSUPPORTED;
  std::memcpy(out, tab, sizeof(tab));
  scale_offset[0] = s;
  scale_offset[1] = o;
  return RSLM_OK;
}

int rslm_plan_destroy(rslm_plan *p) {
  if (!p) return RSLM_ERR_INVALID_ARG;
  if (p->d_s1) (void)hipFree(p->d_s1);
  if (p->d_pi) (void)hipFree(p->d_pi);
  if (p->d_dtab) (void)hipFree(p->d_dtab);
  if (p->d_tsrc) (void)hipFree(p->d_tsrc);
  if (p->d_g2tab) (void)hipFree(p->d_g2tab);
  delete p;
  return RSLM_OK;
}

int rslm_plan_get_info(const rslm_plan *p, rslm_plan_info *info) {
  if (!p || !info) return RSLM_ERR_INVALID_ARG;
  info->dim = p->rot.D;
  info->bits = p->codec.bits;
  info->passes = p->rot.passes;
  info->scale_mode = p->codec.global;
  info->K = p->codec.K;
  info->g = p->codec.g;
  info->block = p->rot.B;
  info->n_full_blocks = p->rot.n_full;
  info->d_pad = p->codec.d_pad;
  info->canon_bytes = p->codec.canon_bytes;
  info->tile_records = kTileRecords;
  info->tile_bytes = p->codec.tile_bytes;
  info->emax = p->emax;
  info->lite = p->codec.lead > 0;
  info->record_bytes = p->codec.record_bytes;
  return RSLM_OK;
}

}  // extern "C"
