// Host-side check of librslm's argument validation under AddressSanitizer and
// UndefinedBehaviorSanitizer (built by tests/test_abi_sanitizers.py with the
// sanitizers on the host code only; no GPU needed).  Every entry point is
// called with arguments that validation must reject before any launch, and
// the status strings, version and workspace-size functions are exercised at
// the edges of their ranges.  Exit status 0 when every call returned the
// expected status; the sanitizers abort on any memory or UB error.
#include <cmath>
#include <cstdio>
#include <cstdint>
#include <cstring>
#include <vector>

#include "../include/rslm.h"

static int failures = 0;
#define EXPECT(call, want)                                                     \
  do {                                                                         \
    const int got_ = (call);                                                   \
    if (got_ != (want)) {                                                      \
      std::printf("FAIL %s: got %d want %d\n", #call, got_, int(want));        \
      ++failures;                                                              \
    }                                                                          \
  } while (0)

int main() {
  for (int s = -3; s < 12; ++s) {
    const char *t = rslm_status_string(s);
    if (!t || !std::strlen(t)) ++failures;
  }
  if (std::strlen(rslm_version()) < 5) ++failures;
  (void)rslm_last_hip_error();

  // plan descriptors: valid tables, one field out of range at a time
  std::vector<int8_t> signs(256, 1);
  std::vector<int32_t> perm(128);
  for (int i = 0; i < 128; ++i) perm[i] = 127 - i;
  std::vector<float> cb(64);   // K = 16 centroids of g = 4 (bits 4)
  for (int k = 0; k < 64; ++k) cb[k] = -2.0f + 0.0625f * float(k);   // float16-exact
  std::vector<float> cb8(8);
  for (int k = 0; k < 8; ++k) cb8[k] = -1.0f + 0.25f * float(k);
  rslm_plan_desc d{};
  auto reset = [&]() {
    d.dim = 96; d.bits = 4; d.passes = -1; d.scale_mode = 1;
    d.signs = signs.data(); d.perm = perm.data(); d.codebook = cb.data();
    d.lite = 0; d.codebook_lead = cb8.data();
  };
  rslm_plan *plan = nullptr;
  reset(); d.dim = 0;      EXPECT(rslm_plan_create(&d, &plan), RSLM_ERR_INVALID_ARG);
  reset(); d.dim = 5000;   EXPECT(rslm_plan_create(&d, &plan), RSLM_ERR_INVALID_ARG);
  reset(); d.bits = 5;     EXPECT(rslm_plan_create(&d, &plan), RSLM_ERR_INVALID_ARG);
  reset(); d.passes = 3;   EXPECT(rslm_plan_create(&d, &plan), RSLM_ERR_INVALID_ARG);
  reset(); d.scale_mode = 2; EXPECT(rslm_plan_create(&d, &plan), RSLM_ERR_INVALID_ARG);
  reset(); d.signs = nullptr; EXPECT(rslm_plan_create(&d, &plan), RSLM_ERR_INVALID_ARG);
  reset(); d.lite = 1; d.dim = 32; EXPECT(rslm_plan_create(&d, &plan), RSLM_ERR_INVALID_ARG);
  {
    std::vector<int32_t> bad(perm);
    bad[5] = bad[6];
    reset(); d.perm = bad.data(); EXPECT(rslm_plan_create(&d, &plan), RSLM_ERR_INVALID_ARG);
  }
  {
    std::vector<float> bad(cb);
    bad[3] = 0.1f;   // not float16-exact
    reset(); d.codebook = bad.data(); EXPECT(rslm_plan_create(&d, &plan), RSLM_ERR_INVALID_ARG);
  }
  EXPECT(rslm_plan_create(nullptr, &plan), RSLM_ERR_INVALID_ARG);
  // a valid descriptor passes every check and stops at the device check
  // (no GPU visible), which shows the rejections above came from their fields
  reset(); EXPECT(rslm_plan_create(&d, &plan), RSLM_ERR_NO_DEVICE);
  reset(); d.lite = 1; EXPECT(rslm_plan_create(&d, &plan), RSLM_ERR_NO_DEVICE);
  EXPECT(rslm_plan_destroy(nullptr), RSLM_ERR_INVALID_ARG);
  rslm_plan_info info{};
  EXPECT(rslm_plan_get_info(nullptr, &info), RSLM_ERR_INVALID_ARG);

  // entry points with a null plan or out-of-range sizes
  float fbuf[64] = {0};
  EXPECT(rslm_fwht(nullptr, fbuf, fbuf, 4, 0, nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(rslm_encode(nullptr, fbuf, 1, nullptr, nullptr, 1, nullptr, nullptr, 0, nullptr, nullptr,
                     nullptr, nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(rslm_encode_two_stage(nullptr, nullptr, fbuf, 1, nullptr, nullptr, 1, nullptr, nullptr, 0,
                               nullptr, nullptr, nullptr, nullptr, nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(rslm_encode_sq8(nullptr, fbuf, 1, nullptr, nullptr, 1, nullptr, nullptr, 0, nullptr,
                         nullptr, nullptr, nullptr, nullptr, nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(rslm_decode(nullptr, nullptr, nullptr, 1, nullptr, nullptr, 0, fbuf, nullptr),
         RSLM_ERR_INVALID_ARG);
  EXPECT(rslm_pack_codes(nullptr, nullptr, 1, nullptr, nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(rslm_unpack_codes(nullptr, nullptr, 1, nullptr, nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(rslm_pack_records(nullptr, nullptr, nullptr, 1, nullptr, nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(rslm_score(nullptr, nullptr, 1, nullptr, 1, fbuf, 1, fbuf, nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(ivf_assign_probe(nullptr, 4, 8, nullptr, 0, 1, IVF_ASSIGN_L2, nullptr, nullptr, nullptr, 0,
                          nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(ivf_assign_probe(nullptr, 4, 8, nullptr, 16, 17, IVF_PROBE_IP, nullptr, nullptr, nullptr, 0,
                          nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(ivf_assign_probe(nullptr, 4, 8, nullptr, 16, 2, 7, nullptr, nullptr, nullptr, 0, nullptr),
         RSLM_ERR_INVALID_ARG);
  EXPECT(ivf_assign_probe_noalloc(nullptr, 4, 8, nullptr, 16, 2, IVF_ASSIGN_L2, nullptr, nullptr,
                                  nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(ivf_kmeans_update(nullptr, 4, 8, nullptr, 0, nullptr, nullptr, 0, nullptr),
         RSLM_ERR_INVALID_ARG);
  EXPECT(ivf_kmeans_update(nullptr, int64_t(1) << 40, 8, nullptr, 16, fbuf, nullptr, 0, nullptr),
         RSLM_ERR_INVALID_ARG);
  rslm_index idx{};
  EXPECT(rslm_scan_topk(nullptr, &idx, fbuf, 1, nullptr, fbuf, 1, 10, fbuf, nullptr, nullptr, 0,
                        nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(rslm_sq8_fit(nullptr, 4, 0, nullptr, nullptr, 0, nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(rslm_sq8_encode(nullptr, 4, 0, nullptr, nullptr, nullptr, 0, nullptr, nullptr),
         RSLM_ERR_INVALID_ARG);
  rslm_rescore_codec codec{};
  codec.kind = 7;
  EXPECT(rslm_rescore(&codec, fbuf, 1, fbuf, nullptr, 10, 10, fbuf, nullptr, nullptr),
         RSLM_ERR_UNSUPPORTED);
  codec.kind = RSLM_RESCORE_SQ8;
  codec.dim = 8;
  EXPECT(rslm_rescore(&codec, fbuf, 1, fbuf, nullptr, 10, 20, fbuf, nullptr, nullptr),
         RSLM_ERR_INVALID_ARG);
  EXPECT(rslm_set_timer(5, nullptr, nullptr), RSLM_ERR_INVALID_ARG);
  EXPECT(rslm_calibrate_read(nullptr, 16, nullptr, 1, 0, nullptr), RSLM_ERR_INVALID_ARG);
  // the 2-D nearest-centroid lists: host code, run in full here
  {
    float cb2d[32], so[2];
    uint16_t lists[RSLM_GRID2 * RSLM_GRID2];
    for (int k = 0; k < 9; ++k) {   // a centre code and a ring of 8 (K = 9)
      const double a = 6.283185307179586 * k / 8.0, rad = k ? 1.5 : 0.0;
      cb2d[2 * k] = float(rad * std::cos(a));
      cb2d[2 * k + 1] = float(rad * std::sin(a));
    }
    EXPECT(rslm_grid2_lists(cb2d, 9, 3.36f, lists, so), RSLM_OK);
    float ring[32];   // 16 codes on one ring: the outer corner cells, which
    for (int k = 0; k < 16; ++k) {   // extend to infinity over a quarter of the
      const double a = 6.283185307179586 * k / 16.0;   // directions, need more than four
      ring[2 * k] = float(1.5 * std::cos(a));
      ring[2 * k + 1] = float(1.5 * std::sin(a));
    }
    EXPECT(rslm_grid2_lists(ring, 16, 3.36f, lists, so), RSLM_ERR_UNSUPPORTED);
    EXPECT(rslm_grid2_lists(cb2d, 0, 3.36f, lists, so), RSLM_ERR_INVALID_ARG);
    EXPECT(rslm_grid2_lists(cb2d, 17, 3.36f, lists, so), RSLM_ERR_INVALID_ARG);
    EXPECT(rslm_grid2_lists(cb2d, 9, -1.0f, lists, so), RSLM_ERR_INVALID_ARG);
    EXPECT(rslm_grid2_lists(nullptr, 9, 3.36f, lists, so), RSLM_ERR_INVALID_ARG);
    EXPECT(rslm_grid2_lists(cb2d, 9, 3.36f, nullptr, so), RSLM_ERR_INVALID_ARG);
  }

  // workspace sizes at the edges of their ranges (host arithmetic only)
  (void)ivf_assign_probe_workspace(int64_t(1) << 31, 4096, 65536, 1024, IVF_PROBE_IP);
  (void)ivf_assign_probe_workspace(-1, 4096, 65536, 1024, IVF_PROBE_IP);
  (void)ivf_kmeans_update_workspace(int64_t(1) << 31, 65536);
  (void)ivf_assign_probe_noalloc_limit();
  (void)rslm_scan_topk_workspace(nullptr, &idx, 65535, 1024, 1024);
  for (int call = -1; call < 5; ++call) {
    (void)rslm_workspace_size(call, nullptr, &idx, int64_t(1) << 40, 4096, 65536, 1024, 1024);
    (void)rslm_workspace_size(call, nullptr, nullptr, -5, -1, 0, 0, 0);
  }

  std::printf("%s (%d failures)\n", failures ? "FAILED" : "ok", failures);
  return failures ? 1 : 0;
}
