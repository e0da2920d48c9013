// Host-side checks of the pvlm library under AddressSanitizer (no GPU):
// every entry point's argument validation (NULL pointers, sizes out of
// range, launch limits), the workspace-size queries at extreme sizes, and the
// host-only calls (window size, speedup model, the parallel-decoding
// scheduler driven through long randomised runs).  Built from the library's
// sources with host-side instrumentation only; a memory error aborts with an
// AddressSanitizer report, a wrong status fails with a message.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "pvlm.h"

static int g_fail = 0;
#define EXPECT(cond)                                                   \
  do {                                                                 \
    if (!(cond)) {                                                     \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++g_fail;                                                        \
    }                                                                  \
  } while (0)

static char g_buf[4096];
static void* const F = g_buf;  // a non-NULL pointer the checks never reach

static void validation() {
  for (int s = 0; s <= 6; ++s) EXPECT(pvlm_status_string((pvlm_status)s) != nullptr);
  EXPECT(pvlm_version() == 1);
  EXPECT(pvlm_last_hip_error() != nullptr);
  // verify: NULLs, shapes, unsupported
  auto verify = [](pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D, int64_t n_cap, int64_t max_ctx,
                   float scale, void* q) {
    return pvlm_verify_attn(dt, B, T, Hq, Hkv, D, n_cap, max_ctx, scale, q, F, F, (const int32_t*)F,
                            F, nullptr, nullptr, F, 1 << 30, nullptr, nullptr);
  };
  EXPECT(verify(PVLM_BF16, 1, 5, 8, 2, 128, 100, 95, 0.1f, nullptr) == PVLM_ERR_NULL);
  EXPECT(verify(PVLM_BF16, 0, 5, 8, 2, 128, 100, 95, 0.1f, F) == PVLM_ERR_SHAPE);
  EXPECT(verify(PVLM_BF16, 1, 5, 8, 2, 128, 100, 96, 0.1f, F) == PVLM_ERR_SHAPE);
  EXPECT(verify(PVLM_BF16, 1, 5, 8, 2, 128, 100, 95, NAN, F) == PVLM_ERR_SHAPE);
  EXPECT(verify(PVLM_BF16, 1, 33, 8, 2, 128, 100, 60, 0.1f, F) == PVLM_ERR_UNSUPPORTED);
  EXPECT(verify(PVLM_BF16, 1, 5, 8, 3, 128, 100, 95, 0.1f, F) == PVLM_ERR_UNSUPPORTED);
  EXPECT(verify(PVLM_BF16, 1, 5, 8, 2, 96, 100, 95, 0.1f, F) == PVLM_ERR_UNSUPPORTED);
  EXPECT(verify(PVLM_BF16, 1, 5, 8, 2, 128, (int64_t)1 << 31, 95, 0.1f, F) == PVLM_ERR_SHAPE);
  EXPECT(pvlm_verify_attn_workspace_size(PVLM_BF16, 0, 5, 8, 2, 128, 100, 95) == 0);
  // paged verify / gather / rope: page sizes and counts
  const int pages[] = {0, 16, 31, 48, 100, 1 << 21};
  for (int ps : pages) {
    EXPECT(pvlm_verify_attn_paged(PVLM_BF16, 1, 5, 8, 2, 128, ps, 4, 8, 100, 0.1f, F, F, F,
                                  (const int32_t*)F, (const int32_t*)F, F, nullptr, nullptr, F,
                                  1 << 30, nullptr, nullptr) == PVLM_ERR_SHAPE);
    EXPECT(pvlm_gather_kv_paged(PVLM_BF16, 1, 1, 1, 128, ps, 4, 8, F, F, (const int32_t*)F,
                                (const int32_t*)F, (const int32_t*)F, 4, (const int32_t*)F,
                                (const int32_t*)F, 8, F, F, nullptr, nullptr) == PVLM_ERR_SHAPE);
    EXPECT(pvlm_rope_append_paged(PVLM_BF16, 1, 4, 8, 2, 128, ps, 4, 8, 1e6, nullptr,
                                  (const int32_t*)F, F, F, F, (const int32_t*)F,
                                  (const int32_t*)F, F, F, F, nullptr, nullptr) == PVLM_ERR_SHAPE);
  }
  EXPECT(pvlm_verify_attn_paged(PVLM_F32, 1, 5, 8, 2, 128, 32, 4, 8, 100, 0.1f, F, F, F,
                                (const int32_t*)F, (const int32_t*)F, F, nullptr, nullptr, F,
                                1 << 30, nullptr, nullptr) == PVLM_ERR_UNSUPPORTED);
  EXPECT(pvlm_verify_attn_paged(PVLM_BF16, 1, 5, 8, 2, 128, 32, 4, 8, 100, 0.1f, F, F, F, nullptr,
                                (const int32_t*)F, F, nullptr, nullptr, F, 1 << 30, nullptr,
                                nullptr) == PVLM_ERR_NULL);
  // rope: one launch holds at most 2^32 - 256 rotation pairs
  EXPECT(pvlm_rope_append(PVLM_BF16, 4096, 32, 64, 8, 1024, 64, 1e6, nullptr, (const int32_t*)F, F,
                          F, F, (const int32_t*)F, F, F, F, nullptr, nullptr) == PVLM_ERR_SHAPE);
  const int32_t bad_sections[3] = {10, 10, 10};
  EXPECT(pvlm_rope_append(PVLM_BF16, 1, 4, 8, 2, 128, 64, 1e6, bad_sections, (const int32_t*)F, F,
                          F, F, (const int32_t*)F, F, F, F, nullptr, nullptr) == PVLM_ERR_SHAPE);
  // UV-Prune: launch limits, NULLs, workspace
  EXPECT(pvlm_uvprune_score(PVLM_CRIT_MASS, 8, 1, (int64_t)1 << 30, (const int32_t*)F,
                            (const float*)F, PVLM_BF16, 0, 0, nullptr, nullptr, nullptr, (float*)F,
                            nullptr, 0, nullptr, nullptr) == PVLM_ERR_SHAPE);
  EXPECT(pvlm_uvprune_score(PVLM_CRIT_COSSIM, 17, 2, 10, (const int32_t*)F, nullptr, PVLM_BF16, 8,
                            (1 << 21) - 32, (const int32_t*)F, F, F, (float*)F, F,
                            (size_t)1 << 40, nullptr, nullptr) == PVLM_ERR_SHAPE);
  EXPECT(pvlm_uvprune_criterion_cossim(1, 10, (const int32_t*)F, PVLM_BF16, 16384, 10,
                                       (const int32_t*)F, F, F, (float*)F, F, 1 << 30, nullptr,
                                       nullptr) == PVLM_ERR_UNSUPPORTED);
  EXPECT(pvlm_prefill_epilogue_cossim(1, 10, (const int32_t*)F, 10, (const int32_t*)F, PVLM_BF16,
                                      64, F, nullptr, F, F, F, F, (float*)F, F, 1 << 30, nullptr,
                                      nullptr) == PVLM_ERR_NULL);
  EXPECT(pvlm_uvprune_workspace_size(PVLM_CRIT_COSSIM, 0, 64, 10) == 0);
  // top-k, fused top-k, gather, accept
  EXPECT(pvlm_topk_select(0, 10, (const int32_t*)F, (const int32_t*)F, 4, (const float*)F,
                          (int32_t*)F, nullptr, 0, nullptr, nullptr) == PVLM_ERR_SHAPE);
  EXPECT(pvlm_uvprune_topk_mass(1, 0, 10, (const int32_t*)F, (const float*)F, (const int32_t*)F, 4,
                                nullptr, (int32_t*)F, nullptr, 0, nullptr, nullptr) == PVLM_ERR_SHAPE);
  EXPECT(pvlm_uvprune_topk_mass(1, 1, 10, (const int32_t*)F, nullptr, (const int32_t*)F, 4,
                                nullptr, (int32_t*)F, nullptr, 0, nullptr, nullptr) == PVLM_ERR_NULL);
  EXPECT(pvlm_topk_workspace_size(1, 0) == 0);
  EXPECT(pvlm_gather_kv(PVLM_BF16, 1, 1, 1, 3, 10, F, F, (const int32_t*)F, (const int32_t*)F, 4,
                        (const int32_t*)F, (const int32_t*)F, 8, F, F, nullptr, nullptr) ==
         PVLM_ERR_UNSUPPORTED);
  EXPECT(pvlm_spec_accept(1, 0, 10, 1.0f, (const float*)F, (const float*)F, (const int32_t*)F,
                          (const double*)F, (const double*)F, (int32_t*)F, (int32_t*)F, nullptr, F,
                          1 << 20, nullptr, nullptr) == PVLM_ERR_SHAPE);
  EXPECT(pvlm_spec_accept(1, 2, 10, -1.0f, (const float*)F, (const float*)F, (const int32_t*)F,
                          (const double*)F, (const double*)F, (int32_t*)F, (int32_t*)F, nullptr, F,
                          1 << 20, nullptr, nullptr) == PVLM_ERR_SHAPE);
  EXPECT(pvlm_spec_accept_workspace_size(300, 2, 10) == 0);
  EXPECT(pvlm_verify_attn_noalloc_max_bytes() == (size_t)32 << 20);
}

static void host_math() {
  pvlm_speedup_model m;
  EXPECT(pvlm_speedup(5.0, 0.8, 5, nullptr) == PVLM_ERR_NULL);
  EXPECT(pvlm_speedup(-1.0, 0.8, 5, &m) == PVLM_ERR_SHAPE);
  std::mt19937_64 rng(7);
  std::uniform_real_distribution<double> uc(0.1, 20.0), ut(0.0, 1.0);
  for (int i = 0; i < 20000; ++i) {
    const double c = uc(rng), tau = ut(rng);
    const int g = 1 + (int)(rng() % 64);
    EXPECT(pvlm_speedup(c, tau, g, &m) == PVLM_OK);
    int gamma = 0;
    double cc = 0.0;
    const pvlm_round rd = (pvlm_round)(rng() % 4);
    const pvlm_status st = pvlm_window_size(c * 47.0, 47.0, rd, tau, 64, &gamma, &cc);
    EXPECT(st == PVLM_OK || (rd == PVLM_ROUND_BEST && tau == 0.0));
    if (st == PVLM_OK) EXPECT(gamma >= 1 && gamma <= 64);
  }
  int gamma = 0;
  EXPECT(pvlm_window_size(NAN, 47.0, PVLM_ROUND_DOWN, 0.5, 64, &gamma, nullptr) == PVLM_ERR_SHAPE);
  EXPECT(pvlm_window_size(100.0, 47.0, (pvlm_round)9, 0.5, 64, &gamma, nullptr) == PVLM_ERR_SHAPE);
}

static uint32_t mix(uint64_t h) {
  h ^= h >> 33;
  h *= 0xff51afd7ed558ccdULL;
  h ^= h >> 33;
  return (uint32_t)h;
}

static void scheduler() {
  pvlm_pd* pd = nullptr;
  EXPECT(pvlm_pd_create(0, 3.0, 10, &pd) == PVLM_ERR_SHAPE);
  EXPECT(pvlm_pd_create(3, 3.0, 10, nullptr) == PVLM_ERR_NULL);
  std::mt19937_64 rng(11);
  for (int run = 0; run < 300; ++run) {
    const int gamma = 1 + (int)(rng() % 12), max_len = 1 + (int)(rng() % 400);
    const double c = 0.5 + (double)(rng() % 1000) / 100.0;
    EXPECT(pvlm_pd_create(gamma, c, max_len, &pd) == PVLM_OK);
    pvlm_pd_round rd;
    EXPECT(pvlm_pd_plan(pd, &rd) == PVLM_ERR_SHAPE);  // before start
    std::vector<int32_t> startup(gamma + 1);
    for (auto& t : startup) t = (int32_t)(rng() % 1000);
    EXPECT(pvlm_pd_start(pd, startup.data()) == PVLM_OK);
    EXPECT(pvlm_pd_start(pd, startup.data()) == PVLM_ERR_SHAPE);  // twice
    const uint64_t salt = rng();
    for (int guard = 0; guard < 100000; ++guard) {
      EXPECT(pvlm_pd_plan(pd, &rd) == PVLM_OK);
      if (rd.mode == PVLM_PD_DONE) break;
      std::vector<int32_t> drafted(rd.draft_count);
      for (auto& t : drafted) t = (int32_t)(mix(salt + guard * 131 + (&t - drafted.data())) % 1000);
      // a wrong drafted count leaves the state unchanged
      EXPECT(pvlm_pd_finish(pd, drafted.data(), rd.draft_count + 1, 0, 1) == PVLM_ERR_SHAPE);
      const int acc = (int)(mix(salt ^ (uint64_t)guard) % (uint32_t)(rd.verify_count + 1));
      EXPECT(pvlm_pd_finish(pd, drafted.data(), rd.draft_count, acc, (int32_t)(mix(guard) % 1000)) ==
             PVLM_OK);
    }
    int n = 0;
    EXPECT(pvlm_pd_output(pd, nullptr, 0, &n) == PVLM_OK);
    EXPECT(n >= max_len);
    std::vector<int32_t> out(n);
    EXPECT(pvlm_pd_output(pd, out.data(), n, &n) == PVLM_OK);
    if (n > 1) EXPECT(pvlm_pd_output(pd, out.data(), n - 1, &n) == PVLM_ERR_SHAPE);
    int np = 0;
    EXPECT(pvlm_pd_pending(pd, nullptr, 0, &np) == PVLM_OK);
    std::vector<int32_t> pend(np + 1);
    EXPECT(pvlm_pd_pending(pd, pend.data(), np + 1, &np) == PVLM_OK);
    pvlm_pd_stats st;
    EXPECT(pvlm_pd_get_stats(pd, &st) == PVLM_OK);
    EXPECT(st.committed == n && st.mode == PVLM_PD_DONE);
    EXPECT(pvlm_pd_finish(pd, nullptr, 0, 0, 0) == PVLM_ERR_SHAPE);  // finish when DONE
    pvlm_pd_destroy(pd);
    pd = nullptr;
  }
  pvlm_pd_destroy(nullptr);
}

int main() {
  validation();
  host_math();
  scheduler();
  if (g_fail) {
    std::fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("host checks: ok\n");
  return 0;
}
