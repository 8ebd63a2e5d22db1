// Drives the host side of libdlm (include/dlm.h): configuration checks, the
// workspace and cache layouts, the step planner and every validation path of
// the step entry points, over random and edge-case arguments, for a build of
// the library's host code with AddressSanitizer and UndefinedBehaviorSanitizer
// (tests/test_sanitizers.py). Device pointers are fake: no call here reaches a
// kernel launch (each step is rejected before anything is enqueued), so the
// driver runs without a GPU.
#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

#include "../../include/dlm.h"

static int failures = 0;
#define EXPECT(cond)                                                      \
  do {                                                                    \
    if (!(cond)) {                                                        \
      std::fprintf(stderr, "line %d: %s\n", __LINE__, #cond);             \
      ++failures;                                                         \
    }                                                                     \
  } while (0)

int main() {
  std::mt19937_64 rng(11);
  auto ri = [&](int a, int b) { return std::uniform_int_distribution<int>(a, b)(rng); };
  char* fake = reinterpret_cast<char*>(uintptr_t(1) << 40);   // never dereferenced on the host
  const dlm_config shapes[] = {
      {2, 256, 4, 4, 64, 688, 2048, 2047, 1e-5f, 1e4f, 13.f, DLM_F32},
      {32, 4096, 32, 32, 128, 12288, 126464, 126463, 1e-5f, 1e4f, 8.f, DLM_BF16},
      {28, 3584, 28, 4, 128, 18944, 152064, 152063, 1e-5f, 1e4f, 11.f, DLM_BF16}};
  for (const dlm_config& cfg : shapes) {
    std::vector<dlm_layer_weights> lw(cfg.n_layers,
                                      dlm_layer_weights{(const float*)fake, fake, fake,
                                                        (const float*)fake, fake, fake});
    dlm_weights w{fake, fake, (const float*)fake, lw.data()};
    dlm_model* m = nullptr;
    EXPECT(dlm_load_weights(&cfg, &w, &m) == DLM_OK && m);
    size_t ws = 0, need = 0;
    for (int rows : {1, 17, 64, 255, 256, 512, 1000, 2048}) {
      EXPECT(dlm_workspace_bytes(m, rows, ri(1, 64), &ws) == DLM_OK && ws > 0);
    }
    EXPECT(dlm_workspace_bytes(m, 0, 1, &ws) == DLM_EINVAL);
    const int slots = 8, smax = 2304;
    EXPECT(dlm_kv_cache_alloc(m, slots, smax, nullptr, 0, &need, nullptr) == DLM_OK && need > 0);
    dlm_cache* c = nullptr;
    EXPECT(dlm_kv_cache_alloc(m, slots, smax, fake, need - 1, &need, &c) == DLM_ESIZE);
    EXPECT(dlm_kv_cache_alloc(m, slots, smax, fake, need, &need, &c) == DLM_OK && c);
    std::vector<int32_t> counts(64);
    dlm_step_out out{counts.data(), (int32_t*)fake, (int32_t*)fake, (float*)fake, nullptr,
                     nullptr, nullptr};
    for (int trial = 0; trial < 400; ++trial) {
      const int n = ri(1, slots);
      std::vector<dlm_req> reqs(n);
      std::vector<float> thr(n);
      int off = 0;
      for (int r = 0; r < n; ++r) {
        const int P = ri(0, 1500), G = ri(1, 700), B = ri(1, 64);
        const int L = std::min(P + G, smax);
        const int bs = std::min(P + B * ri(0, 3), L - 1);
        dlm_req q{r, L, std::min(P, bs), bs, std::min(B, L - bs), off, ri(0, 3) ? DLM_REQ_REFRESH : 0};
        if (ri(0, 19) == 0) q.slot = ri(-1, slots);           // sometimes invalid
        if (ri(0, 19) == 0) q.block_len = ri(-1, 70);
        if (ri(0, 29) == 0) q.tok_offset = off - 1;          // overlapping ranges
        reqs[r] = q;
        off += L + ri(0, 5);
        thr[r] = ri(0, 29) == 0 ? 1.5f : (float)ri(0, 100) / 100.f;
      }
      dlm_batch b{n, reqs.data(), (int32_t*)fake, (uint8_t*)fake, ri(0, 2), nullptr};
      // no workspace: rejected after planning, nothing enqueued
      const dlm_status s = dlm_denoise_step(m, c, &b, thr.data(), &out, nullptr, 0, nullptr);
      EXPECT(s == DLM_EINVAL || s == DLM_ESIZE || s == DLM_ESTATE);
      EXPECT(dlm_last_error()[0] != 0);
      EXPECT(dlm_cache_refresh(m, c, &b, nullptr, 0, nullptr) != DLM_OK);
      dlm_trace tr{};
      tr.layer = ri(-1, cfg.n_layers);
      EXPECT(dlm_debug_trace(m, c, &b, &tr, nullptr, 0, nullptr) != DLM_OK);
      // the fixed-scratch step: oversized steps are rejected before any device call
      const dlm_status s2 = dlm_denoise_step_noalloc(m, c, &b, thr.data(), &out, nullptr);
      EXPECT(s2 != DLM_OK);
    }
    EXPECT(dlm_cache_invalidate(c, slots) == DLM_EINVAL);
    EXPECT(dlm_cache_invalidate(c, 0) == DLM_OK);
    dlm_profile_entry pe[4];
    int32_t np = -1;
    EXPECT(dlm_profile_read(m, pe, 4, &np) == DLM_OK && np == 0);
    dlm_cache_destroy(c);
    dlm_model_destroy(m);
  }
  dlm_config bad = shapes[1];
  bad.head_dim = 96;
  dlm_model* m = nullptr;
  EXPECT(dlm_load_weights(&bad, nullptr, &m) != DLM_OK);
  std::printf("planner driver: %d failures\n", failures);
  return failures ? 1 : 0;
}
