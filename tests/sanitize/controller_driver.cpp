// Drives every entry point of the threshold controller (include/dlm_ctl.h)
// over random and edge-case arguments, for a build with AddressSanitizer and
// UndefinedBehaviorSanitizer (tests/test_sanitizers.py). Exit status 0 when
// every call returned and every valid call returned DLM_OK.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "../../include/dlm_ctl.h"

static int failures = 0;
#define EXPECT(cond)                                                      \
  do {                                                                    \
    if (!(cond)) {                                                        \
      std::fprintf(stderr, "line %d: %s\n", __LINE__, #cond);             \
      ++failures;                                                         \
    }                                                                     \
  } while (0)

int main() {
  std::mt19937_64 rng(7);
  auto uni = [&](double a, double b) { return std::uniform_real_distribution<double>(a, b)(rng); };
  auto ri = [&](int a, int b) { return std::uniform_int_distribution<int>(a, b)(rng); };
  for (int trial = 0; trial < 2000; ++trial) {
    const int ng = ri(1, 32);
    std::vector<double> gam(ng);
    for (int i = 0; i < ng; ++i) gam[i] = 0.01 + 0.03 * i;
    const int np = ri(1, 6), nc = ri(0, 4);
    std::vector<double> pt(np), pl(np), ct(nc), cl(nc);
    double t = 0;
    for (int i = 0; i < np; ++i) { t += uni(1, 500); pt[i] = t; pl[i] = uni(0.001, 0.2); }
    t = 0;
    for (int i = 0; i < nc; ++i) { t += uni(1, 300); ct[i] = t; cl[i] = uni(0.001, 0.05); }
    dlm_ctl_profile prof{{np, pt.data(), pl.data()}, {nc, nc ? ct.data() : nullptr, nc ? cl.data() : nullptr}};
    dlm_ctl_params P{ng, gam.data(), ri(0, 1) ? 32 : 0, ri(1, 64), uni(0.5, 30)};
    const int n = ri(0, 70);
    std::vector<std::vector<double>> steps(n, std::vector<double>(ng));
    std::vector<dlm_ctl_req> reqs(n);
    for (int i = 0; i < n; ++i) {
      double s = uni(1, 5);
      for (int g = 0; g < ng; ++g) { s += uni(0, 20); steps[i][g] = s; }
      reqs[i] = dlm_ctl_req{uni(16, 4096), std::floor(uni(0, steps[i][0])), steps[i].data(),
                            uni(0, 50), 0u, -1};
    }
    double lat = 0, cap = 0, tl = 0, ld = 0;
    EXPECT(dlm_ctl_latency(&prof.recompute, uni(0, 5000), &lat) == DLM_OK && lat > -1e300);
    const dlm_ctl_profile profs[3] = {prof, prof, prof};
    EXPECT(dlm_ctl_capacity(&P, profs, ri(0, 3), uni(64, 4096), &cap) == DLM_OK);
    const double c = ri(0, 3) == 0 ? INFINITY : cap * uni(0, 2);
    EXPECT(dlm_ctl_update_allowed(&P, n ? reqs.data() : nullptr, n, c) == DLM_OK);
    dlm_ctl_instance inst{&prof, uni(0, 8000), ri(0, 64)};
    for (int i = 0; i < n; ++i) {
      EXPECT(reqs[i].allowed & 1u);
      EXPECT(dlm_ctl_update_threshold(&P, &inst, &reqs[i]) == DLM_OK);
      EXPECT(reqs[i].gamma_idx >= 0 && reqs[i].gamma_idx < ng);
      const int g = ri(0, ng - 1);
      EXPECT(dlm_ctl_predicted_time_left(&P, &inst, &reqs[i], g, &tl) == DLM_OK);
      EXPECT(dlm_ctl_req_load(&P, &reqs[i], g, &ld) == DLM_OK);
    }
    // rejected arguments leave everything untouched and set a message
    if (n > 0) {
      dlm_ctl_req r = reqs[0];
      r.allowed = 0;
      EXPECT(dlm_ctl_update_threshold(&P, &inst, &r) == DLM_EINVAL);
      EXPECT(dlm_ctl_last_error()[0] != 0);
      EXPECT(dlm_ctl_predicted_time_left(&P, &inst, &reqs[0], ng, &tl) == DLM_EINVAL);
      EXPECT(dlm_ctl_req_load(&P, &reqs[0], -1, &ld) == DLM_EINVAL);
      EXPECT(dlm_ctl_update_allowed(&P, reqs.data(), n, NAN) == DLM_EINVAL);
    }
    EXPECT(dlm_ctl_update_allowed(nullptr, nullptr, 0, 1.0) == DLM_EINVAL);
    EXPECT(dlm_ctl_update_allowed(&P, nullptr, 3, 1.0) == DLM_EINVAL);
    EXPECT(dlm_ctl_latency(nullptr, 1.0, &lat) == DLM_EINVAL);
    EXPECT(dlm_ctl_capacity(&P, nullptr, 2, 100.0, &cap) == DLM_EINVAL);
  }
  std::printf("controller driver: %d failures\n", failures);
  return failures ? 1 : 0;
}
