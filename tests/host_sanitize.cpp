// Host half of the library (planner, flow export, traffic accounting, model,
// lower bounds, timeline) exercised under AddressSanitizer and
// UndefinedBehaviorSanitizer: built with g++ from optcc_plan.cpp only, no
// device code.  Sweeps one-GPU-per-server and several-GPUs-per-server
// profiles (p up to 1024, empty and ragged N, every slot range) and the
// error paths, and checks the invariants every plan must satisfy: segment
// lengths add up to N, the flow list has num_flows entries whose ranges lie
// inside [0, N), and the model time is not below the lower bound.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "optcc.h"
#include "optcc_internal.hpp"

// The executor (device code) defines this; the host-only build frees the
// plan directly, since no device tables were ever allocated.
extern "C" void optcc_plan_free(optcc_plan_t *pl) { delete pl; }

static int g_fail = 0;
#define EXPECT(c, ...)                     \
  do {                                     \
    if (!(c)) {                            \
      std::fprintf(stderr, __VA_ARGS__);   \
      std::fprintf(stderr, "\n");          \
      ++g_fail;                            \
    }                                      \
  } while (0)

static void exercise(optcc_plan_t *pl, const double *bw, bool servers, int q, int g) {
  optcc_plan_info_t info;
  EXPECT(optcc_plan_info(pl, &info, nullptr, nullptr, nullptr) == OPTCC_OK, "info");
  std::vector<int32_t> ring((size_t)std::max(info.healthy, 1)), strag((size_t)std::max(info.m, 1));
  std::vector<double> ell((size_t)info.p);
  EXPECT(optcc_plan_info(pl, &info, ring.data(), strag.data(), ell.data()) == OPTCC_OK, "info arrays");
  std::vector<int64_t> off((size_t)info.num_segments), len((size_t)info.num_segments),
      p2p((size_t)info.num_segments);
  EXPECT(optcc_plan_segments(pl, off.data(), len.data(), p2p.data()) == OPTCC_OK, "segments");
  int64_t total = 0;
  for (int s = 0; s < info.num_segments; ++s) total += len[(size_t)s];
  EXPECT(total == info.n, "segments cover %lld of %lld elements", (long long)total, (long long)info.n);
  const int64_t nf = optcc_plan_num_flows(pl);
  EXPECT(nf == info.num_flows, "num_flows");
  std::vector<optcc_flow_t> fl((size_t)std::max<int64_t>(nf, 1));
  EXPECT(optcc_plan_get_flows(pl, fl.data(), nf) == nf, "get_flows");
  EXPECT(optcc_plan_get_flows(pl, fl.data(), nf / 2) == nf, "get_flows with a short buffer");
  for (int64_t i = 0; i < nf; ++i) {
    const optcc_flow_t &f = fl[(size_t)i];
    EXPECT(f.offset >= 0 && f.length > 0 && f.offset + f.length <= info.n, "flow range");
    EXPECT(f.src >= 0 && f.src < info.p && f.dst >= 0 && f.dst < info.p && f.src != f.dst, "flow ranks");
    EXPECT(f.slot >= 0 && f.slot < info.num_slots, "flow slot");
  }
  for (int dt = 0; dt < 3; ++dt)
    for (int b = 0; b <= info.num_slots; ++b)
      for (int e = b; e <= info.num_slots; ++e)
        for (int launches = 0; launches <= 1; ++launches) {
          int64_t r = -1, w = -1;
          EXPECT(optcc_plan_traffic(pl, (optcc_dtype_t)dt, b, e, launches, &r, &w) == OPTCC_OK &&
                     r >= 0 && w >= 0,
                 "traffic");
        }
  const double t = optcc_model_time(pl, nullptr);
  EXPECT(t == optcc_model_time(pl, bw), "model time with the plan's bandwidths");
  const double lb = servers ? optcc_lower_bound_servers(q, g, bw, info.n)
                            : optcc_lower_bound(info.p, bw, info.n);
  EXPECT(std::isfinite(t) && std::isfinite(lb) && t >= lb * (1 - 1e-12), "model %g < bound %g", t, lb);
  if (nf <= 20000) {
    std::vector<double> st((size_t)std::max<int64_t>(nf, 1)), fi((size_t)std::max<int64_t>(nf, 1));
    double mk = -1;
    EXPECT(optcc_plan_timeline(pl, st.data(), fi.data(), nf, &mk) == OPTCC_OK, "timeline");
    EXPECT(mk >= lb * (1 - 1e-9), "evaluated %g < bound %g", mk, lb);
    for (int64_t i = 0; i < nf; ++i) EXPECT(fi[(size_t)i] > st[(size_t)i] && st[(size_t)i] >= 0, "flow times");
  }
}

int main() {
  std::mt19937_64 rng(2606);
  const int64_t sizes[] = {0, 1, 63, 64, 65, 1000, 64 * 53 + 9, 100003};
  // one GPU per server
  for (int p : {3, 4, 5, 6, 7, 8, 9, 12, 16, 33, 64, 128, 256, 1024}) {
    for (int m = 0; m <= 4; ++m) {
      if (p - m < 2) continue;
      std::vector<double> bw((size_t)p, 1.0);
      std::uniform_real_distribution<double> u(0.2, 0.999);
      for (int i = 0; i < m; ++i) bw[(size_t)(rng() % (uint64_t)p)] = u(rng);
      for (int64_t n : sizes) {
        for (int k : {4, 8, 12, 64}) {
          if (p >= 256 && k > 8 && n > 1000) continue;
          optcc_plan_t *pl = nullptr;
          const int rc = optcc_plan(p, bw.data(), n, k, &pl);
          if (rc == OPTCC_EUNSUPPORTED) continue;  // repeated picks left < 2 healthy
          EXPECT(rc == OPTCC_OK && pl, "optcc_plan p=%d n=%lld k=%d: %d %s", p, (long long)n, k, rc,
                 optcc_last_error());
          if (!pl) continue;
          exercise(pl, bw.data(), false, p, 1);
          optcc_plan_free(pl);
        }
      }
    }
  }
  // several GPUs per server
  for (int q : {3, 4, 5, 8, 16}) {
    for (int g : {2, 3, 4, 8}) {
      std::vector<double> bw((size_t)q, 1.0);
      bw[(size_t)(rng() % (uint64_t)q)] = std::uniform_real_distribution<double>(0.2, 0.999)(rng);
      for (int64_t n : sizes) {
        for (int k : {24, 32}) {
          optcc_plan_t *pl = nullptr;
          const int rc = optcc_plan_servers(q, g, bw.data(), n, k, &pl);
          EXPECT(rc == OPTCC_OK && pl, "optcc_plan_servers q=%d g=%d: %d %s", q, g, rc, optcc_last_error());
          if (!pl) continue;
          exercise(pl, bw.data(), true, q, g);
          optcc_plan_free(pl);
        }
      }
    }
  }
  // error paths: a status and a message, nothing allocated
  {
    double bw[4] = {1, 1, 1, 0.5}, bad[4] = {1, NAN, 1, 1};
    optcc_plan_t *pl = nullptr;
    EXPECT(optcc_plan(4, bw, 10, 6, &pl) == OPTCC_EINVAL && !pl, "k = 6");
    EXPECT(optcc_plan(4, bad, 10, 4, &pl) == OPTCC_EINVAL && !pl, "NaN bandwidth");
    EXPECT(optcc_plan(4, nullptr, 10, 4, &pl) == OPTCC_EINVAL && !pl, "NULL bandwidths");
    EXPECT(optcc_plan(4, bw, -1, 4, &pl) == OPTCC_EINVAL && !pl, "N < 0");
    EXPECT(optcc_plan(2, bw, 10, 4, &pl) == OPTCC_EUNSUPPORTED && !pl, "p = 2");
    EXPECT(optcc_plan(4, bw, 10, 4, nullptr) == OPTCC_EINVAL, "NULL out");
    EXPECT(optcc_plan_servers(4, 2, bw, 10, 20, &pl) == OPTCC_EINVAL && !pl, "servers k = 20");
    EXPECT(optcc_plan_servers(4, 1, bw, 10, 24, &pl) == OPTCC_EINVAL && !pl, "servers g = 1");
    EXPECT(std::isnan(optcc_lower_bound(2, bw, 10)), "lower bound p = 2");
    EXPECT(std::isnan(optcc_model_time(nullptr, bw)), "model time of NULL");
    EXPECT(optcc_plan_info(nullptr, nullptr, nullptr, nullptr, nullptr) == OPTCC_EINVAL, "info NULL");
    EXPECT(optcc_last_error()[0] != 0, "an error message");
    optcc_plan_free(nullptr);
  }
  if (g_fail) {
    std::fprintf(stderr, "host_sanitize: %d failure(s)\n", g_fail);
    return 1;
  }
  std::printf("host_sanitize: ok\n");
  return 0;
}
