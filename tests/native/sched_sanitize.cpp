// Host driver for the scheduler built with AddressSanitizer and
// UndefinedBehaviorSanitizer: every entry point of sd_sched.h over random
// task sets (sizes 1 .. 48, lengths 1 .. 2048, l_max 1 .. 12, with and
// without a memory budget and separate prefill) and over invalid arguments.
// Any out-of-bounds access, leak or undefined operation aborts the run; the
// driver also checks the invariants every valid result must satisfy.
#include "sd_sched.h"

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#define REQUIRE(c)                                                    \
  do {                                                                \
    if (!(c)) {                                                       \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      std::exit(2);                                                   \
    }                                                                 \
  } while (0)

int main() {
  std::mt19937 rng(7);
  auto uni = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
  int runs = 0;
  for (int trial = 0; trial < 400; ++trial) {
    sd_sched_cfg c{};
    c.draft = {uni(1, 4), 256 * uni(1, 8), 512 * uni(1, 8)};
    c.target = {uni(4, 40), 512 * uni(2, 10), 1024 * uni(2, 14)};
    c.c1_draft = 1e-13 * uni(1, 9);
    c.c2_draft = 1e-5 * uni(0, 9);
    c.c1_verify = 1e-13 * uni(1, 9);
    c.c2_verify = 1e-4 * uni(0, 9);
    c.alpha = uni(0, 100) / 100.0;
    c.o_max = uni(1, 64);
    c.mem_budget = uni(0, 1) ? 0.0 : 1e6 * uni(1, 4000);
    c.prefill_separate = uni(0, 1);
    const int K = uni(1, 48), l_max = uni(1, 12);
    std::vector<int32_t> len(K), batch_of(K);
    for (int k = 0; k < K; ++k) len[k] = uni(1, 2048);
    std::vector<double> by_l(l_max);
    int nb = 0, lb = 0;
    double t = 0;
    const int rc = sd_sched_plan(&c, K, len.data(), l_max, batch_of.data(), &nb, &lb, &t, by_l.data());
    if (rc != 0) continue;   // e.g. no batch fits the memory budget
    ++runs;
    REQUIRE(nb >= 1 && nb <= K && lb >= 1 && lb <= l_max && std::isfinite(t) && t > 0);
    for (int k = 0; k < K; ++k) REQUIRE(batch_of[k] >= 0 && batch_of[k] < nb);
    double t2 = 0;
    REQUIRE(sd_sched_latency(&c, K, len.data(), nb, batch_of.data(), lb, &t2) == 0);
    REQUIRE(std::fabs(t2 - t) <= 1e-9 * t);
    int nb2 = 0;
    double t3 = 0;
    REQUIRE(sd_sched_batching(&c, K, len.data(), lb, batch_of.data(), &nb2, &t3) == 0);
    REQUIRE(std::fabs(t3 - t) <= 1e-9 * t);
    std::vector<double> snr(K), w(K);
    for (int k = 0; k < K; ++k) snr[k] = uni(1, 1000) / 10.0;
    double tc = 0;
    REQUIRE(sd_sched_uplink(K, len.data(), snr.data(), 16.0, 1e6 * uni(1, 100), w.data(), &tc) == 0);
    double ws = 0;
    for (int k = 0; k < K; ++k) ws += w[k];
    REQUIRE(std::fabs(ws - 1.0) < 1e-9 && tc > 0);
  }
  // invalid arguments are refused without touching the outputs
  sd_sched_cfg c{};
  c.draft = {1, 256, 512};
  c.target = {2, 512, 1024};
  c.c1_draft = c.c1_verify = 1e-12;
  c.alpha = 0.5;
  c.o_max = 8;
  int32_t len[2] = {4, 5}, bo[2] = {0, 0};
  int nb = 0, lb = 0;
  double t = 0, by_l[1];
  REQUIRE(sd_sched_plan(&c, 0, len, 1, bo, &nb, &lb, &t, by_l) != 0);
  REQUIRE(sd_sched_plan(&c, 2, nullptr, 1, bo, &nb, &lb, &t, by_l) != 0);
  REQUIRE(sd_sched_plan(&c, 2, len, 0, bo, &nb, &lb, &t, by_l) != 0);
  REQUIRE(sd_sched_latency(&c, 2, len, 0, bo, 1, &t) != 0);
  bo[1] = 3;
  REQUIRE(sd_sched_latency(&c, 2, len, 2, bo, 1, &t) != 0);
  c.alpha = 1.5;
  REQUIRE(sd_sched_batching(&c, 2, len, 1, bo, &nb, &t) != 0);
  double snr[2] = {1.0, -1.0}, w[2];
  REQUIRE(sd_sched_uplink(2, len, snr, 16.0, 1e6, w, &t) != 0);
  REQUIRE(runs > 100);
  std::printf("scheduler under sanitizers: %d plans checked\n", runs);
  return 0;
}
