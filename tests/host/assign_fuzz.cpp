// Randomised host check of gcpsl_assign (static client clustering, Alg. 1,
// Sec. IV-A), built with the host sanitizers by tests/test_host_sanitizers.py.
// Every rule on random client populations (empty clients, empty classes,
// C = 1 and C = K included) must return a cluster in [0, C) for every client
// and keep the cluster sizes its rule documents; invalid arguments must fail.
// The error helpers of the library's API layer are replaced by stubs so that
// the clustering source links on its own.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <string>
#include <vector>

#include "../../include/gcpsl.h"

int gcpsl_fail(int code, const std::string &) { return code; }
void gcpsl_clear_error() {}

int main(int argc, char **argv) {
  const int iters = argc > 1 ? std::atoi(argv[1]) : 200;
  const int max_k = argc > 2 ? std::atoi(argv[2]) : 120;
  std::mt19937_64 g(argc > 3 ? std::strtoull(argv[3], nullptr, 10) : 7);
  int bad = 0, calls = 0;
  for (int it = 0; it < iters; ++it) {
    const int K = 1 + (int)(g() % max_k);
    const int C = it % 7 == 0 ? K : 1 + (int)(g() % K);
    const int L = 1 + (int)(g() % 12);
    std::vector<int64_t> hist((size_t)K * L), counts(K);
    int64_t total = 0;
    for (int k = 0; k < K; ++k) {
      int64_t s = 0;
      for (int l = 0; l < L; ++l) {
        const int64_t v = g() % 4 == 0 ? 0 : (int64_t)(g() % 50);
        hist[(size_t)k * L + l] = v;
        s += v;
      }
      counts[k] = s;
      total += s;
    }
    const int cap = (K + C - 1) / C, floor_kc = K / C, slack = K / (4 * C) > 1 ? K / (4 * C) : 1;
    for (int rule = GCPSL_RULE_RANDOM; rule <= GCPSL_RULE_LABEL_JSD; ++rule) {
      std::vector<int32_t> out(K, -1);
      const int rc = gcpsl_assign(K, C, rule, g(), counts.data(), hist.data(), L, out.data());
      ++calls;
      if (rc != 0) {
        if (!(rule == GCPSL_RULE_LABEL_JSD && total == 0)) {
          std::printf("rc %d for K %d C %d L %d rule %d\n", rc, K, C, L, rule);
          ++bad;
        }
        continue;
      }
      std::vector<int> n(C, 0);
      bool range_ok = true;
      for (int k = 0; k < K; ++k) {
        if (out[k] < 0 || out[k] >= C) range_ok = false;
        else ++n[out[k]];
      }
      if (!range_ok) {
        std::printf("cluster out of range: K %d C %d rule %d\n", K, C, rule);
        ++bad;
        continue;
      }
      for (int c = 0; c < C; ++c) {
        const bool ok = rule == GCPSL_RULE_LABEL_JSD ? (n[c] >= floor_kc - slack && n[c] <= cap + slack)
                        : rule == GCPSL_RULE_RANDOM  ? (n[c] == floor_kc || n[c] == cap)
                                                       : n[c] <= cap;
        if (!ok) {
          std::printf("cluster %d holds %d clients: K %d C %d rule %d\n", c, n[c], K, C, rule);
          ++bad;
          break;
        }
      }
    }
  }
  std::vector<int32_t> o(4);
  const int64_t neg[4] = {1, 2, 3, -1}, h[4] = {1, 2, 3, 0};
  if (gcpsl_assign(4, 2, GCPSL_RULE_SIZE, 0, neg, h, 1, o.data()) == 0) ++bad;       // negative count
  if (gcpsl_assign(4, 5, GCPSL_RULE_RANDOM, 0, nullptr, nullptr, 1, o.data()) == 0) ++bad;  // C > K
  if (gcpsl_assign(4, 2, 9, 0, nullptr, nullptr, 1, o.data()) == 0) ++bad;            // unknown rule
  if (gcpsl_assign(4, 2, GCPSL_RULE_SIZE, 0, nullptr, nullptr, 1, o.data()) == 0) ++bad;  // no counts
  if (gcpsl_assign(0, 1, GCPSL_RULE_RANDOM, 0, nullptr, nullptr, 1, o.data()) == 0) ++bad;  // K < 1
  std::printf("calls %d bad %d\n", calls, bad);
  return bad != 0;
}
