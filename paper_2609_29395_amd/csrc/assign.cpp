// Static client clustering, Alg. 1 (Sec. IV-A): host-only.
//
//  random    permute the clients, deal them round-robin.  Durstenfeld's
//            Fisher-Yates (i = K-1 .. 1, j uniform in [0, i]) on a SplitMix64
//            stream seeded with seed + TAG_ASSIGN; j by Lemire's
//            multiply-shift with rejection (2019).  perm[i] -> cluster i mod C.
//  size      clients by (count desc, id asc), each to the allowed cluster
//            (fewer than ceil(K/C) members) with the smallest summed count,
//            ties to the lower index.
//  label_l1  same order; a client with samples goes to the allowed cluster
//            minimising || (h_n + h_k)/(w_n + w_k) - g/W ||_1 after placement,
//            compared exactly as sum_c |(h_n+h_k)[c] W - (w_n+w_k) g[c]| over
//            W (w_n + w_k) by cross-multiplication; ties to the smaller w_n,
//            then the lower index.  A client without samples goes to the
//            allowed cluster with the fewest members, ties to the lower index.
#include <algorithm>
#include <cstdint>
#include <numeric>
#include <vector>

#include "../../include/gcpsl.h"
#include "rng.h"
#include "runtime.h"

namespace {

struct SplitMix64 {
  uint64_t state;
  uint64_t next() {
    state += GCPSL_GOLDEN;
    return gc_mix64(state);
  }
};

uint64_t bounded(SplitMix64 &g, uint64_t r) {
  unsigned __int128 m = (unsigned __int128)g.next() * r;
  uint64_t low = (uint64_t)m;
  if (low < r) {
    const uint64_t threshold = (0 - r) % r;
    while (low < threshold) {
      m = (unsigned __int128)g.next() * r;
      low = (uint64_t)m;
    }
  }
  return (uint64_t)(m >> 64);
}

std::vector<int32_t> client_order(int32_t K, const int64_t *counts) {
  std::vector<int32_t> order(K);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    if (counts[a] != counts[b]) return counts[a] > counts[b];
    return a < b;
  });
  return order;
}

}  // namespace

extern "C" int gcpsl_assign(int32_t K, int32_t C, int32_t rule, uint64_t seed,
                            const int64_t *counts, const int64_t *hist, int32_t L,
                            int32_t *cluster_of_client) {
  gcpsl_clear_error();
  if (K < 1 || C < 1 || C > K) return gcpsl_fail(GCPSL_EINVAL, "assign: need 1 <= C <= K");
  if (!cluster_of_client) return gcpsl_fail(GCPSL_EINVAL, "assign: null output");
  if (rule != GCPSL_RULE_RANDOM && rule != GCPSL_RULE_SIZE && rule != GCPSL_RULE_LABEL_L1)
    return gcpsl_fail(GCPSL_EINVAL, "assign: unknown rule");
  if (rule != GCPSL_RULE_RANDOM) {
    if (!counts) return gcpsl_fail(GCPSL_EINVAL, "assign: counts required");
    for (int32_t k = 0; k < K; ++k)
      if (counts[k] < 0) return gcpsl_fail(GCPSL_EINVAL, "assign: negative count");
  }
  if (rule == GCPSL_RULE_LABEL_L1) {
    if (!hist || L < 1) return gcpsl_fail(GCPSL_EINVAL, "assign: histograms required");
    for (int32_t k = 0; k < K; ++k) {
      int64_t s = 0;
      for (int32_t c = 0; c < L; ++c) {
        if (hist[(int64_t)k * L + c] < 0) return gcpsl_fail(GCPSL_EINVAL, "assign: negative histogram");
        s += hist[(int64_t)k * L + c];
      }
      if (s != counts[k]) return gcpsl_fail(GCPSL_EINVAL, "assign: histogram row != count");
    }
  }

  if (rule == GCPSL_RULE_RANDOM) {
    SplitMix64 g{seed + GCPSL_TAG_ASSIGN};
    std::vector<int32_t> perm(K);
    std::iota(perm.begin(), perm.end(), 0);
    for (int32_t i = K - 1; i >= 1; --i) {
      const int32_t j = (int32_t)bounded(g, (uint64_t)i + 1);
      std::swap(perm[i], perm[j]);
    }
    for (int32_t i = 0; i < K; ++i) cluster_of_client[perm[i]] = i % C;
    return GCPSL_OK;
  }

  const int32_t cap = (K + C - 1) / C;
  std::vector<int32_t> members(C, 0);
  std::vector<int64_t> load(C, 0);
  const std::vector<int32_t> order = client_order(K, counts);

  if (rule == GCPSL_RULE_SIZE) {
    for (int32_t k : order) {
      int32_t best = -1;
      for (int32_t n = 0; n < C; ++n) {
        if (members[n] >= cap) continue;
        if (best < 0 || load[n] < load[best]) best = n;
      }
      cluster_of_client[k] = best;
      members[best] += 1;
      load[best] += counts[k];
    }
    return GCPSL_OK;
  }

  // label_l1
  std::vector<int64_t> g(L, 0);
  for (int32_t k = 0; k < K; ++k)
    for (int32_t c = 0; c < L; ++c) g[c] += hist[(int64_t)k * L + c];
  const int64_t W = std::accumulate(g.begin(), g.end(), (int64_t)0);
  std::vector<int64_t> H((size_t)C * L, 0);
  for (int32_t k : order) {
    const int64_t wk = counts[k];
    const int64_t *hk = hist + (int64_t)k * L;
    int32_t best = -1;
    if (wk == 0) {
      for (int32_t n = 0; n < C; ++n)
        if (members[n] < cap && (best < 0 || members[n] < members[best])) best = n;
    } else {
      unsigned __int128 best_num = 0, best_den = 1;
      for (int32_t n = 0; n < C; ++n) {
        if (members[n] >= cap) continue;
        const int64_t den = load[n] + wk;
        unsigned __int128 num = 0;
        for (int32_t c = 0; c < L; ++c) {
          const __int128 v = (__int128)(H[(size_t)n * L + c] + hk[c]) * W - (__int128)den * g[c];
          num += (unsigned __int128)(v < 0 ? -v : v);
        }
        bool better;
        if (best < 0) {
          better = true;
        } else {
          const unsigned __int128 lhs = num * best_den, rhs = best_num * (unsigned __int128)den;
          better = lhs < rhs || (lhs == rhs && load[n] < load[best]);
        }
        if (better) {
          best = n;
          best_num = num;
          best_den = (unsigned __int128)den;
        }
      }
    }
    cluster_of_client[k] = best;
    members[best] += 1;
    load[best] += wk;
    for (int32_t c = 0; c < L; ++c) H[(size_t)best * L + c] += hk[c];
  }
  return GCPSL_OK;
}
