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
//  label_jsd the paper's label-aware rule (Eq. 4): from the size-balanced
//            assignment, apply the single-client move with the lowest
//            J(C) = sum_n |w_n - w_bar| / |D| + sum_n (w_n / |D|) JSD(p_n, p)
//            while it lowers J, at most 4K moves.  A move keeps the source at
//            >= floor(K/C) - s and the destination at <= ceil(K/C) + s
//            members, s = max(1, K / (4C)).  JSD in nats, 0 log 0 = 0; an empty
//            cluster contributes |0 - w_bar| only.  J = S1 / |D| + S2, each sum
//            in cluster order; moves scanned client-ascending then
//            destination-ascending, first strict minimum wins.  The fp64
//            operations follow one fixed order (no contraction) so that the
//            result is reproducible bit for bit.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <numeric>
#include <vector>

#pragma clang fp contract(off)

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

// Jensen-Shannon divergence in nats: (1/2) KL(P||M) + (1/2) KL(Q||M).
double jsd(const std::vector<double> &P, const std::vector<double> &Q) {
  double a = 0.0, b = 0.0;
  for (size_t c = 0; c < P.size(); ++c) {
    const double m = 0.5 * (P[c] + Q[c]);
    if (P[c] > 0) a += P[c] * std::log(P[c] / m);
    if (Q[c] > 0) b += Q[c] * std::log(Q[c] / m);
  }
  return 0.5 * a + 0.5 * b;
}

struct Terms {
  double size_term, jsd_term;  // |w_n - w_bar| and (w_n / |D|) JSD(p_n, p)
};

Terms cluster_terms(int64_t w, const int64_t *h, const std::vector<double> &q, int64_t D, double wbar) {
  Terms t{std::fabs((double)w - wbar), 0.0};
  if (w == 0) return t;
  std::vector<double> P(q.size());
  for (size_t c = 0; c < q.size(); ++c) P[c] = (double)h[c] / (double)w;
  t.jsd_term = ((double)w / (double)D) * jsd(P, q);
  return t;
}

// Eq. 4 from per-cluster terms, with clusters a and b replaced by ta, tb.
double objective(const std::vector<Terms> &terms, int32_t a, const Terms &ta, int32_t b, const Terms &tb,
                 int64_t D) {
  double s1 = 0.0, s2 = 0.0;
  const int32_t C = (int32_t)terms.size();
  for (int32_t n = 0; n < C; ++n) s1 += (n == a ? ta : n == b ? tb : terms[n]).size_term;
  for (int32_t n = 0; n < C; ++n) s2 += (n == a ? ta : n == b ? tb : terms[n]).jsd_term;
  return s1 / (double)D + s2;
}

void label_jsd_search(int32_t K, int32_t C, const int64_t *counts, const int64_t *hist, int32_t L,
                      int32_t *out) {
  int64_t D = 0;
  std::vector<int64_t> g(L, 0);
  for (int32_t k = 0; k < K; ++k) {
    D += counts[k];
    for (int32_t c = 0; c < L; ++c) g[c] += hist[(int64_t)k * L + c];
  }
  std::vector<double> q(L);
  for (int32_t c = 0; c < L; ++c) q[c] = (double)g[c] / (double)D;
  const double wbar = (double)D / (double)C;
  const int32_t s = std::max(1, K / (4 * C));
  const int32_t lo = std::max(1, K / C - s), hi = (K + C - 1) / C + s;
  std::vector<int32_t> size(C, 0);
  std::vector<int64_t> w(C, 0), h((size_t)C * L, 0);
  for (int32_t k = 0; k < K; ++k) {
    const int32_t n = out[k];
    size[n] += 1;
    w[n] += counts[k];
    for (int32_t c = 0; c < L; ++c) h[(size_t)n * L + c] += hist[(int64_t)k * L + c];
  }
  std::vector<Terms> terms(C);
  for (int32_t n = 0; n < C; ++n) terms[n] = cluster_terms(w[n], &h[(size_t)n * L], q, D, wbar);
  double J = objective(terms, -1, terms[0], -1, terms[0], D);
  std::vector<int64_t> ha(L), hb(L);
  for (int32_t moves = 0; moves < 4 * K; ++moves) {
    bool found = false;
    double bestJ = 0.0;
    int32_t bk = -1, bb = -1;
    Terms bta{}, btb{};
    for (int32_t k = 0; k < K; ++k) {
      const int32_t a = out[k];
      if (size[a] - 1 < lo) continue;
      const int64_t *hk = hist + (int64_t)k * L;
      for (int32_t c = 0; c < L; ++c) ha[c] = h[(size_t)a * L + c] - hk[c];
      const Terms ta = cluster_terms(w[a] - counts[k], ha.data(), q, D, wbar);
      for (int32_t b = 0; b < C; ++b) {
        if (b == a || size[b] + 1 > hi) continue;
        for (int32_t c = 0; c < L; ++c) hb[c] = h[(size_t)b * L + c] + hk[c];
        const Terms tb = cluster_terms(w[b] + counts[k], hb.data(), q, D, wbar);
        const double Jn = objective(terms, a, ta, b, tb, D);
        if (!found || Jn < bestJ) {
          found = true;
          bestJ = Jn;
          bk = k;
          bb = b;
          bta = ta;
          btb = tb;
        }
      }
    }
    if (!found || !(bestJ < J)) break;
    const int32_t a = out[bk];
    const int64_t *hk = hist + (int64_t)bk * L;
    out[bk] = bb;
    size[a] -= 1;
    size[bb] += 1;
    w[a] -= counts[bk];
    w[bb] += counts[bk];
    for (int32_t c = 0; c < L; ++c) {
      h[(size_t)a * L + c] -= hk[c];
      h[(size_t)bb * L + c] += hk[c];
    }
    terms[a] = bta;
    terms[bb] = btb;
    J = bestJ;
  }
}

}  // namespace

extern "C" int gcpsl_assign(int32_t K, int32_t C, int32_t rule, uint64_t seed,
                            const int64_t *counts, const int64_t *hist, int32_t L,
                            int32_t *cluster_of_client) {
  gcpsl_clear_error();
  if (K < 1 || C < 1 || C > K) return gcpsl_fail(GCPSL_EINVAL, "assign: need 1 <= C <= K");
  if (!cluster_of_client) return gcpsl_fail(GCPSL_EINVAL, "assign: null output");
  if (rule != GCPSL_RULE_RANDOM && rule != GCPSL_RULE_SIZE && rule != GCPSL_RULE_LABEL_L1 &&
      rule != GCPSL_RULE_LABEL_JSD)
    return gcpsl_fail(GCPSL_EINVAL, "assign: unknown rule");
  if (rule != GCPSL_RULE_RANDOM) {
    if (!counts) return gcpsl_fail(GCPSL_EINVAL, "assign: counts required");
    for (int32_t k = 0; k < K; ++k)
      if (counts[k] < 0) return gcpsl_fail(GCPSL_EINVAL, "assign: negative count");
  }
  if (rule == GCPSL_RULE_LABEL_L1 || rule == GCPSL_RULE_LABEL_JSD) {
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

  if (rule == GCPSL_RULE_LABEL_JSD) {
    int64_t D = 0;
    for (int32_t k = 0; k < K; ++k) D += counts[k];
    if (D == 0) return gcpsl_fail(GCPSL_EINVAL, "assign: label_jsd needs at least one sample");
  }

  if (rule == GCPSL_RULE_SIZE || rule == GCPSL_RULE_LABEL_JSD) {
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
    if (rule == GCPSL_RULE_LABEL_JSD) label_jsd_search(K, C, counts, hist, L, cluster_of_client);
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
