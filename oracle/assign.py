"""Static client clustering (Alg. 1, Sec. IV-A).

Three rules map K clients to C fixed clusters before training:
  random      permute the clients, then deal them round-robin
              (Sec. IV-A, "Random clustering").  Reading: Durstenfeld's
              Fisher-Yates (i = K-1 .. 1, j uniform in [0, i]) on a SplitMix64
              stream started at seed + TAG_ASSIGN; client perm[i] goes to
              cluster i mod C.
  size        sort by decreasing sample count and place each client in the
              lightest allowed cluster (Sec. IV-A, "Size-balanced
              clustering").  Reading: order (count desc, id asc); a cluster is
              allowed while it holds fewer than ceil(K/C) clients; the
              lightest is the smallest summed count, ties to the lower index.
  label_l1    the greedy label-aware rule of the 16-cluster workload: clients
              in (count desc, id asc) order go to the allowed cluster whose
              label histogram after placement has the smallest L1 distance
              between its normalised histogram and the global one.  Compared
              exactly in integers (cross-multiplied); ties go to the smaller
              cluster count, then the lower index.  A client with no samples
              goes to the allowed cluster with the fewest clients (ties to the
              lower index).  The 16-cluster workload's rule; the paper's own
              label-aware rule is label_jsd.
  label_jsd   the paper's label-aware rule (Sec. IV-A, Eq. 4, Alg. 1): from a
              balanced start, repeatedly apply the single-client move that
              lowers J(C) = sum_n |w_n - w_bar| / |D| + sum_n (w_n / |D|)
              JSD(p_n, p) the most, until no allowed move lowers J or a move
              limit is reached.  Readings (the paper leaves them open): the
              start is the size-balanced assignment; a move is allowed while
              the source keeps at least floor(K/C) - s and the destination at
              most ceil(K/C) + s clients, s = max(1, K // (4C)); JSD uses the
              natural logarithm with 0 log 0 = 0; an empty cluster contributes
              |0 - w_bar| and no JSD term; the move limit is 4K; J is the sum
              S1 / |D| + S2 with S1 and S2 summed in cluster order; moves are
              scanned client-ascending, destination-ascending and the first
              strict minimum wins.
"""
from __future__ import annotations

import math

import numpy as np

from .rng import SplitMix64, TAG_ASSIGN, bounded

RULES = ("random", "size", "label_l1", "label_jsd")


def _order(counts):
    K = len(counts)
    return sorted(range(K), key=lambda k: (-int(counts[k]), k))


def assign_random(K: int, C: int, seed: int) -> np.ndarray:
    gen = SplitMix64(seed + TAG_ASSIGN)
    perm = list(range(K))
    for i in range(K - 1, 0, -1):
        j = bounded(gen, i + 1)
        perm[i], perm[j] = perm[j], perm[i]
    out = np.empty(K, dtype=np.int32)
    for i, k in enumerate(perm):
        out[k] = i % C
    return out


def assign_size(K: int, C: int, counts) -> np.ndarray:
    cap = -(-K // C)
    size = [0] * C
    load = [0] * C
    out = np.empty(K, dtype=np.int32)
    for k in _order(counts):
        best = None
        for n in range(C):
            if size[n] >= cap:
                continue
            if best is None or load[n] < load[best]:
                best = n
        out[k] = best
        size[best] += 1
        load[best] += int(counts[k])
    return out


def l1_score(hist_n, w_n, g, W):
    """Numerator of the L1 distance ||hist_n / w_n - g / W||_1 scaled by W*w_n:
    sum_c |hist_n[c] * W - w_n * g[c]|.  The distance itself is this value
    divided by W * w_n."""
    return sum(abs(int(hist_n[c]) * W - w_n * int(g[c])) for c in range(len(g)))


def assign_label_l1(K: int, C: int, counts, hist) -> np.ndarray:
    hist = np.asarray(hist, dtype=np.int64)
    L = hist.shape[1]
    g = hist.sum(axis=0)
    W = int(g.sum())
    cap = -(-K // C)
    size = [0] * C
    load = [0] * C
    H = [[0] * L for _ in range(C)]
    out = np.empty(K, dtype=np.int32)
    for k in _order(counts):
        wk = int(counts[k])
        best = None
        if wk == 0:
            for n in range(C):
                if size[n] < cap and (best is None or size[n] < size[best]):
                    best = n
        else:
            best_num = best_den = None
            for n in range(C):
                if size[n] >= cap:
                    continue
                den = load[n] + wk
                num = l1_score([H[n][c] + int(hist[k, c]) for c in range(L)], den, g, W)
                if best is None:
                    better = True
                else:
                    lhs, rhs = num * best_den, best_num * den
                    better = lhs < rhs or (lhs == rhs and load[n] < load[best])
                if better:
                    best, best_num, best_den = n, num, den
        out[k] = best
        size[best] += 1
        load[best] += wk
        for c in range(L):
            H[best][c] += int(hist[k, c])
    return out


def jsd(P, Q) -> float:
    """Jensen-Shannon divergence in nats of two distributions given as lists:
    (1/2) KL(P || M) + (1/2) KL(Q || M), M = (P + Q) / 2, with 0 log 0 = 0."""
    a = 0.0
    b = 0.0
    for c in range(len(P)):
        m = 0.5 * (P[c] + Q[c])
        if P[c] > 0:
            a += P[c] * math.log(P[c] / m)
        if Q[c] > 0:
            b += Q[c] * math.log(Q[c] / m)
    return 0.5 * a + 0.5 * b


def cluster_terms(w_n: int, h_n, q, D: int, wbar: float):
    """Cluster n's two contributions to Eq. 4: |w_n - w_bar| and
    (w_n / |D|) JSD(p_n, p), where p_n = h_n / w_n and q = p."""
    t1 = abs(float(w_n) - wbar)
    if w_n == 0:
        return t1, 0.0
    P = [float(h_n[c]) / float(w_n) for c in range(len(h_n))]
    return t1, (float(w_n) / float(D)) * jsd(P, q)


def objective(terms, D: int) -> float:
    """Eq. 4 from the per-cluster terms: S1 / |D| + S2, both summed in
    cluster order."""
    s1 = 0.0
    s2 = 0.0
    for t1, t2 in terms:
        s1 += t1
    for t1, t2 in terms:
        s2 += t2
    return s1 / float(D) + s2


def jsd_move_bounds(K: int, C: int):
    s = max(1, K // (4 * C))
    return max(1, K // C - s), -(-K // C) + s


def assign_label_jsd(K: int, C: int, counts, hist, max_moves: int = None):
    """The paper's label-aware rule; returns (cluster_of_client, moves made,
    J of the start, J of the result)."""
    counts = [int(x) for x in counts]
    hist = np.asarray(hist, dtype=np.int64)
    L = hist.shape[1]
    D = sum(counts)
    g = [int(x) for x in hist.sum(axis=0)]
    q = [float(g[c]) / float(D) for c in range(L)]
    wbar = float(D) / float(C)
    lo, hi = jsd_move_bounds(K, C)
    if max_moves is None:
        max_moves = 4 * K
    out = assign_size(K, C, counts)
    size = [0] * C
    w = [0] * C
    h = [[0] * L for _ in range(C)]
    for k in range(K):
        n = int(out[k])
        size[n] += 1
        w[n] += counts[k]
        for c in range(L):
            h[n][c] += int(hist[k, c])
    terms = [cluster_terms(w[n], h[n], q, D, wbar) for n in range(C)]
    J = objective(terms, D)
    J0 = J
    moves = 0
    while moves < max_moves:
        best = None  # (J', k, b, terms of a, terms of b)
        for k in range(K):
            a = int(out[k])
            if size[a] - 1 < lo:
                continue
            ha = [h[a][c] - int(hist[k, c]) for c in range(L)]
            ta = cluster_terms(w[a] - counts[k], ha, q, D, wbar)
            for b in range(C):
                if b == a or size[b] + 1 > hi:
                    continue
                hb = [h[b][c] + int(hist[k, c]) for c in range(L)]
                tb = cluster_terms(w[b] + counts[k], hb, q, D, wbar)
                trial = list(terms)
                trial[a] = ta
                trial[b] = tb
                Jn = objective(trial, D)
                if best is None or Jn < best[0]:
                    best = (Jn, k, b, ta, tb)
        if best is None or not best[0] < J:
            break
        Jn, k, b, ta, tb = best
        a = int(out[k])
        out[k] = b
        size[a] -= 1
        size[b] += 1
        w[a] -= counts[k]
        w[b] += counts[k]
        for c in range(L):
            h[a][c] -= int(hist[k, c])
            h[b][c] += int(hist[k, c])
        terms[a] = ta
        terms[b] = tb
        J = Jn
        moves += 1
    return out, moves, J0, J


def assign(rule: str, K: int, C: int, seed: int, counts=None, hist=None) -> np.ndarray:
    """Alg. 1: cluster_of_client int32[K] under the named rule."""
    if rule == "random":
        return assign_random(K, C, seed)
    if rule == "size":
        return assign_size(K, C, counts)
    if rule == "label_l1":
        return assign_label_l1(K, C, counts, hist)
    if rule == "label_jsd":
        return assign_label_jsd(K, C, counts, hist)[0]
    raise ValueError(rule)
