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
              lower index).  This replaces the paper's move search on Eq. 4,
              which is a different rule.
"""
from __future__ import annotations

import numpy as np

from .rng import SplitMix64, TAG_ASSIGN, bounded

RULES = ("random", "size", "label_l1")


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


def assign(rule: str, K: int, C: int, seed: int, counts=None, hist=None) -> np.ndarray:
    """Alg. 1: cluster_of_client int32[K] under the named rule."""
    if rule == "random":
        return assign_random(K, C, seed)
    if rule == "size":
        return assign_size(K, C, counts)
    if rule == "label_l1":
        return assign_label_l1(K, C, counts, hist)
    raise ValueError(rule)
