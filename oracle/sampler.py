"""Cluster-local global sampling and direct data participation.

GPSL draws one fixed-size batch of B examples from the pooled data of the
workload's clients rather than concatenating per-client mini-batches
(Sec. I, Sec. II-A); an epoch ends once every example of the cluster has been
scheduled once (Sec. III-A).  Within cluster n the requested counts satisfy
sum_k b_{k,t} = B and A_{n,t} = {k in C_n : b_{k,t} > 0} (Eq. 1, Eq. 3).

Reading used for the sampling law (the paper fixes none):
  * the cluster's examples are listed in ascending global id;
  * each (cluster n, epoch e) has its own keyed permutation pi of [0, n_n);
    step t of the epoch takes positions [tB, (t+1)B), an epoch has
    S_n = floor(n_n / B) steps and the remainder is left out, so every batch
    has exactly B examples;
  * pi is a 4-round balanced Feistel network on the smallest domain 2^(2h)
    that covers n_n, with cycle walking back into [0, n_n) (Black and
    Rogaway, "Ciphers with arbitrary finite domains", 2002).  Round i maps
    (L, R) -> (R, L xor F_i(R)) with F_i(R) = mix64(key xor ((i+1) << 32 | R))
    masked to h bits; key = derive_key(seed, TAG_SAMPLE, n, e).

Direct data participation counts, per step and cluster, the clients that
supply at least one example (Sec. III-A); over a horizon of T steps the
participation is sum_t sum_n |A_{n,t}| / (K T) (Sec. V-E; clusters are
disjoint, so the union of Eq. 7 is a plain sum).

The permutation is evaluated with numpy uint64 arrays (wrap-around products
are the modulo-2^64 arithmetic the definition asks for).
"""
from __future__ import annotations

import numpy as np

from .rng import TAG_SAMPLE, derive_key

_U = np.uint64


def _mix64_np(z):
    z = z ^ (z >> _U(30))
    z = z * _U(0xBF58476D1CE4E5B9)
    z = z ^ (z >> _U(27))
    z = z * _U(0x94D049BB133111EB)
    return z ^ (z >> _U(31))


def feistel_half_bits(n: int) -> int:
    """h such that 2^(2h) is the smallest even-bit power of two >= n (h >= 1)."""
    bits = max(1, (n - 1).bit_length())
    return (bits + 1) // 2


def _feistel_pass(x, key: int, h: int):
    mask = _U((1 << h) - 1)
    left, right = x >> _U(h), x & mask
    k = _U(key)
    for i in range(4):
        f = _mix64_np(k ^ (_U((i + 1) << 32) | right)) & mask
        left, right = right, left ^ f
    return (left << _U(h)) | right


def permute(positions, n: int, key: int) -> np.ndarray:
    """pi(positions) for the keyed permutation of [0, n)."""
    pos = np.asarray(positions, dtype=np.uint64)
    if n == 1:
        return np.zeros_like(pos, dtype=np.int64)
    h = feistel_half_bits(n)
    with np.errstate(over="ignore"):
        x = _feistel_pass(pos, key, h)
        todo = x >= _U(n)
        while todo.any():
            x[todo] = _feistel_pass(x[todo], key, h)
            todo = x >= _U(n)
    return x.astype(np.int64)


def cluster_examples(client_of_example, cluster_of_client, C: int):
    """Per-cluster example lists in ascending global id."""
    owner = np.asarray(cluster_of_client)[np.asarray(client_of_example)]
    return [np.flatnonzero(owner == n).astype(np.int64) for n in range(C)]


def epoch_steps(n_n: int, B: int) -> int:
    return n_n // B


def batch_indices(ids_n, B: int, seed: int, n: int, step: int) -> np.ndarray:
    """Global example ids of cluster n's batch at (0-based) local round `step`."""
    n_n = len(ids_n)
    S = epoch_steps(n_n, B)
    if S < 1:
        raise ValueError("cluster holds fewer than B examples")
    e, t = divmod(step, S)
    key = derive_key(seed, TAG_SAMPLE, n, e)
    pos = permute(np.arange(t * B, (t + 1) * B), n_n, key)
    return ids_n[pos]


def active_clients(idx, client_of_example) -> int:
    """|A_{n,t}|: distinct clients supplying at least one example of the batch."""
    return int(np.unique(np.asarray(client_of_example)[np.asarray(idx)]).size)


def participation(active_counts, K: int) -> float:
    """Direct data participation over the horizon: active slots / (K T)."""
    a = np.asarray(active_counts, dtype=np.int64)
    return float(a.sum()) / (K * a.shape[0])
