"""Pins for the oracle's cluster-local sampler (Eq. 1-3, Eq. 7) and participation."""
import math

import numpy as np
import pytest

from oracle.rng import TAG_SAMPLE, derive_key
from oracle.sampler import (active_clients, batch_indices, cluster_examples, epoch_steps,
                            feistel_half_bits, participation, permute)


def test_half_bits_hand_values():
    # smallest even-bit power of two >= n, half width at least 1
    for n, h in [(1, 1), (2, 1), (3, 1), (4, 1), (5, 2), (16, 2), (17, 3), (64, 3),
                 (65, 4), (256, 4), (257, 5), (50000, 8), (65536, 8), (65537, 9)]:
        assert feistel_half_bits(n) == h, n


def test_permutation_is_a_bijection_brute_force():
    key = derive_key(0, TAG_SAMPLE, 3, 1)
    for n in list(range(1, 1200)) + [2047, 2048, 2049, 4095, 4096, 4097, 12544, 50000]:
        out = permute(np.arange(n), n, key)
        assert np.array_equal(np.sort(out), np.arange(n)), n


def test_permutation_depends_on_key():
    n = 1000
    a = permute(np.arange(n), n, derive_key(0, TAG_SAMPLE, 0, 0))
    b = permute(np.arange(n), n, derive_key(0, TAG_SAMPLE, 0, 1))
    c = permute(np.arange(n), n, derive_key(1, TAG_SAMPLE, 0, 0))
    assert (a != b).mean() > 0.9 and (a != c).mean() > 0.9
    # not the identity, and not a shift of it
    assert (a == np.arange(n)).mean() < 0.05


def _toy_cluster(seed=0, n_clients=20, B=32):
    rng = np.random.default_rng(seed)
    counts = rng.integers(1, 40, size=n_clients)
    coe = np.repeat(np.arange(n_clients), counts)
    coe = rng.permutation(coe).astype(np.int32)
    return coe, counts, B


def test_batch_exact_size_distinct_and_own_cluster():
    coe, counts, B = _toy_cluster()
    K = len(counts)
    cluster_of_client = np.arange(K) % 3
    ids = cluster_examples(coe, cluster_of_client, 3)
    for n in range(3):
        owned = set(ids[n].tolist())
        for step in range(12):
            idx = batch_indices(ids[n], B, 0, n, step)
            assert len(idx) == B and len(set(idx.tolist())) == B
            assert set(idx.tolist()) <= owned
            # Eq. 1 / Eq. 3: requested counts per client sum to B
            b_k = np.bincount(coe[idx], minlength=K)
            assert b_k.sum() == B
            assert (b_k[cluster_of_client != n] == 0).all()


def test_epoch_covers_each_example_once_when_divisible():
    B = 16
    ids = np.arange(1000, 1000 + 4 * B) * 3  # ascending ids, n_n = 4B
    seen = np.concatenate([batch_indices(ids, B, 7, 2, s) for s in range(4)])
    assert np.array_equal(np.sort(seen), ids)
    nxt = np.concatenate([batch_indices(ids, B, 7, 2, s) for s in range(4, 8)])
    assert np.array_equal(np.sort(nxt), ids)
    assert not np.array_equal(seen, nxt)  # a fresh permutation for epoch 1


def test_epoch_drops_remainder_without_duplicates():
    B = 10
    ids = np.arange(47)
    assert epoch_steps(47, B) == 4
    seen = np.concatenate([batch_indices(ids, B, 1, 0, s) for s in range(4)])
    assert len(set(seen.tolist())) == 40


def test_mean_active_clients_matches_hypergeometric_closed_form():
    # For a uniform B-subset of n examples, client k (n_k examples) is absent
    # with probability C(n - n_k, B) / C(n, B).
    coe, counts, B = _toy_cluster(seed=4, n_clients=30, B=24)
    ids = np.arange(len(coe))
    n = len(ids)
    expect = sum(1 - math.comb(n - int(c), B) / math.comb(n, B) for c in counts)
    obs = np.array([active_clients(batch_indices(ids, B, 11, 0, s), coe) for s in range(2500)])
    se = obs.std(ddof=1) / math.sqrt(len(obs))
    assert abs(obs.mean() - expect) < 4 * se + 1e-9, (obs.mean(), expect, se)


def test_idle_bounds_eq2_eq3_eq7():
    coe, counts, B = _toy_cluster(seed=5, n_clients=24, B=8)
    K, C = len(counts), 3
    cl = np.arange(K) % C
    ids = cluster_examples(coe, cl, C)
    for step in range(30):
        total = 0
        for n in range(C):
            a = active_clients(batch_indices(ids[n], B, 0, n, step), coe)
            size = int((cl == n).sum())
            assert 1 - a / size >= max(0.0, 1 - B / size) - 1e-12  # Eq. 3
            assert a <= min(B, size)
            total += a
        assert 1 - total / K >= max(0.0, 1 - C * B / K) - 1e-12  # Eq. 7


def test_active_clients_and_participation_brute_force():
    coe = np.array([0, 0, 1, 2, 2, 2, 3], dtype=np.int32)
    assert active_clients([0, 1], coe) == 1
    assert active_clients([0, 3, 4], coe) == 2      # clients 0, 2, 2
    assert active_clients([1, 2, 5, 6], coe) == 4   # clients 0, 1, 2, 3
    assert active_clients([3, 4, 5, 6], coe) == 2   # clients 2, 2, 2, 3
    # two steps, two clusters, K = 4: (1 + 2 + 2 + 1) / (4 * 2)
    assert participation([[1, 2], [2, 1]], 4) == pytest.approx(6 / 8)


def test_cluster_examples_ascending_and_partition():
    coe = np.array([2, 0, 1, 2, 1, 0, 3], dtype=np.int32)
    ids = cluster_examples(coe, np.array([0, 1, 0, 1]), 2)
    # owners: ex0 c2->0, ex1 c0->0, ex2 c1->1, ex3 c2->0, ex4 c1->1, ex5 c0->0, ex6 c3->1
    assert ids[0].tolist() == [0, 1, 3, 5] and ids[1].tolist() == [2, 4, 6]
