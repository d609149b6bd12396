"""Pins for the oracle's integer streams and for static clustering (Alg. 1)."""
from fractions import Fraction

import numpy as np
import pytest

from oracle.assign import assign, assign_label_l1, assign_random, assign_size
from oracle.rng import MASK64, TAG_ASSIGN, SplitMix64, bounded, mix64

from conftest import load_golden

# SplitMix64 known-answer vector from the generator's published reference
# implementation (state seeded with 1234567), stored in tests/golden.
_G = load_golden("splitmix64_seed1234567.txt")
assert _G["seed"] == [1234567]
SPLITMIX_1234567 = _G["outputs"]


def test_splitmix64_published_vector():
    g = SplitMix64(1234567)
    assert [g.next() for _ in range(5)] == SPLITMIX_1234567


def test_mix64_zero_fixed_point_and_bijective_sample():
    assert mix64(0) == 0
    xs = [mix64(i) for i in range(1, 5000)]
    assert len(set(xs)) == len(xs)


def test_bounded_power_of_two_is_top_bits():
    # For r = 2^k, 2^64 mod r = 0: nothing is rejected and the draw is the
    # top k bits of the stream output.
    for k in (1, 3, 17, 63):
        g1, g2 = SplitMix64(1234567), SplitMix64(1234567)
        for _ in range(5):
            assert bounded(g1, 1 << k) == g2.next() >> (64 - k)


def test_bounded_hand_traced():
    # r = 3 on the first published output: 6457827717110365317 * 3 =
    # 1 * 2^64 + 926739077621544335, low word >= 3 so no rejection -> 1.
    assert bounded(SplitMix64(1234567), 3) == 1
    # r = 1 always yields 0.
    g = SplitMix64(5)
    assert all(bounded(g, 1) == 0 for _ in range(10))


def test_bounded_range_and_rough_uniformity():
    g = SplitMix64(99)
    draws = [bounded(g, 7) for _ in range(7000)]
    counts = np.bincount(draws, minlength=7)
    assert counts.min() > 850 and counts.max() < 1150


def test_random_assignment_hand_traced():
    # Seed chosen so the assignment stream is the published SplitMix64 stream.
    seed = (1234567 - TAG_ASSIGN) & MASK64
    # K=2: j = bounded(2) = top bit of 6457827717110365317 = 0 -> swap -> perm
    # [1, 0]; client 1 -> cluster 0, client 0 -> cluster 1.
    assert assign_random(2, 2, seed).tolist() == [1, 0]
    # K=3: i=2: j = 1 (traced above) -> perm [0, 2, 1]; i=1: j = top bit of
    # 3203168211198807973 = 0 -> perm [2, 0, 1]; round-robin over C=2 gives
    # client 2 -> 0, client 0 -> 1, client 1 -> 0.
    assert assign_random(3, 2, seed).tolist() == [1, 0, 0]


@pytest.mark.parametrize("K,C", [(16, 2), (256, 4), (256, 16), (10, 3), (7, 7)])
def test_random_assignment_is_round_robin_of_a_permutation(K, C):
    a = assign_random(K, C, 0)
    sizes = np.bincount(a, minlength=C)
    assert sizes.sum() == K
    assert sizes.max() - sizes.min() <= 1
    assert (sizes[: K % C] == K // C + 1).all() if K % C else (sizes == K // C).all()
    assert np.array_equal(a, assign_random(K, C, 0))
    assert not np.array_equal(assign_random(256, 4, 0), assign_random(256, 4, 1))


def test_size_balanced_hand_built():
    # counts [5, 3, 3, 1], C=2, cap 2.  Order 0,1,2,3.  0 -> c0 (tie, lower
    # index); 1 -> c1 (0 < 5); 2 -> c1 (3 < 5), c1 now full; 3 -> c0.
    assert assign_size(4, 2, [5, 3, 3, 1]).tolist() == [0, 1, 1, 0]
    # Ties in count are broken by client id: clients 1 and 2 both have 4.
    # Order 0(6), 1(4), 2(4), 3(2), 4(1), cap ceil(5/2)=3.
    # 0 -> c0; 1 -> c1; 2 -> c1 (4 < 6); 3 -> c0 (6 < 8); 4 -> c0 (8 = 8,
    # lower index) and c0 reaches the cap of 3.
    assert assign_size(5, 2, [6, 4, 4, 2, 1]).tolist() == [0, 1, 1, 0, 0]


def test_size_balanced_cap_forces_placement():
    # One huge client and three small ones, C=2, cap 2: after 0 -> c0 and
    # 1 -> c1, 2 -> c1 (lighter); c1 is full so 3 must go to c0.
    assert assign_size(4, 2, [100, 1, 1, 1]).tolist() == [0, 1, 1, 0]


def test_label_l1_hand_built():
    # Two classes, global histogram g = [4, 4] (W = 8).  Clients (counts):
    # 0: [3,0] (3), 1: [0,3] (3), 2: [1,0] (1), 3: [0,1] (1).  C=2, cap 2.
    # 0 -> c0 (all empty: tie -> lower index).
    # 1: c0 after = [3,3] -> distance 0; c1 after = [0,3] -> distance 1. -> c0.
    # c0 is full; 2 -> c1, 3 -> c1.
    hist = np.array([[3, 0], [0, 3], [1, 0], [0, 1]])
    assert assign_label_l1(4, 2, hist.sum(1), hist).tolist() == [0, 0, 1, 1]
    # Zero-sample clients go to the allowed cluster with the fewest clients.
    hist = np.array([[2, 2], [0, 0], [1, 1], [0, 0]])
    # order: 0(4), 2(2), 1(0), 3(0).  0 -> c0; 2: c0 after [3,3] d=0, c1
    # after [1,1] d=0, tie -> smaller count (c1 has 0) -> c1.  1 (empty) ->
    # fewest clients: both 1 -> c0.  3 -> c1 (c0 full).
    assert assign_label_l1(4, 2, hist.sum(1), hist).tolist() == [0, 0, 1, 1]


def _l1(hn, wn, g, W):
    return sum(abs(Fraction(int(hn[c]), wn) - Fraction(int(g[c]), W)) for c in range(len(g)))


def test_label_l1_each_choice_is_the_exact_rational_argmin():
    rng = np.random.default_rng(3)
    K, C, L = 40, 5, 6
    hist = rng.integers(0, 9, size=(K, L)) * (rng.random((K, L)) < 0.4)
    counts = hist.sum(1)
    a = assign_label_l1(K, C, counts, hist)
    g, W, cap = hist.sum(0), int(hist.sum()), -(-K // C)
    H = np.zeros((C, L), dtype=np.int64)
    size = np.zeros(C, dtype=np.int64)
    for k in sorted(range(K), key=lambda k: (-int(counts[k]), k)):
        allowed = [n for n in range(C) if size[n] < cap]
        if counts[k] == 0:
            want = min(allowed, key=lambda n: (size[n], n))
        else:
            want = min(allowed, key=lambda n: (_l1(H[n] + hist[k], int(H[n].sum() + counts[k]), g, W),
                                               int(H[n].sum()), n))
        assert a[k] == want
        H[want] += hist[k]
        size[want] += 1


@pytest.mark.parametrize("rule", ["random", "size", "label_l1"])
def test_every_client_once_and_cap(rule):
    rng = np.random.default_rng(0)
    K, C, L = 37, 6, 5
    hist = rng.integers(0, 20, size=(K, L))
    a = assign(rule, K, C, 0, hist.sum(1), hist)
    assert a.shape == (K,) and a.min() >= 0 and a.max() < C
    assert np.bincount(a, minlength=C).max() <= -(-K // C)
