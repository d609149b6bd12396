"""Pins of the oracle's label-aware move search (Sec. IV-A, Eq. 4, Alg. 1).

The objective is pinned to closed forms and to scipy's Jensen-Shannon
distance (an independent library routine); the search result is pinned by
brute force: no allowed single-client move lowers J, the cardinality bounds
hold, J never rises, and a move limit of zero returns the size-balanced start.
"""
import math

import numpy as np
import pytest
from scipy.spatial.distance import jensenshannon

from oracle.assign import (assign_label_jsd, assign_size, cluster_terms, jsd, jsd_move_bounds,
                           objective)


def test_jsd_closed_forms():
    # P = (1, 0), Q = (1/2, 1/2): M = (3/4, 1/4), KL(P||M) = log(4/3),
    # KL(Q||M) = (1/2) log(2/3) + (1/2) log 2 = (1/2) log(4/3)
    assert jsd([1.0, 0.0], [0.5, 0.5]) == pytest.approx(0.75 * math.log(4 / 3), rel=1e-15)
    assert jsd([0.2, 0.3, 0.5], [0.2, 0.3, 0.5]) == 0.0
    assert jsd([1.0, 0.0, 0.0], [0.0, 0.5, 0.5]) == pytest.approx(math.log(2), rel=1e-15)  # disjoint supports
    p, q = [0.1, 0.6, 0.3], [0.5, 0.25, 0.25]
    assert jsd(p, q) == pytest.approx(jsd(q, p), rel=1e-15)


def test_jsd_matches_scipy():
    rng = np.random.default_rng(3)
    for _ in range(50):
        L = int(rng.integers(2, 12))
        p = rng.random(L) * (rng.random(L) < 0.7)
        q = rng.random(L) + 0.01
        if p.sum() == 0:
            p[0] = 1.0
        p, q = p / p.sum(), q / q.sum()
        assert jsd(list(p), list(q)) == pytest.approx(jensenshannon(p, q) ** 2, rel=1e-10, abs=1e-15)


def objective_scipy(assign, counts, hist, C):
    """Eq. 4 written out independently (numpy + scipy)."""
    counts = np.asarray(counts, dtype=np.float64)
    hist = np.asarray(hist, dtype=np.float64)
    D = counts.sum()
    p = hist.sum(axis=0) / D
    J = 0.0
    for n in range(C):
        m = assign == n
        w = counts[m].sum()
        J += abs(w - D / C) / D
        if w > 0:
            J += (w / D) * jensenshannon(hist[m].sum(axis=0) / w, p) ** 2
    return J


def test_objective_hand_example():
    # 4 clients, 2 clusters {0,1} and {2,3}; class histograms chosen so that
    # cluster 0 is all class 0 and cluster 1 is half/half
    counts = [2, 2, 2, 2]
    hist = [[2, 0], [2, 0], [1, 1], [1, 1]]
    D, wbar = 8, 4.0
    q = [6 / 8, 2 / 8]
    terms = [cluster_terms(4, [4, 0], q, D, wbar), cluster_terms(4, [2, 2], q, D, wbar)]
    # size term 0; JSD((1,0),(3/4,1/4)) and JSD((1/2,1/2),(3/4,1/4)) by hand
    j0 = 0.5 * math.log(1 / (7 / 8)) + 0.5 * (0.75 * math.log(0.75 / (7 / 8)) + 0.25 * math.log(0.25 / (1 / 8)))
    j1 = (0.5 * (0.5 * math.log(0.5 / 0.625) + 0.5 * math.log(0.5 / 0.375))
          + 0.5 * (0.75 * math.log(0.75 / 0.625) + 0.25 * math.log(0.25 / 0.375)))
    want = 0.5 * j0 + 0.5 * j1
    assert objective(terms, D) == pytest.approx(want, rel=1e-14)
    assert objective(terms, D) == pytest.approx(objective_scipy(np.array([0, 0, 1, 1]), counts, hist, 2),
                                                rel=1e-10)


def random_instance(rng, K, L, alpha=0.3):
    counts = rng.integers(0, 40, size=K)
    hist = np.zeros((K, L), dtype=np.int64)
    for k in range(K):
        p = rng.dirichlet([alpha] * L)
        hist[k] = rng.multinomial(counts[k], p)
    return hist.sum(axis=1), hist


def allowed_moves(assign, K, C):
    lo, hi = jsd_move_bounds(K, C)
    size = np.bincount(assign, minlength=C)
    for k in range(K):
        a = assign[k]
        if size[a] - 1 < lo:
            continue
        for b in range(C):
            if b != a and size[b] + 1 <= hi:
                yield k, b


@pytest.mark.parametrize("K,C,L,seed", [(6, 2, 3, 0), (12, 3, 4, 1), (24, 4, 5, 2), (40, 5, 10, 3)])
def test_search_ends_at_local_optimum(K, C, L, seed):
    rng = np.random.default_rng(seed)
    counts, hist = random_instance(rng, K, L)
    out, moves, J0, J = assign_label_jsd(K, C, counts, hist)
    assert moves < 4 * K
    lo, hi = jsd_move_bounds(K, C)
    size = np.bincount(out, minlength=C)
    assert size.min() >= lo and size.max() <= hi and size.sum() == K
    assert J <= J0
    Jb = objective_scipy(out, counts, hist, C)
    assert J == pytest.approx(Jb, rel=1e-9)
    for k, b in allowed_moves(out, K, C):
        trial = out.copy()
        trial[k] = b
        assert objective_scipy(trial, counts, hist, C) >= Jb - 1e-12, (k, b)


def test_zero_move_limit_is_the_size_balanced_start():
    rng = np.random.default_rng(5)
    counts, hist = random_instance(rng, 20, 4)
    out, moves, J0, J = assign_label_jsd(20, 4, counts, hist, max_moves=0)
    assert moves == 0 and J == J0
    assert np.array_equal(out, assign_size(20, 4, counts))


def test_separated_labels_get_mixed():
    # clients 0-3 hold only class 0, clients 4-7 only class 1; the size-balanced
    # start pairs them by count, the search must reach clusters whose label mix
    # equals the global one (J = 0 is reachable: two of each kind per cluster)
    counts = [10, 10, 10, 10, 10, 10, 10, 10]
    hist = [[10, 0]] * 4 + [[0, 10]] * 4
    out, moves, J0, J = assign_label_jsd(8, 2, counts, hist)
    for n in range(2):
        members = [k for k in range(8) if out[k] == n]
        assert sum(1 for k in members if k < 4) == sum(1 for k in members if k >= 4)
    assert J == pytest.approx(0.0, abs=1e-15)


def test_each_move_lowers_j():
    rng = np.random.default_rng(11)
    counts, hist = random_instance(rng, 30, 6)
    prev = None
    for limit in range(0, 12):
        out, moves, J0, J = assign_label_jsd(30, 3, counts, hist, max_moves=limit)
        if prev is not None:
            assert J <= prev
            if moves == limit:
                assert J < prev or limit == 0
        prev = J
