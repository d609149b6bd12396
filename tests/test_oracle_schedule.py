"""Pins for the oracle's epoch-barrier schedule (Sec. III-A; Sec. IV-D,
"Schedule and Cost", Eq. 6): each cluster takes floor(n_n / B) rounds per
system epoch, shorter clusters wait without updates, fusion closes the epoch."""
from fractions import Fraction

import numpy as np

from conftest import load_golden
from gcpsl_inputs import get_config
from oracle.sampler import batch_indices
from oracle.train import GCPSLOracle, epoch_rounds, ideal_schedule_speedup


def test_eq6_worked_example():
    g = load_golden("schedule_eq6_worked.txt")
    r, R = epoch_rounds(g["sizes"], g["B"][0])
    assert r == g["rounds"] and R == g["slots"][0]
    S, E = ideal_schedule_speedup(r)
    assert Fraction(S).limit_denominator(1000) == Fraction(g["speedup_num"][0], g["speedup_den"][0])
    assert Fraction(E).limit_denominator(1000) == Fraction(g["efficiency_num"][0], g["efficiency_den"][0])
    assert [sum(t < rn for rn in r) for t in range(R)] == g["active_per_slot"]
    # S <= N, with equality exactly when all clusters have the same length
    assert S <= len(r) and ideal_schedule_speedup([5, 5, 5])[0] == 3


def test_waiting_clusters_are_untouched_and_round_counts():
    cfg = get_config("tiny_epoch")
    o = GCPSLOracle(cfg)
    r, R = epoch_rounds(o.weights, cfg["B"])
    assert r == [6, 9] and R == 9
    taken = [0] * cfg["C"]
    for s in range(2 * R):
        t = s % R
        before = [(th.copy(), mo.copy()) for th, mo in zip(o.theta, o.mom)]
        losses = o.slot(s)
        assert sorted(losses) == [n for n in range(cfg["C"]) if t < r[n]]
        for n in range(cfg["C"]):
            if t < r[n]:
                taken[n] += 1
                assert not np.array_equal(o.mom[n], before[n][1])
            elif t != R - 1:  # waits: no update of parameters or momentum
                assert np.array_equal(o.theta[n], before[n][0]) and np.array_equal(o.mom[n], before[n][1])
            else:  # waits, then the fusion barrier: momentum stays local
                assert np.array_equal(o.mom[n], before[n][1])
            assert o.active[-1][n] == 0 or t < r[n]
        if t == R - 1:  # fused: every replica holds the same parameters
            assert all(np.array_equal(o.theta[0], th) for th in o.theta)
    assert taken == [2 * rn for rn in r]


def test_epoch_batches_cover_each_cluster_once():
    cfg = get_config("tiny_epoch")
    o = GCPSLOracle(cfg)
    r, R = epoch_rounds(o.weights, cfg["B"])
    for m in range(2):
        for n in range(cfg["C"]):
            got = np.concatenate([batch_indices(o.ids[n], cfg["B"], cfg["seed"], n, m * r[n] + t)
                                  for t in range(r[n])])
            # r_n B distinct examples of the cluster: the epoch schedules each
            # example at most once and drops fewer than B
            assert got.size == r[n] * cfg["B"] == len(np.unique(got))
            assert np.isin(got, o.ids[n]).all() and len(o.ids[n]) - got.size < cfg["B"]


def test_equal_cluster_lengths_match_lockstep_fusion_every_epoch():
    # r_n = 1 for both clusters (197 and 315 examples, B = 160): the epoch
    # schedule is the lockstep schedule fused after every round
    cfg = get_config("tiny_epoch", B=160)
    a = GCPSLOracle(cfg).run_epoch_schedule(3)
    b = GCPSLOracle(cfg).run(3, F=1)
    for n in range(cfg["C"]):
        assert np.array_equal(a.theta[n], b.theta[n]) and np.array_equal(a.mom[n], b.mom[n])
    assert a.active == b.active


def test_participation_counts_waiting_clusters_as_inactive():
    cfg = get_config("tiny_epoch")
    o = GCPSLOracle(cfg).run_epoch_schedule(9)
    r, R = epoch_rounds(o.weights, cfg["B"])
    act = np.array(o.active)
    assert act.shape == (9, 2)
    assert (act[6:, 0] == 0).all() and (act[:6, 0] > 0).all() and (act[:, 1] > 0).all()
    # Eq. 7 bound per slot: at most B clients of each running cluster
    assert (act <= cfg["B"]).all()
