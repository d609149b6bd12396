"""Pins of the Sec. V-E metrics in the oracle: batch deviation (exact rational
brute force, closed forms, bounds) and logical payload (message-by-message
enumeration of a run against the oracle's per-category totals)."""
from fractions import Fraction

import numpy as np
import pytest

from gcpsl_inputs import get_config, norm_layout, param_layout
from oracle.metrics import batch_deviation_numerator, class_histogram
from oracle.model import split_forward_backward
from oracle.sampler import batch_indices
from oracle.train import GCPSLOracle


def test_batch_deviation_equals_the_l1_distance_of_distributions():
    # brute force in exact rationals: sum_c |h_c / B - g_c / |D||
    rng = np.random.default_rng(3)
    for _ in range(200):
        L = int(rng.integers(2, 12))
        g = rng.integers(0, 50, size=L)
        g[rng.integers(0, L)] += 1
        B = int(rng.integers(1, 40))
        labels = rng.integers(0, L, size=B)
        D = int(g.sum())
        want = sum(abs(Fraction(int(np.sum(labels == c)), B) - Fraction(int(g[c]), D)) for c in range(L))
        num = batch_deviation_numerator(labels, g.tolist())
        assert Fraction(num, B * D) == want
        assert 0 <= num <= 2 * B * D  # an l1 distance of two distributions lies in [0, 2]


def test_batch_deviation_closed_forms():
    g = [30, 10, 20, 40]  # |D| = 100
    # a batch with the global proportions has deviation 0
    assert batch_deviation_numerator([0, 0, 0, 1, 2, 2, 3, 3, 3, 3], g) == 0
    # a batch of one class c: (1 - p_c) + sum_{c' != c} p_c' = 2 (1 - p_c)
    for c in range(4):
        num = batch_deviation_numerator([c] * 7, g)
        assert Fraction(num, 7 * 100) == 2 * (1 - Fraction(g[c], 100))
    # a class absent from the data set and present in the batch counts fully
    assert Fraction(batch_deviation_numerator([1, 1], [5, 0, 5]), 2 * 10) == 2


def test_class_histogram():
    assert class_histogram(np.array([2, 0, 2, 2]), 4) == [1, 0, 3, 0]


def _enumerate_messages(o, cfg, T, fused_after, schedule_rounds=None):
    """Every tensor handed between endpoints in T steps, one entry at a time:
    (category, bytes)."""
    e = 2 if cfg["dtype"] == "bf16" else 4
    C = cfg["C"]
    # the cut activation's size from the model itself
    idx = batch_indices(o.ids[0], cfg["B"], cfg["seed"], 0, 0)
    _, _, rec = split_forward_backward(cfg, o.theta[0], o.images[idx].astype(np.float64),
                                       o.labels[idx].astype(np.int64), keep=True)
    cut_elems = int(np.prod(rec["acts"][cfg["cut"]].shape[1:]))
    pc = sum(int(np.prod(shp)) for li, _, shp, _ in param_layout(cfg) if li < cfg["cut"])
    P = sum(int(np.prod(shp)) for _, _, shp, _ in param_layout(cfg))
    S = sum(int(shp[0]) for _, _, shp, _ in norm_layout(cfg))
    msgs = []
    for s in range(T):
        for n in range(C):
            if schedule_rounds is None:
                local = s
            else:
                rounds, R = schedule_rounds
                m, t = divmod(s, R)
                if t >= rounds[n]:
                    continue  # waits at the barrier
                local = m * rounds[n] + t
            batch = batch_indices(o.ids[n], cfg["B"], cfg["seed"], n, local)
            for ex in batch:
                msgs.append(("activations", cut_elems * e))  # client -> server
                msgs.append(("activations", 4))              # its label
                msgs.append(("cut_grads", cut_elems * e))    # server -> client
            for k in sorted({int(o.coe[ex]) for ex in batch}):
                msgs.append(("client_grads", pc * 4))        # active client -> averaging
            for k in range(cfg["K"]):
                if o.assignment[k] == n:
                    msgs.append(("client_model", pc * 4))    # average -> every replica
        if s in fused_after:
            for n in range(C):
                msgs.append(("fusion", (P + S) * 4))         # replica -> fusion
                msgs.append(("fusion", (P + S) * 4))         # fused -> replica
    out = {}
    for k, b in msgs:
        out[k] = out.get(k, 0) + b
    return out


@pytest.mark.parametrize("name", ["tiny", "ragged_bf16", "tiny_norm", "resnet_tiny"])
def test_payload_counts_every_message(name):
    cfg = get_config(name)
    T = 5
    o = GCPSLOracle(cfg).run(T)
    fused = {s for s in range(T) if cfg["F"] and (s + 1) % cfg["F"] == 0}
    want = _enumerate_messages(GCPSLOracle(cfg), cfg, T, fused)
    assert {k: v for k, v in o.payload.items() if v} == want
    # and the deviation of every batch against its own labels
    g = class_histogram(o.labels, cfg["L"])
    D = sum(g)
    for s in range(T):
        for n in range(cfg["C"]):
            idx = batch_indices(o.ids[n], cfg["B"], cfg["seed"], n, s)
            h = [int(np.sum(o.labels[idx] == c)) for c in range(cfg["L"])]
            assert o.deviation[s][n] == sum(abs(h[c] * D - cfg["B"] * g[c]) for c in range(cfg["L"]))


def test_payload_epoch_schedule_counts_only_rounds_taken():
    cfg = get_config("tiny_epoch")
    o = GCPSLOracle(cfg)
    from oracle.train import epoch_rounds
    rounds, R = epoch_rounds(o.weights, cfg["B"])
    T = R + 3
    o.run_epoch_schedule(T)
    want = _enumerate_messages(GCPSLOracle(cfg), cfg, T, {R - 1}, schedule_rounds=(rounds, R))
    assert {k: v for k, v in o.payload.items() if v} == want
    for s in range(T):
        for n in range(cfg["C"]):
            assert (o.deviation[s][n] == -1) == (s % R >= rounds[n])
