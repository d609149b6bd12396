"""The bf16 bars for networks of residual blocks, derived on the CPU.

The GPU and the oracle round at the same points (the oracle's module
docstring lists them) but accumulate in different orders and precisions
(fp32 against fp64), so the values they round to bf16 differ by a few fp32
ulps and now and then round to neighbouring bf16 values.  Here the oracle is
run against itself with exactly that difference (gpu_match.noisy_rounding:
relative noise of 8 fp32 ulps before every bf16 rounding) under the same
ReLU and max-pool decisions, and compared the way the GPU parity tests
compare the GPU:

  * first-round gradients of the ResNet stack of ten normalised blocks move
    beyond the general bf16 bar and stay within the deep-network bar;
  * a shallow bf16 network keeps well within the general bar;
  * over rounds with a fusion, updates and momenta of the deep network are
    held to a bar calibrated per tensor by a twin run under the noise: a
    second noisy run (a stand-in for a correct GPU) passes it, and runs with
    a term of the recipe dropped (Nesterov momentum; label smoothing) fail it.
"""
import numpy as np
import pytest

from gcpsl_inputs import get_config
from gpu_match import BF16_DEEP, TOL, bar, compare_params, deep_bf16, master_ulp, noisy_rounding, twin_bar
from oracle.model import split_forward_backward
from oracle.train import GCPSLOracle


def _grads(cfg, seed):
    o = GCPSLOracle(cfg)
    _, x, y = o.batch(0, 0)
    _, g0, rec = split_forward_backward(cfg, o.theta[0], x, y, keep=True)

    def same(kind, i, own, values):
        return rec["relu_mask"][i] if kind == "relu" else rec["pool_arg"][i]

    with noisy_rounding(seed):
        _, g1, _ = split_forward_backward(cfg, o.theta[0], x, y, choose=same)
    return g0, g1


@pytest.mark.parametrize("seed", [1, 2])
def test_deep_bf16_network_self_sensitivity(seed):
    cfg = get_config("resnet_tiny_bf16")
    assert deep_bf16(cfg) and bar(cfg) == BF16_DEEP
    g0, g1 = _grads(cfg, seed)
    compare_params(g1, g0, cfg, BF16_DEEP / 1.4, "self")  # within the bar with margin
    with pytest.raises(AssertionError):
        compare_params(g1, g0, cfg, TOL["bf16"], "self")  # and beyond the general bar


def test_shallow_bf16_network_keeps_the_general_bar():
    cfg = get_config("ragged_bf16")
    assert not deep_bf16(cfg) and bar(cfg) == TOL["bf16"]
    g0, g1 = _grads(cfg, 1)
    compare_params(g1, g0, cfg, TOL["bf16"] / 2, "self")


class _Record:
    """Records one replica's decisions in call order, or replays them."""

    def __init__(self, store, key, replay=False):
        self.store, self.key, self.k, self.replay = store, key, 0, replay

    def __call__(self, kind, i, own, values):
        k = (self.key, self.k)
        self.k += 1
        if self.replay:
            return self.store[k]
        self.store[k] = own
        return own


def _run(cfg, T, store, replay, seed=None):
    o = GCPSLOracle(cfg)
    for s in range(T):
        choose = {n: _Record(store, (s, n), replay) for n in range(cfg["C"])}
        if seed is None:
            o.round(s, choose=choose)
        else:
            with noisy_rounding(seed * 1000 + s):
                o.round(s, choose=choose)
        if cfg["F"] and (s + 1) % cfg["F"] == 0:
            o.fuse()
    return o


@pytest.mark.parametrize("T", [2, 4])
def test_calibrated_bar_accepts_noise_and_catches_dropped_terms(T):
    cfg = get_config("resnet_tiny_bf16")  # fuses every 2 rounds
    store = {}
    ref = _run(cfg, T, store, replay=False)
    twin = _run(cfg, T, store, replay=True, seed=1)
    theta0 = GCPSLOracle(cfg).theta[0]
    C, tol = cfg["C"], bar(cfg)
    ulps = [master_ulp(ref.theta[n], T + T // cfg["F"]) for n in range(C)]
    tol_u = twin_bar(tol, cfg, [(twin.theta[n] - theta0, ref.theta[n] - theta0, ulps[n]) for n in range(C)])
    tol_m = twin_bar(tol, cfg, [(twin.mom[n], ref.mom[n], None) for n in range(C)])
    assert tol_u <= 0.12 and tol_m <= 0.2

    def check(o):
        for n in range(C):
            compare_params(o.theta[n] - theta0, ref.theta[n] - theta0, cfg, tol_u, ("update", n), ulp=ulps[n])
            compare_params(o.mom[n], ref.mom[n], cfg, tol_m, ("momentum", n))

    for seed in (2, 3):
        check(_run(cfg, T, store, replay=True, seed=seed))  # other runs under the noise pass
    for wrong in (dict(nesterov=False), dict(label_smoothing=0.0)):
        with pytest.raises(AssertionError):
            check(_run(dict(cfg, **wrong), T, store, replay=True, seed=2))
