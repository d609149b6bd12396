"""Seeded synthetic data and initial parameters.

The data stand in for CIFAR-10: N_ex images of H x W x Cin float32 in NHWC
order, L balanced classes.  Every class has one mean image with entries drawn
from N(0, 1); an example is its class mean plus independent N(0, noise_std^2)
pixel noise.  Examples are split over K clients with the per-class Dirichlet
recipe of Hsu et al. (2019): for every class, its examples are shuffled, a
share vector p ~ Dir(alpha * 1_K) is drawn, and the shuffled list is cut at
floor(cumsum(p) * n_class).

Initial parameters follow the PyTorch default bound: every weight and bias of
a layer with fan-in f is drawn from U(-1/sqrt(f), 1/sqrt(f)); normalisation
layers start at gamma = 1, beta = 0.  All replicas start from this one
vector.
"""
from __future__ import annotations

import functools

import numpy as np

from .configs import norm_layout, param_layout


@functools.lru_cache(maxsize=4)
def _dataset(N_ex, H, W, Cin, L, K, alpha, noise_std, seed):
    if N_ex % L:
        raise ValueError("N_ex must be a multiple of L (balanced classes)")
    rng = np.random.default_rng(seed)
    means = rng.standard_normal((L, H, W, Cin), dtype=np.float32)
    labels = rng.permutation(np.repeat(np.arange(L, dtype=np.int32), N_ex // L))
    images = np.empty((N_ex, H, W, Cin), dtype=np.float32)
    chunk = 4096
    for lo in range(0, N_ex, chunk):
        hi = min(N_ex, lo + chunk)
        noise = rng.standard_normal((hi - lo, H, W, Cin), dtype=np.float32)
        images[lo:hi] = means[labels[lo:hi]] + np.float32(noise_std) * noise
    client_of_example = np.empty(N_ex, dtype=np.int32)
    for c in range(L):
        ids = rng.permutation(np.flatnonzero(labels == c))
        p = rng.dirichlet(alpha * np.ones(K))
        cuts = (np.cumsum(p) * len(ids)).astype(np.int64)[:-1]
        for k, part in enumerate(np.split(ids, cuts)):
            client_of_example[part] = k
    for a in (images, labels, client_of_example):
        a.setflags(write=False)
    return images, labels, client_of_example


def make_dataset(cfg: dict):
    """(images f32[N_ex,H,W,Cin], labels i32[N_ex], client_of_example i32[N_ex])."""
    return _dataset(cfg["N_ex"], cfg["H"], cfg["W"], cfg["Cin"], cfg["L"], cfg["K"],
                    float(cfg["alpha"]), float(cfg["noise_std"]), int(cfg["seed"]))


def client_stats(cfg: dict, labels, client_of_example):
    """Per-client metadata: counts i64[K] and class histograms i64[K, L]."""
    K, L = cfg["K"], cfg["L"]
    hist = np.zeros((K, L), dtype=np.int64)
    np.add.at(hist, (client_of_example, labels), 1)
    return hist.sum(axis=1), hist


def init_params(cfg: dict) -> np.ndarray:
    """Initial flat parameter vector theta_0 (float32[P])."""
    rng = np.random.default_rng([int(cfg["seed"]), 1])
    layout = param_layout(cfg)
    total = layout[-1][3] + int(np.prod(layout[-1][2]))
    theta = np.empty(total, dtype=np.float32)
    for i, tag, shp, off in layout:
        spec = cfg["layers"][i]
        if spec[0] in ("bnorm", "gnorm") or tag.startswith("n"):  # gamma = 1, beta = 0 (PyTorch default)
            theta[off:off + int(np.prod(shp))] = 1.0 if tag[-1] == "w" else 0.0
            continue
        if spec[0] == "block":  # fan-in of the block's conv the tag names
            fan_in = {"1": 9 * spec[1], "2": 9 * spec[2], "p": spec[1]}[tag[1]]
        else:
            fan_in = 9 * spec[1] if spec[0] == "conv" else spec[1]
        bound = 1.0 / np.sqrt(fan_in)
        n = int(np.prod(shp))
        theta[off:off + n] = rng.uniform(-bound, bound, size=n).astype(np.float32)
    return theta


def init_norm_state(cfg: dict) -> np.ndarray:
    """Initial normalisation state (float32[S]): running mean 0, running
    variance 1, counter 0 for every bnorm layer (the PyTorch defaults)."""
    layout = norm_layout(cfg)
    total = 0 if not layout else layout[-1][3] + int(np.prod(layout[-1][2]))
    state = np.zeros(total, dtype=np.float32)
    for i, tag, shp, off in layout:
        if tag == "var":
            state[off:off + int(np.prod(shp))] = 1.0
    return state
