"""GCPSL training loop (Alg. 2) over the C ABI.

Builds the fixed clusters with gcpsl_assign (Alg. 1), starts all replicas
from one initial parameter vector, then for every local round samples the
cluster batches (Eq. 1, Eq. 3), runs the round for all clusters at once and
fuses the replicas every F rounds (Eq. 5).  Host orchestration only: every
computation runs in libgcpsl's kernels.
"""
from __future__ import annotations

import numpy as np

from gcpsl_inputs import client_stats, init_params, make_dataset

from . import gcpsl


def setup(cfg, max_steps=None, max_window=1, device="cuda"):
    """Inputs, Alg. 1 assignment and a Context for a workload."""
    images, labels, coe = make_dataset(cfg)
    counts, hist = client_stats(cfg, labels, coe)
    assignment = gcpsl.assign(cfg["rule"], cfg["K"], cfg["C"], cfg["seed"], counts, hist)
    ctx = gcpsl.Context(cfg, images, labels, coe, assignment, init_params(cfg),
                        max_steps=max_steps, max_window=max_window, device=device)
    return ctx, assignment


def train(ctx, steps, F=None, start=0, window=1, losses=None, stream=None):
    """Run local rounds [start, start + steps), fusing after every F-th round.

    losses: optional device tensor [steps, C] receiving each round's losses."""
    F = ctx.cfg["F"] if F is None else F
    s = start
    end = start + steps
    while s < end:
        w = min(window, end - s)
        ctx.sample(s, w, stream=stream)
        for j in range(w):
            out = None if losses is None else losses[s + j - start]
            ctx.step(s + j, out, stream=stream)
            if F and (s + j + 1) % F == 0:
                ctx.fuse(stream=stream)
        s += w
    return ctx
