"""GCPSL training loop (Alg. 2) over the C ABI.

Builds the fixed clusters with gcpsl_assign (Alg. 1), starts all replicas
from one initial parameter vector, then for every local round samples the
cluster batches (Eq. 1, Eq. 3), runs the round for all clusters at once and
fuses the replicas every F rounds (Eq. 5).  Host orchestration only: every
computation runs in libgcpsl's kernels.
"""
from __future__ import annotations

import numpy as np

from gcpsl_inputs import client_stats, init_norm_state, init_params, make_dataset

from . import gcpsl


def setup(cfg, max_steps=None, max_window=1, device="cuda", schedule=None, static=False):
    """Inputs, Alg. 1 assignment and a Context for a workload (schedule:
    the workload's own unless given; static: gcpsl_create_static)."""
    schedule = cfg.get("schedule", "lockstep") if schedule is None else schedule
    images, labels, coe = make_dataset(cfg)
    counts, hist = client_stats(cfg, labels, coe)
    assignment = gcpsl.assign(cfg["rule"], cfg["K"], cfg["C"], cfg["seed"], counts, hist)
    ctx = gcpsl.Context(cfg, images, labels, coe, assignment, init_params(cfg),
                        max_steps=max_steps, max_window=max_window, device=device, schedule=schedule,
                        norm_state0=init_norm_state(cfg), static=static)
    return ctx, assignment


def _round(ctx, step, out, serial, stream):
    """One step: all its clusters in one launch per kernel, or (serial) one
    cluster after another."""
    if not serial:
        ctx.step(step, out, stream=stream)
        return
    rounds, R = ctx.epoch_rounds()
    t = step % R if ctx.schedule == "epoch" else 0
    for n in range(ctx.cfg["C"]):
        if ctx.schedule != "epoch" or t < rounds[n]:
            ctx.step_replica(step, n, out, stream=stream)


def train(ctx, steps, F=None, start=0, window=1, losses=None, stream=None, serial=False):
    """Run steps [start, start + steps).  Lockstep schedule: every cluster
    takes a round per step and the replicas are fused after every F-th step.
    Epoch schedule (Alg. 2 with the fusion barrier of Sec. III-A): a step is
    a slot of the system epoch and the replicas are fused after the last slot
    of every epoch.  serial: run the clusters of a step one after another.

    losses: optional device tensor [steps, C] receiving each step's losses."""
    if ctx.schedule == "epoch":
        F = ctx.epoch_rounds()[1]
    else:
        F = ctx.cfg["F"] if F is None else F
    s = start
    end = start + steps
    while s < end:
        w = min(window, end - s)
        ctx.sample(s, w, stream=stream)
        for j in range(w):
            out = None if losses is None else losses[s + j - start]
            _round(ctx, s + j, out, serial, stream)
            if F and (s + j + 1) % F == 0:
                ctx.fuse(stream=stream)
        s += w
    return ctx
