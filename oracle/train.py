"""GCPSL training loop (Alg. 2), SGD update and sample-weighted fusion (Eq. 5).

Alg. 2: build the fixed clusters (Alg. 1), start every split-model replica
from the same parameters, run the clusters' GPSL rounds side by side, and at
the synchronisation points fuse client and server parameters with the weights
q_n = |D_{C_n}| / |D| and give the fused model to every replica (Sec. IV-C).
Optimiser state stays local to each cluster and is never fused (Sec. IV-C).

Readings:
  * Parameters and momentum are held as fp32 values (the workloads keep fp32
    master weights); each update is computed in fp64 and rounded once to
    fp32 when stored.
  * SGD with momentum, PyTorch convention, v starts at 0: with weight decay
    wd the step gradient is g + wd theta (L2 term, Sec. V-A); v <- mu v + g;
    theta <- theta - lr v, or with the Nesterov term (Sec. V-A)
    theta <- theta - lr (g + mu v).  wd = 0 and no Nesterov term unless the
    workload asks for them.
  * Fusion happens after every F-th round (1-based: after rounds F, 2F, ...);
    all clusters advance in lockstep.  F = 0 disables fusion.
  * Fused value: (sum_n n_n theta_n) / W accumulated in fp64 in cluster
    order and rounded once to fp32, n_n = |D_{C_n}|, W = sum_n n_n (the
    dropped epoch remainder still counts in n_n).  For fp32 replicas every
    product n_n theta_n and every partial sum is exact in fp64, so fusing
    identical replicas returns them unchanged, bit for bit.
  * The reported loss of a round is the forward loss before that round's
    update.
  * The server normalisation state (each BatchNorm layer's running mean,
    running variance and batch counter, Sec. IV-B) is updated by every round
    of its replica and fused with the same weights as the parameters
    (Sec. IV-C), in fp64 and rounded once to fp32 like them.

Epoch-barrier schedule (Sec. III-A, Sec. IV-D "Schedule and Cost", Eq. 6):
cluster n takes r_n = floor(n_n / B) local rounds per epoch (the sampler's
epoch length); the system epoch has R = max_n r_n slots.  At slot t of
system epoch m every cluster with t < r_n takes its local round m r_n + t
(epoch m, batch position t); the others wait at the fusion barrier without
updates and without participating clients.  After the last slot the
replicas are fused.  Sequential execution of the same work needs sum_n r_n
round slots, concurrent execution R: S = sum_n r_n / R <= N, E = S / N.
"""
from __future__ import annotations

import numpy as np

from gcpsl_inputs import client_stats, init_norm_state, init_params, make_dataset, norm_layout, param_counts

from .assign import assign
from .metrics import CATEGORIES, batch_deviation_numerator, class_histogram, fusion_payload, round_payload
from .model import bn_running_update, split_forward_backward
from .sampler import active_clients, batch_indices, cluster_examples


def epoch_rounds(weights, B):
    """r_n = floor(n_n / B) local rounds of each cluster per epoch, and the
    system-epoch length R = max_n r_n."""
    r = [int(w) // B for w in weights]
    return r, max(r)


def ideal_schedule_speedup(rounds):
    """Eq. 6: S = sum_n r_n / max_n r_n and E = S / N."""
    S = sum(rounds) / max(rounds)
    return S, S / len(rounds)


def sgd_update(theta, mom, grad, lr, mu, wd=0.0, nesterov=False):
    """In place on fp32 state: g <- g + wd theta; v <- mu v + g;
    theta <- theta - lr v (or theta - lr (g + mu v) with the Nesterov term).
    Computed in fp64; the momentum is rounded to fp32 when stored, and the
    stored value is the one the parameter step uses."""
    g = np.asarray(grad, dtype=np.float64) + wd * theta.astype(np.float64)
    v = mu * mom.astype(np.float64) + g
    mom[...] = v.astype(np.float32)
    step = g + mu * mom.astype(np.float64) if nesterov else mom.astype(np.float64)
    theta[...] = (theta.astype(np.float64) - lr * step).astype(np.float32)


def sgd_args(cfg):
    """The workload's SGD settings as sgd_update arguments after theta, mom, grad."""
    return (cfg["lr"], cfg["momentum"], cfg.get("weight_decay", 0.0), bool(cfg.get("nesterov", False)))


def fuse(thetas, weights):
    """Eq. 5: sum_n (n_n / W) theta_n, accumulated in fp64 in cluster order."""
    W = int(sum(int(w) for w in weights))
    acc = np.zeros(np.shape(thetas[0]), dtype=np.float64)
    for th, w in zip(thetas, weights):
        acc += float(int(w)) * np.asarray(th, dtype=np.float64)
    return (acc / W).astype(np.float32)


class GCPSLOracle:
    """State of one GCPSL run: C replicas, their momenta, the participation log."""

    def __init__(self, cfg, data=None, theta0=None, cluster_of_client=None):
        self.cfg = cfg
        self.images, self.labels, self.coe = data if data is not None else make_dataset(cfg)
        counts, hist = client_stats(cfg, self.labels, self.coe)
        if cluster_of_client is None:
            cluster_of_client = assign(cfg["rule"], cfg["K"], cfg["C"], cfg["seed"], counts, hist)
        self.assignment = np.asarray(cluster_of_client, dtype=np.int32)
        self.ids = cluster_examples(self.coe, self.assignment, cfg["C"])
        self.weights = [len(x) for x in self.ids]
        t0 = init_params(cfg) if theta0 is None else theta0
        self.theta = [np.asarray(t0, dtype=np.float32).copy() for _ in range(cfg["C"])]
        self.mom = [np.zeros_like(self.theta[0]) for _ in range(cfg["C"])]
        self.norm = [init_norm_state(cfg) for _ in range(cfg["C"])]
        self.active = []
        self.losses = []
        # Sec. V-E metrics: batch deviation numerators per round and cluster
        # (-1: no batch) over the denominator B |D|, and logical payload bytes
        self.global_hist = class_histogram(self.labels, cfg["L"])
        self.deviation = []
        self.payload = {k: 0 for k in CATEGORIES}
        self.clients_in = [int(np.sum(self.assignment == n)) for n in range(cfg["C"])]
        self.P_client = param_counts(cfg)[0]

    def _account(self, n, idx, active):
        """Sec. V-E records of cluster n's round: its batch deviation
        numerator (returned) and its payload (added)."""
        for k, v in round_payload(self.cfg, active, self.clients_in[n], self.P_client).items():
            self.payload[k] += v
        return batch_deviation_numerator(self.labels[idx], self.global_hist)

    def batch(self, step, n):
        idx = batch_indices(self.ids[n], self.cfg["B"], self.cfg["seed"], n, step)
        return idx, self.images[idx].astype(np.float64), self.labels[idx].astype(np.int64)

    def _update_norm_state(self, n, bn_batch):
        """Running statistics of replica n's BatchNorm layers after a round."""
        st = self.norm[n]
        for i, tag, shp, off in norm_layout(self.cfg):
            if tag != "mean":
                continue
            ch = shp[0]
            mean, var, count = bn_batch[i]
            rm = st[off:off + ch].astype(np.float64)
            rv = st[off + ch:off + 2 * ch].astype(np.float64)
            cnt = float(st[off + 2 * ch])
            rm, rv, cnt = bn_running_update(rm, rv, cnt, mean, var, count)
            st[off:off + ch] = rm.astype(np.float32)
            st[off + ch:off + 2 * ch] = rv.astype(np.float32)
            st[off + 2 * ch] = np.float32(cnt)

    def round(self, step, replicas=None, choose=None):
        """One local round for the given replicas (default: all).

        Returns (losses, grads) per replica; updates theta / momentum and
        records |A_{n,t}| for every cluster when all replicas ran.
        choose: optional {replica: decision callback} handed to
        split_forward_backward (the discrete decisions at near-ties)."""
        cfg = self.cfg
        reps = range(cfg["C"]) if replicas is None else replicas
        losses, grads, active, dev = {}, {}, {}, {}
        for n in reps:
            idx, x, y = self.batch(step, n)
            active[n] = active_clients(idx, self.coe)
            if replicas is None:
                dev[n] = self._account(n, idx, active[n])
            loss, g, rec = split_forward_backward(cfg, self.theta[n], x, y,
                                                  choose=None if choose is None else choose.get(n))
            sgd_update(self.theta[n], self.mom[n], g, *sgd_args(cfg))
            self._update_norm_state(n, rec["bn_batch"])
            losses[n], grads[n] = loss, g
        if replicas is None:
            self.active.append([active[n] for n in range(cfg["C"])])
            self.losses.append([losses[n] for n in range(cfg["C"])])
            self.deviation.append([dev[n] for n in range(cfg["C"])])
        return losses, grads

    def fuse(self):
        for k, v in fusion_payload(self.cfg["C"], len(self.theta[0]), len(self.norm[0])).items():
            self.payload[k] += v
        fused = fuse(self.theta, self.weights)
        for n in range(self.cfg["C"]):
            self.theta[n] = fused.copy()
        if len(self.norm[0]):
            fused_norm = fuse(self.norm, self.weights)
            for n in range(self.cfg["C"]):
                self.norm[n] = fused_norm.copy()

    def slot(self, s, choose=None):
        """Slot s of the epoch-barrier schedule; fuses after the epoch's last
        slot.  Returns {cluster: loss} of the clusters that took a round.
        choose: as for round()."""
        cfg = self.cfg
        rounds, R = epoch_rounds(self.weights, cfg["B"])
        m, t = divmod(s, R)
        losses, active, dev = {}, [], []
        for n in range(cfg["C"]):
            if t < rounds[n]:
                idx, x, y = self.batch(m * rounds[n] + t, n)
                active.append(active_clients(idx, self.coe))
                dev.append(self._account(n, idx, active[-1]))
                loss, g, rec = split_forward_backward(cfg, self.theta[n], x, y,
                                                      choose=None if choose is None else choose.get(n))
                sgd_update(self.theta[n], self.mom[n], g, *sgd_args(cfg))
                self._update_norm_state(n, rec["bn_batch"])
                losses[n] = loss
            else:
                active.append(0)  # waits at the barrier: no batch, no update
                dev.append(-1)
        self.active.append(active)
        self.deviation.append(dev)
        self.losses.append([losses.get(n, float("nan")) for n in range(cfg["C"])])
        if t == R - 1:
            self.fuse()
        return losses

    def run_epoch_schedule(self, slots):
        for s in range(slots):
            self.slot(s)
        return self

    def run(self, steps, F=None):
        F = self.cfg["F"] if F is None else F
        for s in range(steps):
            self.round(s)
            if F and (s + 1) % F == 0:
                self.fuse()
        return self
