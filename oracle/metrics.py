"""Batch deviation and logical application payload (Sec. V-E, "Metrics and
Execution Environment").  TEST INFRASTRUCTURE ONLY (see oracle/__init__).

Batch deviation: the l1 distance between a batch's class distribution and
the global training distribution,

    dev = sum_c | h_c / B - g_c / |D| |,

with h_c the batch's examples of class c, B the batch size, g_c the examples
of class c in the whole training set D.  Kept exact as the integer numerator
sum_c | h_c |D| - B g_c | over the denominator B |D|.

Logical application payload sums the client, server and fusion tensors that
application endpoints handle.  The paper names the three groups but not
their byte composition; the reading here (one entry per tensor handed from
one endpoint to another, in the precision the workload stores it) is:

  per local round of cluster n (Sec. III-A, Alg. 2):
    "activations"  each sampled example's cut activation, client -> server,
                   E_cut elements of the activation precision, plus its label
                   (int32: the server computes the loss);
    "cut_grads"    each example's cut gradient, server -> client, E_cut
                   elements of the activation precision;
    "client_grads" each active client's client-segment gradient to the
                   cluster's averaging point, P_c fp32 entries (Sec. III-B);
    "client_model" the averaged client segment to every client replica of
                   the cluster, P_c fp32 entries each, including replicas whose
                   owners supplied no data (Sec. IV-B);
  per fusion (Sec. IV-C, Eq. 5):
    "fusion"       every replica's parameters and server normalisation state
                   to the fusion point and the fused state back, 2 (P + S)
                   fp32 entries per replica.
A cluster waiting at the epoch barrier handles nothing in that slot.
"""
from __future__ import annotations

import numpy as np

CATEGORIES = ("activations", "cut_grads", "client_grads", "client_model", "fusion")


def class_histogram(labels, L):
    """Examples per class, as Python ints."""
    h = [0] * L
    for y in np.asarray(labels).ravel().tolist():
        h[int(y)] += 1
    return h


def batch_deviation_numerator(batch_labels, global_hist):
    """sum_c |h_c |D| - B g_c| for a batch (exact integers); the deviation is
    this over B |D|."""
    L = len(global_hist)
    h = class_histogram(batch_labels, L)
    B = sum(h)
    D = sum(int(g) for g in global_hist)
    return sum(abs(h[c] * D - B * int(global_hist[c])) for c in range(L))


def cut_elements(cfg):
    """Elements of one example's activation at the cut (the client segment's
    output)."""
    h, w, c = cfg["H"], cfg["W"], cfg["Cin"]
    for spec in cfg["layers"][:cfg["cut"]]:
        if spec[0] == "conv":
            c = spec[2]
        elif spec[0] == "block":  # 3x3 conv with pad 1 and the block's stride
            c = spec[2]
            h, w = (h - 1) // spec[3] + 1, (w - 1) // spec[3] + 1
        elif spec[0] == "maxpool":
            h, w = h // 2, w // 2
    return h * w * c


def round_payload(cfg, active, clients_in_cluster, P_client):
    """Bytes one cluster's local round hands between endpoints, by category
    (active: |A_{n,t}|; clients_in_cluster: |C_n|)."""
    e = 2 if cfg["dtype"] == "bf16" else 4
    E = cut_elements(cfg)
    B = cfg["B"]
    return {"activations": B * (E * e + 4), "cut_grads": B * E * e,
            "client_grads": int(active) * P_client * 4, "client_model": int(clients_in_cluster) * P_client * 4,
            "fusion": 0}


def fusion_payload(C, P, S):
    """Bytes of one fusion: every replica's state up, the fused state down."""
    return {"activations": 0, "cut_grads": 0, "client_grads": 0, "client_model": 0,
            "fusion": 2 * C * (P + S) * 4}
