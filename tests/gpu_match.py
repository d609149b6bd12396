"""Helpers of the GPU parity tests: tolerances, the per-tensor comparison and
the matching of discrete decisions.

A training round takes two kinds of discrete decisions: whether a ReLU
passes a value (R18: mask = output > 0) and which pixel of a 2 x 2 window
the max pool takes (the first maximum in row-major order).  The GPU computes
in fp32 (and rounds to bf16 at the workload's rounding points), the oracle in
fp64, so where a pre-activation is within rounding of zero, or two window
values are within rounding of each other, the two can decide differently.
Both decisions are correct results at the working precision, and each one
changes its gradient entry completely, which the tensor comparison would
then report as a kernel error.

`GpuChoices` reads the decisions the GPU took from its stored activations
(the mask is act > 0, the routing the first maximum of the stored window,
exactly as the GPU's backward kernels take them), checks every one that
differs from the oracle's own decision to be such a near-tie of the
oracle's values (an assertion otherwise), and hands the GPU's decision to
the oracle through `split_forward_backward(choose=...)`.  The oracle then
computes every value itself under the same decisions, and all tensors are
held to the workload's bar with no exemption.  Nothing else of the GPU's
output enters the oracle.
"""
from __future__ import annotations

import numpy as np
import torch

TOL = {"f32": 1e-4, "bf16": 2e-2}

# Near-tie bounds, relative to the tensor's largest magnitude (ReLU: the
# pre-activation is within this of zero) or (relative to the window maximum,
# relative to the tensor's largest magnitude) for a max-pool window.  fp32:
# a few ulps (2^-23) of accumulation-order difference against fp64.  bf16:
# one ulp is 2^-8 = 3.9e-3 relative, and one-ulp differences upstream move the
# values of deeper layers by several ulps of their scale; the bound is the
# per-element bar of the tensor comparison itself (tol of the largest
# magnitude), so a decision counts as a near-tie exactly when the two
# candidates are within what the activation comparison accepts.
KINK = {"f32": 1e-5, "bf16": 2e-2}
TIE = {"f32": (1e-5, 1e-6), "bf16": (2e-2, 2e-2)}


def close(a, b, tol):
    """||a - b||_2 <= tol ||b||_2 and max|a - b| <= tol max|b|."""
    a = np.asarray(a, dtype=np.float64).ravel()
    b = np.asarray(b, dtype=np.float64).ravel()
    assert a.shape == b.shape, (a.shape, b.shape)
    nb = np.linalg.norm(b)
    err = np.linalg.norm(a - b)
    mx = np.abs(b).max() if b.size else 0.0
    ok = err <= tol * nb + 1e-30 and np.abs(a - b).max() <= tol * mx + 1e-30
    return ok, (err / (nb + 1e-30), np.abs(a - b).max() / (mx + 1e-30))


def to_np(t):
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy()


def pool_windows(x):
    """[Bt,H,W,C] -> [Bt,H/2,W/2,4,C], window positions in row-major order."""
    Bt, H, W, C = x.shape
    return (x.reshape(Bt, H // 2, 2, W // 2, 2, C).transpose(0, 1, 3, 2, 4, 5)
            .reshape(Bt, H // 2, W // 2, 4, C))


def layer_shapes(cfg):
    """Output shape [B, ...] of every layer of the workload's model."""
    h, w, c = cfg["H"], cfg["W"], cfg["Cin"]
    out = []
    for spec in cfg["layers"]:
        kind = spec[0]
        if kind == "conv":
            c = spec[2]
        elif kind == "maxpool":
            h, w = h // 2, w // 2
        elif kind == "avgpool":
            h = w = None
        elif kind == "linear":
            c = spec[2]
        out.append((cfg["B"], h, w, c) if h is not None else (cfg["B"], c))
    return out


def replica_tensor(ctx, name, n, shape):
    """Replica n's slice of workspace tensor `name` (None if not stored)."""
    from paper_2609_29395_amd import gcpsl
    try:
        t = ctx.tensor(name)
    except gcpsl.GCPSLError:
        return None
    per = int(np.prod(shape))
    return to_np(t.reshape(-1)[n * per:(n + 1) * per]).reshape(shape)


class GpuChoices:
    """The GPU's ReLU and max-pool decisions of one replica's last round,
    validated against the oracle's values as they are taken (see module
    docstring).  flips[(kind, layer)] counts the decisions that differed."""

    def __init__(self, ctx, cfg, n):
        self.kink = KINK[cfg["dtype"]]
        self.tie = TIE[cfg["dtype"]]
        shapes = layer_shapes(cfg)
        layers = cfg["layers"]
        self.relu, self.pool, self.flips = {}, {}, {}
        self.worst = 0.0  # largest near-tie distance seen, as a fraction of its tensor's scale
        for i, spec in enumerate(layers):
            kind = spec[0]
            normed = i + 1 < len(layers) and layers[i + 1][0] in ("bnorm", "gnorm")
            if (kind == "conv" and not normed) or kind in ("bnorm", "gnorm"):
                a = replica_tensor(ctx, f"act{i}", n, shapes[i])
                if a is not None:
                    self.relu[i] = a > 0
                    if i + 1 < len(layers) and layers[i + 1][0] == "maxpool":
                        self.pool[i + 1] = np.argmax(pool_windows(a), axis=3)

    def __call__(self, kind, i, own, values):
        if kind == "relu":
            gpu = self.relu.get(i)
            assert gpu is not None, f"layer {i}: the GPU's activation is not stored"
            assert gpu.shape == own.shape, (i, gpu.shape, own.shape)
            diff = gpu != own
            if diff.any():
                scale = np.abs(values).max()
                self.worst = max(self.worst, np.abs(values[diff]).max() / scale)
                far = np.abs(values[diff]) > self.kink * scale
                assert not far.any(), ("ReLU decision differs away from a kink", i, int(far.sum()),
                                       values[diff][far][:4], scale)
        else:
            gpu = self.pool.get(i)
            assert gpu is not None, f"layer {i}: the GPU's pool input is not stored"
            assert gpu.shape == own.shape, (i, gpu.shape, own.shape)
            diff = gpu != own
            if diff.any():
                rel, absolute = self.tie
                top = np.take_along_axis(values, own[:, :, :, None, :], axis=3)[:, :, :, 0, :]
                got = np.take_along_axis(values, gpu[:, :, :, None, :], axis=3)[:, :, :, 0, :]
                gap = (top - got)[diff]
                bound = rel * np.abs(top[diff]) + absolute * np.abs(values).max()
                self.worst = max(self.worst, gap.max() / np.abs(values).max())
                far = gap > bound
                assert not far.any(), ("max-pool routing differs away from a tie", i, int(far.sum()),
                                       gap[far][:4], bound[far][:4])
        self.flips[(kind, i)] = int(diff.sum())
        return gpu


class LazyChoices(dict):
    """{replica: GpuChoices} built on first use, for GCPSLOracle.round."""

    def __init__(self, ctx, cfg, reps=None):
        super().__init__()
        self.ctx, self.cfg = ctx, cfg
        self.reps = set(range(cfg["C"])) if reps is None else set(reps)

    def get(self, n, default=None):
        if n not in self.reps:
            return default
        if n not in self:
            self[n] = GpuChoices(self.ctx, self.cfg, n)
        return self[n]


def vanishing_biases(cfg):
    """Layers whose bias has an exactly zero loss gradient in exact
    arithmetic: a conv followed by batch norm (the batch mean subtracts any
    per-channel constant).  Both sides then hold rounding noise of their own
    precision in its gradient, momentum and update."""
    layers = cfg["layers"]
    return {i for i, sp in enumerate(layers)
            if sp[0] == "conv" and i + 1 < len(layers) and layers[i + 1][0] == "bnorm"}


def master_ulp(theta):
    """Spacing of the fp32 masters at theta: two updates of the same master
    that round differently differ by at least this much."""
    return np.spacing(np.abs(np.asarray(theta, dtype=np.float32))).astype(np.float64)


def compare_params(got, want, cfg, tol, what, ulp=None):
    """Every layer's weight and bias of a flat parameter-shaped vector on its
    own, so an error in one layer cannot hide behind another's magnitude.  A
    bias whose gradient vanishes exactly (vanishing_biases) is compared
    elementwise on the scale of its layer's weight: max|a - b| <= tol
    max|weight entries of b|.  ulp (for differences of fp32 masters, e.g. an
    update theta_T - theta_0): per-element resolution of the stored values,
    allowed on top of the max-element bound (a gradient that differs in its
    last bits can round a master to the neighbouring fp32 value)."""
    from gcpsl_inputs import param_layout
    zero = vanishing_biases(cfg)
    wmax = {}
    for li, tag, shp, off in param_layout(cfg):
        size = int(np.prod(shp))
        a = np.asarray(got[off:off + size], dtype=np.float64)
        b = np.asarray(want[off:off + size], dtype=np.float64)
        res = 0.0 if ulp is None else ulp[off:off + size]
        if tag == "w":
            wmax[li] = np.abs(b).max()
        if tag == "b" and li in zero:
            err = (np.abs(a - b) - res).max()
            assert err <= tol * wmax[li], (what, li, tag, "vanishing", err, wmax[li])
            continue
        nb = np.linalg.norm(b)
        err = np.linalg.norm(a - b)
        worst = (np.abs(a - b) - res).max()
        ok = err <= tol * nb + 1e-30 and worst <= tol * np.abs(b).max() + 1e-30
        assert ok, (what, li, tag, err / (nb + 1e-30), worst / (np.abs(b).max() + 1e-30))
