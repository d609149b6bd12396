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
exactly as the GPU's backward kernels take them), or, for a conv whose
max pool keeps routing codes instead of the unpooled output, from the codes
(the routed position of each window, or none; the ReLU decisions at a
window's other positions change nothing and stay the oracle's), checks every one that
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
# relative to the tensor's largest magnitude) for a max-pool window: the
# per-element bar of the tensor comparison itself (tol of the largest
# magnitude), so a decision counts as a near-tie exactly when the two
# candidates are within what the activation comparison accepts.  (fp32
# differences start at a few ulps, 2^-23, of accumulation order against fp64;
# bf16 ones at one ulp, 2^-8; normalisations over few values and deeper layers
# enlarge both.)
KINK = {"f32": 1e-4, "bf16": 2e-2}
TIE = {"f32": (1e-4, 1e-4), "bf16": (2e-2, 2e-2)}

# bf16 networks of residual blocks (ten normalised 3x3 convs and more between
# input and loss) sit at the edge of the bf16 bar on their own: noise of the
# size of fp32 accumulation order before each bf16 rounding moves the oracle's
# own first-round gradients by up to 3.5 % of a tensor's largest entry
# (test_parity_bar pins this), so the GPU, which differs from the oracle by
# exactly such noise, is held to 5e-2 there, for tensors and near-ties alike.
# Over several rounds the per-tensor updates and momenta of such a network
# drift further apart under that noise alone (up to 5e-2 and 9e-2 after two
# to four rounds), so those comparisons take a bar calibrated by a twin
# oracle run under the noise (noisy_rounding, twin_bar).
BF16_DEEP = 5e-2

# relative standard deviation of the calibration noise: 8 fp32 ulps
NOISE_REL = 8 * 2.0 ** -24


def deep_bf16(cfg):
    return cfg["dtype"] == "bf16" and any(spec[0] == "block" for spec in cfg["layers"])


def bar(cfg):
    """The workload's comparison bar (TOL, KINK and TIE in one figure)."""
    return BF16_DEEP if deep_bf16(cfg) else TOL[cfg["dtype"]]


class noisy_rounding:
    """Within the block, the oracle's bf16 rounding first multiplies each
    value by (1 + NOISE_REL z), z standard normal (seeded): the oracle
    then differs from itself the way the GPU differs from it, by
    accumulation-order noise ahead of the same rounding points."""

    def __init__(self, seed):
        self.rng = np.random.default_rng(seed)

    def __enter__(self):
        import oracle.model as om
        self.om, self.exact = om, om.round_bf16
        rng, exact = self.rng, self.exact

        def rnd(x):
            x = np.asarray(x, dtype=np.float64)
            return exact(x * (1.0 + rng.standard_normal(x.shape) * NOISE_REL))
        om.round_bf16 = rnd
        return self

    def __exit__(self, *exc):
        self.om.round_bf16 = self.exact
        return False


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


def unpool_windows(w):
    """Inverse of pool_windows: [Bt,H/2,W/2,4,C] -> [Bt,H,W,C]."""
    Bt, Hp, Wp, _, C = w.shape
    return (w.reshape(Bt, Hp, Wp, 2, 2, C).transpose(0, 1, 3, 2, 4, 5)
            .reshape(Bt, 2 * Hp, 2 * Wp, C))


def routed_gradient(g, route):
    """The pre-activation gradient of a conv whose 2 x 2 max pool keeps
    routing codes (route [Bt,H/2,W/2,C]: window position 0..3 of the
    gradient g [Bt,H/2,W/2,C], 4 for none): g at the routed position of each
    window, zero elsewhere, [Bt,H,W,C]."""
    w = np.zeros(g.shape[:3] + (4,) + g.shape[3:], dtype=g.dtype)
    for k in range(4):
        w[:, :, :, k, :] = np.where(route == k, g, 0)
    return unpool_windows(w)


def layer_shapes(cfg):
    """Output shape [B, ...] of every layer of the workload's model."""
    h, w, c = cfg["H"], cfg["W"], cfg["Cin"]
    out = []
    for spec in cfg["layers"]:
        kind = spec[0]
        if kind == "conv":
            c = spec[2]
        elif kind == "block":
            c = spec[2]
            h, w = (h - 1) // spec[3] + 1, (w - 1) // spec[3] + 1
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
        self.kink = bar(cfg)
        self.tie = (bar(cfg), bar(cfg))
        shapes = layer_shapes(cfg)
        layers = cfg["layers"]
        self.relu, self.pool, self.flips = {}, {}, {}
        self.route = {}  # conv i -> routing codes of its max pool (no unpooled output stored)
        self.worst = 0.0  # largest near-tie distance seen, as a fraction of its tensor's scale
        for i, spec in enumerate(layers):
            kind = spec[0]
            normed = i + 1 < len(layers) and layers[i + 1][0] in ("bnorm", "gnorm")
            if (kind == "conv" and not normed) or kind in ("bnorm", "gnorm", "block"):
                a = replica_tensor(ctx, f"act{i}", n, shapes[i])
                if a is not None:
                    self.relu[i] = a > 0
                    if i + 1 < len(layers) and layers[i + 1][0] == "maxpool":
                        self.pool[i + 1] = np.argmax(pool_windows(a), axis=3)
                elif i + 1 < len(layers) and layers[i + 1][0] == "maxpool":
                    r = replica_tensor(ctx, f"route{i + 1}", n, shapes[i + 1])
                    if r is not None:
                        r = r.astype(np.int64)
                        assert r.max() <= 4, ("routing code out of range", i + 1)
                        self.route[i] = r
                        # an all-zero window routes nothing; its first maximum is position 0
                        self.pool[i + 1] = np.where(r < 4, r, 0)
            if kind == "block":  # the block's inner ReLU, after its first norm
                a1 = replica_tensor(ctx, f"act{i}.n1", n, shapes[i])
                if a1 is not None:
                    self.relu[(i, "n1")] = a1 > 0

    def __call__(self, kind, i, own, values):
        if kind == "relu" and i in self.route:
            # on at each window's routed position, off at all four where
            # nothing is routed, the oracle's own elsewhere
            r = self.route[i]
            w = pool_windows(own).copy()
            for k in range(4):
                w[:, :, :, k, :] = np.where(r == 4, False, np.where(r == k, True, w[:, :, :, k, :]))
            self.relu[i] = unpool_windows(w)
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


def replayed(choices):
    """The GPU's decisions of a round whose LazyChoices the exact oracle has
    already validated, handed on unchecked (for the twin oracle of twin_bar,
    whose noisy values sit further from the GPU's than the exact oracle's)."""
    def one(c):
        return lambda kind, i, own, values: c.relu[i] if kind == "relu" else c.pool[i]
    return {n: one(c) for n, c in choices.items()}


def vanishing_biases(cfg):
    """{(layer, bias tag): weight tag} of the biases with an exactly zero
    loss gradient in exact arithmetic: a conv followed by batch norm (the
    batch mean subtracts any per-channel constant), in a block with batch
    norm every conv's.  Both sides then hold rounding noise of their own
    precision in its gradient, momentum and update."""
    layers = cfg["layers"]
    out = {}
    for i, sp in enumerate(layers):
        if sp[0] == "conv" and i + 1 < len(layers) and layers[i + 1][0] == "bnorm":
            out[(i, "b")] = "w"
        if sp[0] == "block" and sp[4] == 0:
            out.update({(i, "b1"): "w1", (i, "b2"): "w2", (i, "bp"): "wp"})
    return out


def master_ulp(theta, roundings=1):
    """Resolution of fp32 masters at theta after `roundings` stored updates
    and fusions: each one rounds the master to fp32, so two runs whose
    arithmetic differs in the last bits can end up to one spacing apart per
    rounding."""
    return roundings * np.spacing(np.abs(np.asarray(theta, dtype=np.float32))).astype(np.float64)


def param_distances(got, want, cfg, ulp=None):
    """Per layer weight and bias of two flat parameter-shaped vectors:
    yields (layer, tag, l2, mx), the relative L2 and max distances.  A bias
    whose gradient vanishes exactly (vanishing_biases) has l2 = 0 and mx on
    the scale of its layer's weight: max|a - b| / max|weight entries of b|.
    ulp (for differences of fp32 masters, e.g. an update theta_T - theta_0):
    per-element resolution of the stored values (master_ulp), subtracted
    from each element's difference first (a gradient that differs in its
    last bits can round a master to the neighbouring fp32 value)."""
    from gcpsl_inputs import param_layout
    zero = vanishing_biases(cfg)
    wmax = {}
    for li, tag, shp, off in param_layout(cfg):
        size = int(np.prod(shp))
        a = np.asarray(got[off:off + size], dtype=np.float64)
        b = np.asarray(want[off:off + size], dtype=np.float64)
        res = 0.0 if ulp is None else ulp[off:off + size]
        beyond = np.maximum(np.abs(a - b) - res, 0.0)
        if tag.startswith("w"):
            wmax[(li, tag)] = np.abs(b).max()
        if (li, tag) in zero:
            yield li, tag, 0.0, beyond.max() / (wmax[(li, zero[(li, tag)])] + 1e-30)
            continue
        yield (li, tag, np.linalg.norm(beyond) / (np.linalg.norm(b) + 1e-30),
               beyond.max() / (np.abs(b).max() + 1e-30))


def compare_params(got, want, cfg, tol, what, ulp=None):
    """Every layer's weight and bias on its own (param_distances), so an
    error in one layer cannot hide behind another's magnitude: both relative
    distances within tol."""
    for li, tag, l2, mx in param_distances(got, want, cfg, ulp):
        assert l2 <= tol and mx <= tol, (what, li, tag, l2, mx)


def twin_bar(tol, cfg, pairs):
    """The bar for a deep bf16 network's per-tensor comparisons after
    several rounds: max(tol, twice the largest distance, over every tensor
    of every (twin, want, ulp) pair, of a twin oracle run under
    noisy_rounding from the exact oracle).  One figure for the whole run:
    a single tensor's distance under the noise varies several-fold from
    one noise sample to the next, the largest over all tensors by less than
    2x (test_parity_bar)."""
    worst = 0.0
    for twin, want, ulp in pairs:
        for _, _, l2, mx in param_distances(twin, want, cfg, ulp):
            worst = max(worst, l2, mx)
    return max(tol, 2.0 * worst)
