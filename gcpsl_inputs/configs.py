"""Workload descriptions.

Each workload names the client population (K clients, C clusters, batch B per
cluster, L classes), the synthetic data set (N_ex images of H x W x Cin, a
Dirichlet(alpha) label split), the split CNN (a list of layers and the cut
index), the compute precision and the optimiser / fusion schedule.

Layer tuples:
    ("conv", cin, cout, residual)   3x3 conv, stride 1, zero pad 1, bias, ReLU;
                                    residual=True adds the layer input before
                                    the ReLU (requires cin == cout)
    ("maxpool",)                    2x2 / stride 2 max pool
    ("avgpool",)                    global average pool over H x W
    ("linear", cin, cout)           fully connected layer producing the logits
    ("bnorm", ch)                   batch normalisation over (batch, H, W) per
                                    channel, affine (gamma, beta), then ReLU;
                                    follows a conv without residual, whose
                                    output it normalises
    ("gnorm", ch, groups)           group normalisation over (H, W, channels
                                    of a group) per example, affine, then ReLU
    ("block", cin, cout, stride, groups)
                                    ResNet basic block: conv3x3 (stride,
                                    pad 1) -> norm -> ReLU -> conv3x3 -> norm,
                                    plus the shortcut (the input itself, or
                                    conv1x1 (stride, no pad) -> norm when
                                    stride > 1 or cin != cout), added before
                                    the final ReLU; norm = batch norm
                                    (groups 0) or group norm (groups)

The client segment is layers[:cut]; the server segment is layers[cut:].

schedule (default "lockstep"): "lockstep" runs every cluster's round at every
step and fuses every F steps; "epoch" runs the epoch-barrier schedule (each
cluster floor(n_n / B) rounds per system epoch, fusion after the epoch).

Parameter layout (one flat fp32 vector of P entries per replica): for every
conv / linear / norm layer in order, its weight followed by its bias.  Conv
weights are stored [cout][3][3][cin] (output channel, kernel row, kernel
column, input channel); linear weights [cout][cin]; a norm layer's weight is
gamma[ch], its bias beta[ch].

Normalisation state (one flat fp32 vector of S entries per replica): for
every bnorm layer in order, running mean[ch], running variance[ch] and the
batch counter.
"""
from __future__ import annotations

import copy

_CIFAR_CLIENT = [("conv", 3, 32, False), ("conv", 32, 64, False), ("maxpool",)]
_SERVER_NARROW = [("conv", 64, 128, False), ("conv", 128, 128, False), ("maxpool",),
                  ("avgpool",), ("linear", 128, 10)]
# Wide residual server: 64->256, then three 256->256 convs whose output is
# ReLU(conv(x) + b + x).
_SERVER_WIDE = [("conv", 64, 256, False), ("conv", 256, 256, True), ("conv", 256, 256, True),
                ("conv", 256, 256, True), ("maxpool",), ("avgpool",), ("linear", 256, 10)]

_CIFAR_DATA = dict(N_ex=50000, H=32, W=32, Cin=3, L=10, noise_std=0.5)


def _resnet(widths, client_groups, blocks=2, classes=10):
    """ResNet-18 for 32 x 32 inputs split after its second stage (Sec. V-A):
    a 3x3 stem conv with group norm, then four stages of `blocks` basic
    blocks of the given widths (stride 2 at the first block of stages 2-4),
    group norm in the client segment (stem and stages 1-2) and batch norm in
    the server segment (stages 3-4), global average pool, linear head."""
    layers = [("conv", 3, widths[0], False), ("gnorm", widths[0], client_groups)]
    cin = widths[0]
    for st, w in enumerate(widths):
        for b in range(blocks):
            stride = 2 if (st > 0 and b == 0) else 1
            layers.append(("block", cin, w, stride, client_groups if st < 2 else 0))
            cin = w
    layers += [("avgpool",), ("linear", cin, classes)]
    return layers, 2 + 2 * blocks  # cut after stage 2

CONFIGS = {
    # Tiny reference workload: 16 clients in 2 random clusters of 8.
    "tiny": dict(
        K=16, C=2, B=8, L=4, N_ex=512, H=8, W=8, Cin=3, noise_std=0.5, alpha=0.5,
        rule="random",
        layers=[("conv", 3, 8, False), ("maxpool",),
                ("conv", 8, 16, False), ("avgpool",), ("linear", 16, 4)],
        cut=2, dtype="f32", lr=0.05, momentum=0.0, F=5, T=10, seed=0),
    # The tiny workload clustered by the paper's label-aware move search
    # (Eq. 4) instead of at random.
    "tiny_jsd": dict(
        K=16, C=2, B=8, L=4, N_ex=512, H=8, W=8, Cin=3, noise_std=0.5, alpha=0.5,
        rule="label_jsd",
        layers=[("conv", 3, 8, False), ("maxpool",),
                ("conv", 8, 16, False), ("avgpool",), ("linear", 16, 4)],
        cut=2, dtype="f32", lr=0.05, momentum=0.0, F=5, T=10, seed=0),
    # Single-workload GPSL baseline (C = 1).
    "gpsl": dict(
        K=256, C=1, B=64, alpha=0.3, rule="random", **_CIFAR_DATA,
        layers=_CIFAR_CLIENT + _SERVER_NARROW, cut=3,
        dtype="f32", lr=0.05, momentum=0.9, F=0, T=500, seed=0),
    # Four random clusters of 64 clients.
    "gcpsl4": dict(
        K=256, C=4, B=64, alpha=0.3, rule="random", **_CIFAR_DATA,
        layers=_CIFAR_CLIENT + _SERVER_NARROW, cut=3,
        dtype="f32", lr=0.05, momentum=0.9, F=50, T=500, seed=0),
    # Eight size-balanced clusters, bf16 activations/weights, fp32 masters.
    "gcpsl8": dict(
        K=256, C=8, B=64, alpha=0.3, rule="size", **_CIFAR_DATA,
        layers=_CIFAR_CLIENT + _SERVER_NARROW, cut=3,
        dtype="bf16", lr=0.05, momentum=0.9, F=25, T=1000, seed=0),
    # Sixteen label-aware clusters, B=128, wide residual server, bf16.
    "gcpsl16": dict(
        K=256, C=16, B=128, alpha=0.1, rule="label_l1", **_CIFAR_DATA,
        layers=_CIFAR_CLIENT + _SERVER_WIDE, cut=3,
        dtype="bf16", lr=0.05, momentum=0.9, F=50, T=1000, seed=0),
    # The paper's model (Sec. V-A): ResNet-18 split after its second stage,
    # group norm in the client segment (32 groups), batch norm in the server
    # segment, on the CIFAR-shaped data: K = 256 clients in N = 4 clusters of
    # the paper's label-aware rule (Eq. 4), B = 64 per cluster, its training
    # recipe (SGD lr 0.01, momentum 0.9, Nesterov, weight decay 5e-4, label
    # smoothing 0.1) and fusion after every epoch (the epoch-barrier
    # schedule).  Precision fp32 (the paper states none).  45,000 training
    # examples: the real-execution study holds 5,000 of CIFAR-10's 50,000 out
    # for validation before partitioning (Sec. V-B).
    "resnet18": dict(
        K=256, C=4, B=64, alpha=0.3, rule="label_jsd", **dict(_CIFAR_DATA, N_ex=45000),
        layers=_resnet((64, 128, 256, 512), 32)[0], cut=_resnet((64, 128, 256, 512), 32)[1],
        dtype="f32", lr=0.01, momentum=0.9, nesterov=True, weight_decay=5e-4, label_smoothing=0.1,
        F=0, T=3, seed=0, schedule="epoch"),
    # The same model and recipe in bf16 (fp32 masters): the paper states no
    # precision, and this is the one the MFMA peak is quoted for.
    "resnet18_bf16": dict(
        K=256, C=4, B=64, alpha=0.3, rule="label_jsd", **dict(_CIFAR_DATA, N_ex=45000),
        layers=_resnet((64, 128, 256, 512), 32)[0], cut=_resnet((64, 128, 256, 512), 32)[1],
        dtype="bf16", lr=0.01, momentum=0.9, nesterov=True, weight_decay=5e-4, label_smoothing=0.1,
        F=0, T=3, seed=0, schedule="epoch"),
    # The same topology at small size (16 x 16 images, widths 8-64), fp32 and
    # bf16: every block kind (identity and projection shortcut, stride 1 and
    # 2, group and batch norm), stage 4 on 2 x 2 maps (batch norm over 64
    # values per channel).
    "resnet_tiny": dict(
        K=16, C=2, B=16, L=4, N_ex=512, H=16, W=16, Cin=3, noise_std=0.5, alpha=0.5,
        rule="random", layers=_resnet((8, 16, 32, 64), 4, classes=4)[0], cut=_resnet((8, 16, 32, 64), 4)[1],
        dtype="f32", lr=0.05, momentum=0.9, F=2, T=4, seed=0),
    "resnet_tiny_bf16": dict(
        K=16, C=2, B=16, L=4, N_ex=512, H=16, W=16, Cin=3, noise_std=0.5, alpha=0.5,
        rule="random", layers=_resnet((8, 16, 32, 64), 4, classes=4)[0], cut=_resnet((8, 16, 32, 64), 4)[1],
        dtype="bf16", lr=0.05, momentum=0.9, F=2, T=4, seed=0, nesterov=True, weight_decay=5e-4,
        label_smoothing=0.1),
    # Small parity workloads whose GEMM sizes are ragged against every tile
    # size (M, N and K tails; more than one N tile; a residual layer).
    "ragged": dict(
        K=24, C=3, B=20, L=7, N_ex=1400, H=12, W=12, Cin=3, noise_std=0.5, alpha=0.5,
        rule="size",
        layers=[("conv", 3, 8, False), ("conv", 8, 24, False), ("maxpool",),
                ("conv", 24, 136, False), ("conv", 136, 136, True), ("maxpool",),
                ("avgpool",), ("linear", 136, 7)],
        cut=3, dtype="f32", lr=0.05, momentum=0.9, F=3, T=7, seed=0),
    "ragged_bf16": dict(
        K=24, C=3, B=20, L=7, N_ex=1400, H=12, W=12, Cin=3, noise_std=0.5, alpha=0.5,
        rule="label_l1",
        layers=[("conv", 3, 8, False), ("conv", 8, 24, False), ("maxpool",),
                ("conv", 24, 136, False), ("conv", 136, 136, True), ("maxpool",),
                ("avgpool",), ("linear", 136, 7)],
        cut=3, dtype="bf16", lr=0.05, momentum=0.9, F=3, T=7, seed=0),
    # Residual server layers whose channel counts are multiples of 64 (the
    # residual is taken from the staged centre tap), with ragged M and no max
    # pool (so no bf16 near-tie routing decision can move a gradient).
    "ragged_res_bf16": dict(
        K=24, C=3, B=19, L=7, N_ex=1400, H=8, W=8, Cin=3, noise_std=0.5, alpha=0.5,
        rule="label_l1",
        layers=[("conv", 3, 16, False), ("conv", 16, 64, False),
                ("conv", 64, 128, False), ("conv", 128, 128, True), ("conv", 128, 128, True),
                ("avgpool",), ("linear", 128, 7)],
        cut=2, dtype="bf16", lr=0.05, momentum=0.9, F=3, T=7, seed=0),
    # 16 x 16 images and 64-channel multiples (the shape of the wide server
    # layers: 256-pixel tiles of one image each), with residual layers and
    # no max pool.
    "halo_res_bf16": dict(
        K=24, C=3, B=3, L=7, N_ex=1400, H=16, W=16, Cin=3, noise_std=0.5, alpha=0.5,
        rule="label_l1",
        layers=[("conv", 3, 16, False), ("conv", 16, 64, False),
                ("conv", 64, 256, False), ("conv", 256, 256, True), ("conv", 256, 256, True),
                ("avgpool",), ("linear", 256, 7)],
        cut=2, dtype="bf16", lr=0.05, momentum=0.9, F=2, T=4, seed=0),
    # The same 16 x 16 residual model at a batch whose weight-gradient plan
    # splits the pixels of each replica into many chunks (chunk boundaries
    # inside images, a shorter last chunk).
    "halo_split_bf16": dict(
        K=24, C=2, B=11, L=7, N_ex=1400, H=16, W=16, Cin=3, noise_std=0.5, alpha=0.5,
        rule="label_l1",
        layers=[("conv", 3, 16, False), ("conv", 16, 64, False),
                ("conv", 64, 256, False), ("conv", 256, 256, True), ("conv", 256, 256, True),
                ("avgpool",), ("linear", 256, 7)],
        cut=2, dtype="bf16", lr=0.05, momentum=0.9, F=2, T=3, seed=0),
    # 16 x 16 images into a 136-channel head conv (one 256-wide tile, 120
    # channels unused) with a 2 x 2 max pool before the mean, the head of
    # the wide 16-cluster workload at small size.
    "halo_maxhead_bf16": dict(
        K=24, C=2, B=5, L=7, N_ex=1400, H=16, W=16, Cin=3, noise_std=0.5, alpha=0.5,
        rule="label_l1",
        layers=[("conv", 3, 16, False), ("conv", 16, 64, False),
                ("conv", 64, 256, False), ("conv", 256, 136, False), ("maxpool",),
                ("avgpool",), ("linear", 136, 7)],
        cut=2, dtype="bf16", lr=0.05, momentum=0.9, F=2, T=3, seed=0),
    # 16 x 16 images into 128-channel server layers (the 8-cluster server's
    # shape): the 128-wide one-buffer halo tile in the forward (one and two
    # 64-channel blocks, a residual layer) and input gradient, and the head's
    # max pool and mean in its epilogue.
    "halo128_bf16": dict(
        K=24, C=2, B=5, L=7, N_ex=1400, H=16, W=16, Cin=3, noise_std=0.5, alpha=0.5,
        rule="label_l1",
        layers=[("conv", 3, 16, False), ("conv", 16, 64, False),
                ("conv", 64, 128, False), ("conv", 128, 128, True), ("conv", 128, 128, False), ("maxpool",),
                ("avgpool",), ("linear", 128, 7)],
        cut=2, dtype="bf16", lr=0.05, momentum=0.9, F=2, T=3, seed=0),
    # 32 x 32 images with the workloads' client layers (3 -> 32 -> 64, max
    # pool), so the image-layer convolution kernels run at small size.
    "img32_bf16": dict(
        K=16, C=2, B=3, L=7, N_ex=602, H=32, W=32, Cin=3, noise_std=0.5, alpha=0.5,
        rule="label_l1",
        layers=[("conv", 3, 32, False), ("conv", 32, 64, False), ("maxpool",),
                ("conv", 64, 64, False), ("avgpool",), ("linear", 64, 7)],
        cut=3, dtype="bf16", lr=0.05, momentum=0.9, F=2, T=3, seed=0),
    # The same client layers on 12 x 12 images: 432 pixels per replica, not
    # a multiple of the image layer's 32-pixel weight-gradient groups.
    "col_ragged_bf16": dict(
        K=16, C=2, B=3, L=7, N_ex=602, H=12, W=12, Cin=3, noise_std=0.5, alpha=0.5,
        rule="label_l1",
        layers=[("conv", 3, 32, False), ("conv", 32, 64, False), ("maxpool",),
                ("conv", 64, 64, False), ("avgpool",), ("linear", 64, 7)],
        cut=3, dtype="bf16", lr=0.05, momentum=0.9, F=2, T=3, seed=0),
    # 20 classes: more than the register-resident classifier head holds, so
    # the LDS-staged head runs (with label smoothing).
    "wide_head_bf16": dict(
        K=16, C=2, B=20, L=20, N_ex=600, H=8, W=8, Cin=3, noise_std=0.5, alpha=0.5,
        rule="label_l1",
        layers=[("conv", 3, 16, False), ("maxpool",), ("conv", 16, 64, False), ("avgpool",),
                ("linear", 64, 20)],
        cut=2, dtype="bf16", lr=0.05, momentum=0.9, F=2, T=4, seed=0, label_smoothing=0.1),
    # GroupNorm in the client segment, BatchNorm in the server segment
    # (Sec. IV-B), whose running statistics are fused with the parameters.
    "tiny_norm": dict(
        K=16, C=2, B=8, L=4, N_ex=512, H=8, W=8, Cin=3, noise_std=0.5, alpha=0.5,
        rule="random",
        layers=[("conv", 3, 8, False), ("gnorm", 8, 2), ("maxpool",),
                ("conv", 8, 16, False), ("bnorm", 16), ("avgpool",), ("linear", 16, 4)],
        cut=3, dtype="f32", lr=0.05, momentum=0.9, F=5, T=10, seed=0),
    # (bf16 without a max pool: normalised bf16 values tie often, and a
    # one-ulp difference would move a max-pool gradient; the fp32 workload
    # above covers norm + max pool)
    "ragged_norm_bf16": dict(
        K=24, C=3, B=20, L=7, N_ex=1400, H=12, W=12, Cin=3, noise_std=0.5, alpha=0.5,
        rule="size",
        layers=[("conv", 3, 8, False), ("gnorm", 8, 4), ("conv", 8, 24, False), ("gnorm", 24, 3),
                ("conv", 24, 136, False), ("bnorm", 136),
                ("conv", 136, 136, False), ("bnorm", 136), ("avgpool",), ("linear", 136, 7)],
        cut=4, dtype="bf16", lr=0.05, momentum=0.9, F=3, T=7, seed=0),
    # The paper's training recipe (Sec. V-A) on the norm models: SGD with
    # momentum 0.9, the Nesterov term and weight decay 5e-4, cross-entropy
    # with label smoothing 0.1.
    "tiny_recipe": dict(
        K=16, C=2, B=8, L=4, N_ex=512, H=8, W=8, Cin=3, noise_std=0.5, alpha=0.5,
        rule="random",
        layers=[("conv", 3, 8, False), ("gnorm", 8, 2), ("maxpool",),
                ("conv", 8, 16, False), ("bnorm", 16), ("avgpool",), ("linear", 16, 4)],
        cut=3, dtype="f32", lr=0.05, momentum=0.9, F=5, T=10, seed=0,
        nesterov=True, weight_decay=5e-4, label_smoothing=0.1),
    "ragged_recipe_bf16": dict(
        K=24, C=3, B=20, L=7, N_ex=1400, H=12, W=12, Cin=3, noise_std=0.5, alpha=0.5,
        rule="size",
        layers=[("conv", 3, 8, False), ("gnorm", 8, 4), ("conv", 8, 24, False), ("gnorm", 24, 3),
                ("conv", 24, 136, False), ("bnorm", 136),
                ("conv", 136, 136, False), ("bnorm", 136), ("avgpool",), ("linear", 136, 7)],
        cut=4, dtype="bf16", lr=0.05, momentum=0.9, F=3, T=7, seed=0,
        nesterov=True, weight_decay=5e-4, label_smoothing=0.1),
    # Epoch-barrier schedule (fusion after every system epoch) on unequal
    # clusters: tiny with B=32 (6 and 9 rounds per epoch), and the ragged
    # shapes under label-L1 clustering with B=100 (7, 4 and 2 rounds).
    "tiny_epoch": dict(
        K=16, C=2, B=32, L=4, N_ex=512, H=8, W=8, Cin=3, noise_std=0.5, alpha=0.5,
        rule="random",
        layers=[("conv", 3, 8, False), ("maxpool",),
                ("conv", 8, 16, False), ("avgpool",), ("linear", 16, 4)],
        cut=2, dtype="f32", lr=0.05, momentum=0.9, F=0, T=18, seed=0, schedule="epoch"),
    "ragged_epoch": dict(
        K=24, C=3, B=100, L=7, N_ex=1400, H=12, W=12, Cin=3, noise_std=0.5, alpha=0.5,
        rule="label_l1",
        layers=[("conv", 3, 8, False), ("conv", 8, 24, False), ("maxpool",),
                ("conv", 24, 136, False), ("conv", 136, 136, True), ("maxpool",),
                ("avgpool",), ("linear", 136, 7)],
        cut=3, dtype="f32", lr=0.05, momentum=0.9, F=0, T=10, seed=0, schedule="epoch"),
    "ragged_bf16_epoch": dict(
        K=24, C=3, B=100, L=7, N_ex=1400, H=12, W=12, Cin=3, noise_std=0.5, alpha=0.5,
        rule="label_l1",
        layers=[("conv", 3, 8, False), ("conv", 8, 24, False), ("maxpool",),
                ("conv", 24, 136, False), ("conv", 136, 136, True), ("maxpool",),
                ("avgpool",), ("linear", 136, 7)],
        cut=3, dtype="bf16", lr=0.05, momentum=0.9, F=0, T=10, seed=0, schedule="epoch"),
}


def block_has_projection(spec) -> bool:
    """A block whose shortcut is a strided 1x1 conv + norm (shape change)."""
    return spec[3] != 1 or spec[1] != spec[2]


# Parameters of a block, in order: (tag, shape) for cin, cout; conv weights
# [cout][r][s][cin], then bias, then the norm's gamma and beta.
def block_params(spec) -> list:
    _, cin, cout, _, _ = spec
    out = [("w1", (cout, 3, 3, cin)), ("b1", (cout,)), ("n1w", (cout,)), ("n1b", (cout,)),
           ("w2", (cout, 3, 3, cout)), ("b2", (cout,)), ("n2w", (cout,)), ("n2b", (cout,))]
    if block_has_projection(spec):
        out += [("wp", (cout, 1, 1, cin)), ("bp", (cout,)), ("npw", (cout,)), ("npb", (cout,))]
    return out


def get_config(name: str, **overrides) -> dict:
    """Return a deep copy of a named workload with optional field overrides."""
    cfg = copy.deepcopy(CONFIGS[name])
    cfg.update(overrides)
    cfg.setdefault("schedule", "lockstep")
    cfg.setdefault("nesterov", False)
    cfg.setdefault("weight_decay", 0.0)
    cfg.setdefault("label_smoothing", 0.0)
    cfg["name"] = name
    return cfg


def model_layers(cfg: dict) -> list:
    """Layer list with the spatial size each layer sees: (spec, H_in, W_in, C_in)."""
    h, w, c = cfg["H"], cfg["W"], cfg["Cin"]
    out = []
    for spec in cfg["layers"]:
        out.append((spec, h, w, c))
        kind = spec[0]
        if kind in ("bnorm", "gnorm"):
            continue
        if kind == "block":
            c = spec[2]
            h, w = (h - 1) // spec[3] + 1, (w - 1) // spec[3] + 1
            continue
        if kind == "conv":
            c = spec[2]
        elif kind == "maxpool":
            h, w = h // 2, w // 2
        elif kind == "avgpool":
            h, w = 1, 1
        elif kind == "linear":
            c = spec[2]
    return out


def param_layout(cfg: dict) -> list:
    """[(layer_index, 'w'|'b', shape, offset)] in the flat parameter order."""
    out, off = [], 0
    for i, spec in enumerate(cfg["layers"]):
        if spec[0] == "conv":
            shapes = [("w", (spec[2], 3, 3, spec[1])), ("b", (spec[2],))]
        elif spec[0] == "linear":
            shapes = [("w", (spec[2], spec[1])), ("b", (spec[2],))]
        elif spec[0] in ("bnorm", "gnorm"):
            shapes = [("w", (spec[1],)), ("b", (spec[1],))]
        elif spec[0] == "block":
            shapes = block_params(spec)
        else:
            continue
        for tag, shp in shapes:
            n = 1
            for d in shp:
                n *= d
            out.append((i, tag, shp, off))
            off += n
    return out


def param_counts(cfg: dict) -> tuple:
    """(P_client, P_server): parameter counts of the two segments."""
    pc = ps = 0
    for i, tag, shp, off in param_layout(cfg):
        n = 1
        for d in shp:
            n *= d
        if i < cfg["cut"]:
            pc += n
        else:
            ps += n
    return pc, ps


def norm_layout(cfg: dict) -> list:
    """[(key, 'mean'|'var'|'count', shape, offset)] of the normalisation
    state: every batch norm in layer order, key = its layer index, or
    (layer index, 'n1' | 'n2' | 'np') for the norms of a block (its first,
    second and shortcut norm, in that order)."""
    out, off = [], 0
    for i, spec in enumerate(cfg["layers"]):
        if spec[0] == "bnorm":
            keys = [(i, spec[1])]
        elif spec[0] == "block" and spec[4] == 0:
            keys = [((i, "n1"), spec[2]), ((i, "n2"), spec[2])]
            if block_has_projection(spec):
                keys.append(((i, "np"), spec[2]))
        else:
            continue
        for key, ch in keys:
            for tag, shp in (("mean", (ch,)), ("var", (ch,)), ("count", (1,))):
                out.append((key, tag, shp, off))
                off += int(shp[0])
    return out
