"""Split CNN forward and backward pass in fp64 (Sec. III-A, Alg. 2).

A participating client evaluates the client segment up to the cut, the
server finishes the forward pass and the loss, and returns the cut gradient,
from which the client segment's gradient follows (Sec. III-A; Alg. 2, the
cluster-local round).  On one device the cut gradient is simply the
gradient with respect to the cut activation.  The client-gradient average of
Sec. III-B is the gradient of the batch-mean loss: a b_k/B weighted mean of
the active clients' mean gradients, i.e. centralised mini-batch SGD on the
cluster's batch.

Layer definitions (readings; the paper's ResNet-18 is replaced by the
workloads' plain CNNs):
  conv       3x3 cross-correlation, stride 1, zero padding 1, bias, then ReLU;
             with residual, ReLU(conv(x) + b + x).  ReLU'(0) = 0.
  maxpool    2x2, stride 2; the gradient goes to the first maximum of the
             window in row-major order (strict >).
  avgpool    mean over the spatial positions.
  linear     logits = h W^T + b.
  loss       softmax cross-entropy, mean over the batch.
  bnorm      batch normalisation of the preceding conv's output (that conv
             then has no ReLU of its own): per channel, mean and biased
             variance over (batch, H, W), x_hat = (z - mean) / sqrt(var +
             1e-5), out = ReLU(gamma x_hat + beta).  The server segment's
             normalisation (Sec. IV-B).
  gnorm      group normalisation (Wu and He 2018): the same with mean and
             variance per example over (H, W, the channels of a group).  The
             client segment's normalisation (Sec. IV-B).

BatchNorm's running statistics (Sec. IV-B: running mean, running variance
and batch counter, the server normalisation state) follow the PyTorch
convention: with momentum 0.1, running_mean <- 0.9 running_mean + 0.1 mean,
running_var <- 0.9 running_var + 0.1 var * n / (n - 1) (the unbiased batch
variance over n values), counter <- counter + 1.

bf16 workloads round to bf16 (round-to-nearest-even) at these points and keep
everything else in fp64: the gathered images; the conv and linear weight
matrices (biases stay at the master's precision); every conv output after
its ReLU, or its raw output when a norm layer follows; every norm output
after its ReLU; the average-pool output; the gradient with respect to each
conv's pre-activation and each norm's pre-ReLU value; and each input
gradient a conv returns (including the cut gradient).  Norm statistics and
parameters stay unrounded.  Logits, loss, logit gradients, parameter gradients stay unrounded.

Conv uses im2col with a library matmul for the forward pass and the weight
gradient, and the textbook col2im scatter for the input gradient.
"""
from __future__ import annotations

import numpy as np
import torch

from gcpsl_inputs import param_layout


def round_bf16(x):
    """Round fp64 values to the nearest bf16 value, ties to even.

    bf16 keeps 8 significant bits and the fp32 exponent range.  For a normal
    fp64 value that is the fp64 bit pattern with its 45 low mantissa bits
    rounded away: add half a bf16 unit minus one plus the kept last bit (ties
    go to the even neighbour) and clear the 45 bits; a carry out of the
    mantissa correctly moves the value to the next binade.  Below 2^-126 bf16
    values are multiples of 2^-133, which is rounded on its own."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    bits = torch.from_numpy(x).view(torch.int64)  # two's complement add == unsigned add
    r = ((bits + (((bits >> 45) & 1) + ((1 << 44) - 1))) & ~((1 << 45) - 1)).view(torch.float64).numpy()
    tiny = np.flatnonzero(np.abs(x) < 2.0 ** -126)
    if tiny.size:
        r.reshape(-1)[tiny] = np.ldexp(np.rint(np.ldexp(x.reshape(-1)[tiny], 133)), -133)
    return r


def _identity(x):
    return np.asarray(x, dtype=np.float64)


def rounder(dtype: str):
    return round_bf16 if dtype == "bf16" else _identity


# ----------------------------------------------------------------- layers

def im2col3x3(x):
    """[Bt,H,W,Ci] -> [Bt*H*W, 9*Ci], column order (kernel row, kernel col, ci):
    column (r, s, i) of pixel (h, w) is x[h + r - 1, w + s - 1, i], zero
    outside the image.  (The nine shifted copies are plain element copies;
    torch's CPU copy only spreads them over the host threads.)"""
    Bt, H, W, Ci = x.shape
    xp = torch.zeros((Bt, H + 2, W + 2, Ci), dtype=torch.float64)
    xp[:, 1:-1, 1:-1, :] = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64))
    cols = torch.empty((Bt, H, W, 3, 3, Ci), dtype=torch.float64)
    for r in range(3):
        for s in range(3):
            cols[:, :, :, r, s, :] = xp[:, r:r + H, s:s + W, :]
    return cols.numpy().reshape(Bt * H * W, 9 * Ci)


def conv3x3_forward(x, w, b):
    """Pre-activation y[b,h,w,o] = b[o] + sum_{r,s,i} x[b,h+r-1,w+s-1,i] w[o,r,s,i]."""
    Bt, H, W, _ = x.shape
    Co = w.shape[0]
    return (im2col3x3(x) @ w.reshape(Co, -1).T + b).reshape(Bt, H, W, Co)


def conv3x3_backward(x, w, gp):
    """Given dL/dpre gp [Bt,H,W,Co]: (dL/dx, dL/dw, dL/db)."""
    Bt, H, W, Ci = x.shape
    Co = w.shape[0]
    gf = gp.reshape(-1, Co)
    dw = (gf.T @ im2col3x3(x)).reshape(w.shape)
    db = gf.sum(axis=0)
    dcols = torch.from_numpy((gf @ w.reshape(Co, -1)).reshape(Bt, H, W, 3, 3, Ci))
    # col2im: each column's value added back to the input pixel it was read
    # from, taps in (r, s) order
    dxp = torch.zeros((Bt, H + 2, W + 2, Ci), dtype=torch.float64)
    for r in range(3):
        for s in range(3):
            dxp[:, r:r + H, s:s + W, :] += dcols[:, :, :, r, s, :]
    return dxp[:, 1:-1, 1:-1, :].numpy(), dw, db


def _windows(x):
    Bt, H, W, C = x.shape
    return (x.reshape(Bt, H // 2, 2, W // 2, 2, C).transpose(0, 1, 3, 2, 4, 5)
            .reshape(Bt, H // 2, W // 2, 4, C))


def maxpool2_forward(x):
    """(pooled, arg) with arg the first row-major maximum of each 2x2 window."""
    win = _windows(x)
    arg = np.argmax(win, axis=3)
    return np.take_along_axis(win, arg[:, :, :, None, :], axis=3)[:, :, :, 0, :], arg


def maxpool2_select(x, arg):
    """Pooled values of x at the given window positions arg."""
    return np.take_along_axis(_windows(x), arg[:, :, :, None, :], axis=3)[:, :, :, 0, :]


def maxpool2_backward(gz, arg):
    Bt, Hh, Wh, C = gz.shape
    win = np.zeros((Bt, Hh, Wh, 4, C))
    np.put_along_axis(win, arg[:, :, :, None, :], gz[:, :, :, None, :], axis=3)
    return (win.reshape(Bt, Hh, Wh, 2, 2, C).transpose(0, 1, 3, 2, 4, 5)
            .reshape(Bt, 2 * Hh, 2 * Wh, C))


EPS_NORM = 1e-5
BN_MOMENTUM = 0.1


def _group_view(z, groups):
    """[Bt,H,W,C] -> [Bt, H*W, groups, C/groups]: per-example sets of a group."""
    Bt, H, W, C = z.shape
    return z.reshape(Bt, H * W, groups, C // groups)


def norm_forward(z, gamma, beta, groups=None):
    """Pre-ReLU output and statistics of batch (groups None) or group
    normalisation.  Returns (u, x_hat, rstd, mean, var_biased)."""
    if groups is None:
        mean = z.mean(axis=(0, 1, 2))
        var = z.var(axis=(0, 1, 2))
        rstd = 1.0 / np.sqrt(var + EPS_NORM)
        x_hat = (z - mean) * rstd
    else:
        zg = _group_view(z, groups)
        mean = zg.mean(axis=(1, 3), keepdims=True)
        var = zg.var(axis=(1, 3), keepdims=True)
        rstd = 1.0 / np.sqrt(var + EPS_NORM)
        x_hat = ((zg - mean) * rstd).reshape(z.shape)
    return gamma * x_hat + beta, x_hat, rstd, mean, var


def norm_backward(du, x_hat, rstd, gamma, groups=None):
    """(dz, dgamma, dbeta) from the gradient du of the pre-ReLU output."""
    dgamma = (du * x_hat).sum(axis=(0, 1, 2))
    dbeta = du.sum(axis=(0, 1, 2))
    dxh = du * gamma
    if groups is None:
        dz = rstd * (dxh - dxh.mean(axis=(0, 1, 2)) - x_hat * (dxh * x_hat).mean(axis=(0, 1, 2)))
    else:
        g = _group_view(dxh, groups)
        xg = _group_view(x_hat, groups)
        dz = (rstd * (g - g.mean(axis=(1, 3), keepdims=True)
                      - xg * (g * xg).mean(axis=(1, 3), keepdims=True))).reshape(du.shape)
    return dz, dgamma, dbeta


def bn_running_update(mean_run, var_run, count, mean, var_biased, n):
    """One running-statistics update (PyTorch convention, momentum 0.1)."""
    m = BN_MOMENTUM
    return ((1.0 - m) * mean_run + m * mean, (1.0 - m) * var_run + m * var_biased * n / (n - 1), count + 1.0)


def softmax_xent(logits, y, eps=0.0):
    """Mean softmax cross-entropy and its gradient with respect to the logits.

    With label smoothing eps (Sec. V-A) the target of an example with label
    y is q = (1 - eps) onehot(y) + eps / L; the loss is -sum_j q_j log p_j
    and its gradient p - q (eps = 0: plain cross-entropy)."""
    Bt, L = logits.shape
    z = logits - logits.max(axis=1, keepdims=True)
    lse = np.log(np.exp(z).sum(axis=1))
    rows = np.arange(Bt)
    q = np.full((Bt, L), eps / L)
    q[rows, y] += 1.0 - eps
    logp = z - lse[:, None]
    loss = float(np.mean(-(q * logp).sum(axis=1)))
    d = np.exp(logp) - q
    return loss, d / Bt


# --------------------------------------------------------- parameter views

def unflatten(cfg, theta):
    """{layer index: {'w': array, 'b': array}} views into a flat vector."""
    out = {}
    for i, tag, shp, off in param_layout(cfg):
        n = int(np.prod(shp))
        out.setdefault(i, {})[tag] = theta[off:off + n].reshape(shp)
    return out


# ------------------------------------------------------------- split step

def split_forward_backward(cfg, theta, x, y, keep=False, choose=None):
    """One cluster-local round's loss and flat gradient for one replica.

    theta: flat parameters (fp64 view of the fp32 master); x: [B,H,W,Cin]
    gathered images; y: [B] labels.  Returns (loss, grad[P], record) where
    record holds each bnorm layer's batch mean, biased variance and value
    count under "bn_batch" and (if keep) every intermediate tensor, keyed by
    name.

    The pass takes two kinds of discrete decisions: whether a ReLU passes a
    value (its output is > 0) and which pixel of a 2 x 2 window the max pool
    takes (the first maximum in row-major order).  Where two candidates are
    within rounding of each other at the working precision, either decision
    is a correct result.  choose, if given, is called at every decision as
    choose(kind, layer, own, values) with kind "relu" (own: boolean mask of
    the layer's output, values: its pre-activation) or "pool" (own: window
    index per pooled value, values: the windows [Bt, H/2, W/2, 4, C]) and
    returns the decision the pass then follows."""
    rnd = rounder(cfg["dtype"])
    layers = cfg["layers"]
    p = unflatten(cfg, np.asarray(theta, dtype=np.float64))
    rec = {}
    acts = [rnd(x)]
    args = {}
    norm = {}
    mask = {}
    rec["bn_batch"] = {}

    def relu(i, v):
        own = rnd(np.maximum(v, 0.0)) > 0
        mask[i] = own if choose is None else np.asarray(choose("relu", i, own, v), dtype=bool)
        return rnd(np.where(mask[i], v, 0.0))

    for i, spec in enumerate(layers):
        a = acts[-1]
        kind = spec[0]
        if kind == "conv":
            pre = conv3x3_forward(a, rnd(p[i]["w"]), p[i]["b"])
            if spec[3]:
                pre = pre + a
            if keep:
                rec[f"pre{i}"] = pre
            normed = i + 1 < len(layers) and layers[i + 1][0] in ("bnorm", "gnorm")
            out = rnd(pre) if normed else relu(i, pre)
        elif kind in ("bnorm", "gnorm"):
            groups = spec[2] if kind == "gnorm" else None
            u, x_hat, rstd, mean, var = norm_forward(a, p[i]["w"], p[i]["b"], groups)
            norm[i] = (x_hat, rstd, groups)
            if kind == "bnorm":
                rec["bn_batch"][i] = (mean, var, a.shape[0] * a.shape[1] * a.shape[2])
            if keep:
                rec[f"pre{i}"] = u
            out = relu(i, u)
        elif kind == "maxpool":
            out, args[i] = maxpool2_forward(a)
            if choose is not None:
                args[i] = np.asarray(choose("pool", i, args[i], _windows(a)))
                out = maxpool2_select(a, args[i])
        elif kind == "avgpool":
            out = rnd(a.mean(axis=(1, 2)))
        elif kind == "linear":
            out = a @ rnd(p[i]["w"]).T + p[i]["b"]
        else:
            raise ValueError(kind)
        acts.append(out)
    loss, g = softmax_xent(acts[-1], y, cfg.get("label_smoothing", 0.0))
    if keep:
        rec["acts"] = acts
        rec["dlogits"] = g
        rec["relu_mask"] = mask
        rec["pool_arg"] = args
    grad = np.zeros(len(theta))
    gview = unflatten(cfg, grad)
    for i in range(len(layers) - 1, -1, -1):
        spec = layers[i]
        a_in, a_out = acts[i], acts[i + 1]
        kind = spec[0]
        if kind == "linear":
            gview[i]["w"][...] = g.T @ a_in
            gview[i]["b"][...] = g.sum(axis=0)
            g = g @ rnd(p[i]["w"])
        elif kind == "avgpool":
            Bt, H, W, C = a_in.shape
            g = np.broadcast_to((g / (H * W))[:, None, None, :], a_in.shape).copy()
        elif kind == "maxpool":
            g = maxpool2_backward(g, args[i])
        elif kind in ("bnorm", "gnorm"):
            du = rnd(g * mask[i])
            if keep:
                rec[f"gpre{i}"] = du
            x_hat, rstd, groups = norm[i]
            dz, dgamma, dbeta = norm_backward(du, x_hat, rstd, p[i]["w"], groups)
            gview[i]["w"][...] = dgamma
            gview[i]["b"][...] = dbeta
            g = rnd(dz)
        elif kind == "conv":
            normed = i + 1 < len(layers) and layers[i + 1][0] in ("bnorm", "gnorm")
            gp = g if normed else rnd(g * mask[i])
            if keep:
                rec[f"gpre{i}"] = gp
            dx, dw, db = conv3x3_backward(a_in, rnd(p[i]["w"]), gp)
            gview[i]["w"][...] = dw
            gview[i]["b"][...] = db
            if i == 0:
                g = None
                break
            g = dx + gp if spec[3] else dx
            g = rnd(g)
        if keep:
            rec[f"gin{i}"] = g
    return loss, grad, rec
