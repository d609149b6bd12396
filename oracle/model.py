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
  block      ResNet basic block (He et al. 2016; the paper's ResNet-18,
             Sec. V-A): conv3x3 with the block's stride (pad 1) -> norm ->
             ReLU -> conv3x3 -> norm; the shortcut is the block input, or a
             1x1 conv with the stride (no pad) -> norm when the shape
             changes; the output is ReLU(second norm + shortcut).  Batch norm
             (groups 0, server) or group norm (client), as above.

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
gradient a conv returns (including the cut gradient).  Inside a block the
same holds for each of its convs and norms (the shortcut norm's output is
rounded; the block output after its ReLU; the gradient at the sum before
that ReLU; the block's input gradient = the rounded sum of its first conv's
input gradient and the shortcut's).  Norm statistics and parameters stay
unrounded.  Logits, loss, logit gradients, parameter gradients stay unrounded.

Conv uses im2col with a library matmul for the forward pass and the weight
gradient, and the textbook col2im scatter for the input gradient.
"""
from __future__ import annotations

import numpy as np
import torch

from gcpsl_inputs import param_layout
from gcpsl_inputs.configs import block_has_projection


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

def conv_out_size(n, k, stride, pad):
    return (n + 2 * pad - k) // stride + 1


def im2col(x, R, S, stride, pad):
    """[Bt,H,W,Ci] -> [Bt*Ho*Wo, R*S*Ci], column order (kernel row, kernel
    col, ci): column (r, s, i) of output pixel (ho, wo) is
    x[ho*stride + r - pad, wo*stride + s - pad, i], zero outside the image.
    (The shifted copies are plain element copies; torch's CPU copy only
    spreads them over the host threads.)"""
    Bt, H, W, Ci = x.shape
    Ho, Wo = conv_out_size(H, R, stride, pad), conv_out_size(W, S, stride, pad)
    xp = torch.zeros((Bt, H + 2 * pad, W + 2 * pad, Ci), dtype=torch.float64)
    xp[:, pad:pad + H, pad:pad + W, :] = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64))
    cols = torch.empty((Bt, Ho, Wo, R, S, Ci), dtype=torch.float64)
    for r in range(R):
        for s in range(S):
            cols[:, :, :, r, s, :] = xp[:, r:r + stride * (Ho - 1) + 1:stride, s:s + stride * (Wo - 1) + 1:stride, :]
    return cols.numpy().reshape(Bt * Ho * Wo, R * S * Ci)


def im2col3x3(x):
    """The 3x3, stride 1, pad 1 columns."""
    return im2col(x, 3, 3, 1, 1)


def conv_forward(x, w, b, stride=1, pad=1):
    """Pre-activation y[b,ho,wo,o] = b[o] + sum_{r,s,i} x[b, ho*stride+r-pad,
    wo*stride+s-pad, i] w[o,r,s,i] (cross-correlation, zero padding)."""
    Bt, H, W, _ = x.shape
    Co, R, S, _ = w.shape
    Ho, Wo = conv_out_size(H, R, stride, pad), conv_out_size(W, S, stride, pad)
    return (im2col(x, R, S, stride, pad) @ w.reshape(Co, -1).T + b).reshape(Bt, Ho, Wo, Co)


def conv_backward(x, w, gp, stride=1, pad=1):
    """Given dL/dpre gp [Bt,Ho,Wo,Co]: (dL/dx, dL/dw, dL/db)."""
    Bt, H, W, Ci = x.shape
    Co, R, S, _ = w.shape
    _, Ho, Wo, _ = gp.shape
    gf = gp.reshape(-1, Co)
    dw = (gf.T @ im2col(x, R, S, stride, pad)).reshape(w.shape)
    db = gf.sum(axis=0)
    dcols = torch.from_numpy((gf @ w.reshape(Co, -1)).reshape(Bt, Ho, Wo, R, S, Ci))
    # col2im: each column's value added back to the input pixel it was read
    # from, taps in (r, s) order
    dxp = torch.zeros((Bt, H + 2 * pad, W + 2 * pad, Ci), dtype=torch.float64)
    for r in range(R):
        for s in range(S):
            dxp[:, r:r + stride * (Ho - 1) + 1:stride, s:s + stride * (Wo - 1) + 1:stride, :] += dcols[:, :, :, r, s, :]
    return dxp[:, pad:pad + H, pad:pad + W, :].numpy(), dw, db


def conv3x3_forward(x, w, b):
    """Pre-activation y[b,h,w,o] = b[o] + sum_{r,s,i} x[b,h+r-1,w+s-1,i] w[o,r,s,i]."""
    return conv_forward(x, w, b, 1, 1)


def conv3x3_backward(x, w, gp):
    """Given dL/dpre gp [Bt,H,W,Co]: (dL/dx, dL/dw, dL/db)."""
    return conv_backward(x, w, gp, 1, 1)


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
        elif kind == "block":
            _, cin, cout, stride, groups = spec
            gr, q = groups or None, p[i]
            z1 = rnd(conv_forward(a, rnd(q["w1"]), q["b1"], stride, 1))
            u1, xh1, rs1, m1, v1 = norm_forward(z1, q["n1w"], q["n1b"], gr)
            a1 = relu((i, "n1"), u1)
            z2 = rnd(conv_forward(a1, rnd(q["w2"]), q["b2"], 1, 1))
            u2, xh2, rs2, m2, v2 = norm_forward(z2, q["n2w"], q["n2b"], gr)
            st = {"n1": (z1, xh1, rs1, m1, v1), "n2": (z2, xh2, rs2, m2, v2), "a1": a1}
            if block_has_projection(spec):
                zp = rnd(conv_forward(a, rnd(q["wp"]), q["bp"], stride, 0))
                up, xhp, rsp, mp, vp = norm_forward(zp, q["npw"], q["npb"], gr)
                st["np"] = (zp, xhp, rsp, mp, vp)
                sc = rnd(up)
            else:
                sc = a
            norm[i] = st
            if gr is None:
                for sub in ("n1", "n2", "np"):
                    if sub in st:
                        z_, _, _, mean_, var_ = st[sub]
                        rec["bn_batch"][(i, sub)] = (mean_, var_, z_.shape[0] * z_.shape[1] * z_.shape[2])
            if keep:
                rec[f"pre{i}"] = u2 + sc
                rec[f"pre{i}.n1"] = u1
                rec[f"z{i}.1"], rec[f"z{i}.2"], rec[f"act{i}.n1"] = z1, z2, a1
                if "np" in st:
                    rec[f"z{i}.p"], rec[f"sc{i}"] = st["np"][0], sc
            out = relu(i, u2 + sc)
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
        elif kind == "block":
            _, cin, cout, stride, groups = spec
            gr, q, st = groups or None, p[i], norm[i]
            du2 = rnd(g * mask[i])  # at the sum before the block's last ReLU
            z2, xh2, rs2, _, _ = st["n2"]
            dz2, gview[i]["n2w"][...], gview[i]["n2b"][...] = norm_backward(du2, xh2, rs2, q["n2w"], gr)
            dz2 = rnd(dz2)
            da1, gview[i]["w2"][...], gview[i]["b2"][...] = conv_backward(st["a1"], rnd(q["w2"]), dz2, 1, 1)
            du1 = rnd(da1 * mask[(i, "n1")])
            z1, xh1, rs1, _, _ = st["n1"]
            dz1, gview[i]["n1w"][...], gview[i]["n1b"][...] = norm_backward(du1, xh1, rs1, q["n1w"], gr)
            dz1 = rnd(dz1)
            dx, gview[i]["w1"][...], gview[i]["b1"][...] = conv_backward(a_in, rnd(q["w1"]), dz1, stride, 1)
            if "np" in st:
                zp, xhp, rsp, _, _ = st["np"]
                dzp, gview[i]["npw"][...], gview[i]["npb"][...] = norm_backward(du2, xhp, rsp, q["npw"], gr)
                dzp = rnd(dzp)
                dxs, gview[i]["wp"][...], gview[i]["bp"][...] = conv_backward(a_in, rnd(q["wp"]), dzp, stride, 0)
                dxs = rnd(dxs)
            else:
                dxs = du2
            if keep:
                rec[f"gpre{i}"], rec[f"gpre{i}.n1"], rec[f"dz{i}.1"], rec[f"dz{i}.2"] = du2, du1, dz1, dz2
                if "np" in st:
                    rec[f"dz{i}.p"], rec[f"gsc{i}"] = dzp, dxs
            g = rnd(dx + dxs)
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
