"""Pins for the oracle's split forward/backward pass.

Each layer is checked against its textbook loop definition, the whole split
step against central finite differences and against torch.autograd on the
unsplit model (a library implementation; C = 1 makes the split model the
plain CNN, Sec. III-A), and the bf16 rounding primitive against torch's
float32 -> bfloat16 conversion.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as tF

from gcpsl_inputs import get_config, init_params, make_dataset, param_layout
from oracle.model import (conv3x3_backward, conv3x3_forward, maxpool2_backward,
                          maxpool2_forward, round_bf16, softmax_xent, split_forward_backward)

torch.set_num_threads(4)


# ------------------------------------------------------------ bf16 rounding

def test_round_bf16_matches_torch_on_fp32_values():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(3.0),
        (rng.standard_normal(2000) * 1e-30).astype(np.float32),
        (rng.standard_normal(2000) * 1e-39).astype(np.float32),   # fp32 subnormals
        np.array([0.0, -0.0, 1.0, 65504.0, 3e38, -3e38], dtype=np.float32),
    ])
    # exact ties: low 16 bits = 0x8000, both even and odd kept parts
    bits = rng.integers(0, 2**31, size=4000, dtype=np.uint32) & np.uint32(0xFFFF0000)
    bits = bits | np.uint32(0x8000)
    ties = bits.view(np.float32)
    ties = ties[np.isfinite(ties)]
    x = np.concatenate([x, ties])
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = round_bf16(x.astype(np.float64))
    assert np.array_equal(got, want)


def test_round_bf16_on_fp64_values_is_single_rounding():
    # 1 + 2^-8 + 2^-40 lies just above the tie between 1 and 1 + 2^-7:
    # correct rounding goes up; rounding via fp32 first would hit the tie and
    # go to even (1).
    v = 1.0 + 2.0 ** -8 + 2.0 ** -40
    assert round_bf16(np.array([v]))[0] == 1.0 + 2.0 ** -7
    assert round_bf16(np.array([1.0 + 2.0 ** -8]))[0] == 1.0          # tie -> even
    assert round_bf16(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6  # tie -> even


# ------------------------------------------------------ textbook definitions

def _conv_loops(x, w, b):
    Bt, H, W, Ci = x.shape
    Co = w.shape[0]
    y = np.zeros((Bt, H, W, Co))
    for n in range(Bt):
        for h in range(H):
            for ww in range(W):
                for o in range(Co):
                    acc = b[o]
                    for r in range(3):
                        for s in range(3):
                            hh, wc = h + r - 1, ww + s - 1
                            if 0 <= hh < H and 0 <= wc < W:
                                acc += np.dot(x[n, hh, wc, :], w[o, r, s, :])
                    y[n, h, ww, o] = acc
    return y


def test_conv_forward_matches_loops():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((2, 5, 4, 3))
    w = rng.standard_normal((4, 3, 3, 3))
    b = rng.standard_normal(4)
    assert np.allclose(conv3x3_forward(x, w, b), _conv_loops(x, w, b), rtol=1e-13, atol=1e-13)


def test_conv_backward_matches_loops():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((2, 4, 3, 2))
    w = rng.standard_normal((3, 3, 3, 2))
    gp = rng.standard_normal((2, 4, 3, 3))
    dx, dw, db = conv3x3_backward(x, w, gp)
    Bt, H, W, Ci = x.shape
    edx = np.zeros_like(x)
    edw = np.zeros_like(w)
    for n in range(Bt):
        for h in range(H):
            for ww in range(W):
                for o in range(3):
                    for r in range(3):
                        for s in range(3):
                            hh, wc = h + r - 1, ww + s - 1
                            if 0 <= hh < H and 0 <= wc < W:
                                edw[o, r, s, :] += gp[n, h, ww, o] * x[n, hh, wc, :]
                                edx[n, hh, wc, :] += gp[n, h, ww, o] * w[o, r, s, :]
    assert np.allclose(dx, edx, atol=1e-13)
    assert np.allclose(dw, edw, atol=1e-13)
    assert np.allclose(db, gp.sum(axis=(0, 1, 2)), atol=1e-13)


def test_maxpool_first_max_tie_rule():
    x = np.zeros((1, 2, 4, 1))
    # window 0: (0,0)=1, (0,1)=3, (1,0)=3, (1,1)=2 -> first max is (0,1)
    x[0, 0, 0, 0], x[0, 0, 1, 0], x[0, 1, 0, 0], x[0, 1, 1, 0] = 1, 3, 3, 2
    # window 1: all equal -> (0,0)
    x[0, :, 2:, 0] = 5
    z, arg = maxpool2_forward(x)
    assert z[0, 0, :, 0].tolist() == [3, 5]
    assert arg[0, 0, :, 0].tolist() == [1, 0]
    g = maxpool2_backward(np.array([[[[7.0], [9.0]]]]), arg)
    want = np.zeros((1, 2, 4, 1))
    want[0, 0, 1, 0] = 7
    want[0, 0, 2, 0] = 9
    assert np.array_equal(g, want)


def test_softmax_xent_matches_torch():
    rng = np.random.default_rng(3)
    logits = rng.standard_normal((9, 5)) * 4
    y = rng.integers(0, 5, size=9)
    loss, d = softmax_xent(logits, y)
    t = torch.tensor(logits, requires_grad=True)
    tl = tF.cross_entropy(t, torch.tensor(y))
    tl.backward()
    assert loss == pytest.approx(tl.item(), rel=1e-14)
    assert np.allclose(d, t.grad.numpy(), atol=1e-15)


@pytest.mark.parametrize("eps", [0.1, 0.3, 0.95])
def test_softmax_xent_label_smoothing_matches_torch(eps):
    rng = np.random.default_rng(4)
    logits = rng.standard_normal((11, 7)) * 3
    y = rng.integers(0, 7, size=11)
    loss, d = softmax_xent(logits, y, eps)
    t = torch.tensor(logits, requires_grad=True)
    tl = tF.cross_entropy(t, torch.tensor(y), label_smoothing=eps)
    tl.backward()
    assert loss == pytest.approx(tl.item(), rel=1e-13)
    assert np.allclose(d, t.grad.numpy(), atol=1e-15)


def test_softmax_xent_label_smoothing_closed_forms():
    # equal logits: p = 1/L for every class, so the loss is log L whatever eps
    # is, and the gradient (p - q)/B is (1 - eps)/(L B) off the label and
    # -(1 - eps)(L - 1)/(L B) on it
    L, B = 5, 3
    for eps in (0.0, 0.1, 0.5):
        loss, d = softmax_xent(np.zeros((B, L)), np.array([0, 2, 4]), eps)
        assert loss == pytest.approx(np.log(L), rel=1e-14)
        assert np.allclose(d.sum(axis=1), 0.0, atol=1e-16)
        off = np.ones((B, L), bool)
        off[[0, 1, 2], [0, 2, 4]] = False
        assert np.allclose(d[off], (1 - eps) / (L * B), rtol=1e-14)
        assert np.allclose(d[~off], -(1 - eps) * (L - 1) / (L * B), rtol=1e-14)
    # a confident correct prediction: with eps = 0 the loss tends to 0, with
    # eps > 0 it tends to eps (L-1)/L times the logit gap
    gap = 40.0
    lg = np.array([[gap, 0.0, 0.0, 0.0]])
    assert softmax_xent(lg, np.array([0]), 0.0)[0] < 1e-15
    want = 0.2 * 3 / 4 * gap
    assert softmax_xent(lg, np.array([0]), 0.2)[0] == pytest.approx(want, rel=1e-12)


# ------------------------------------------------- whole-step pins (fp64)

def _batch(cfg, B=None, seed=0):
    images, labels, _ = make_dataset(cfg)
    rng = np.random.default_rng(seed)
    idx = rng.choice(len(labels), size=B or cfg["B"], replace=False)
    return images[idx].astype(np.float64), labels[idx].astype(np.int64)


class _RoundFwd(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x):
        return torch.from_numpy(round_bf16(x.detach().numpy()))

    @staticmethod
    def backward(ctx, g):
        return g


class _RoundBwd(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x):
        return x.clone()

    @staticmethod
    def backward(ctx, g):
        return torch.from_numpy(round_bf16(g.detach().numpy()))


def torch_split_model_loss(cfg, theta, x, y, with_running=False):
    """Loss and gradient of the unsplit CNN via torch.autograd in fp64.

    bf16 workloads insert rounding nodes at the documented points: forward
    rounding of inputs, weights, conv outputs and the pooled feature;
    backward rounding of each conv's pre-activation gradient and of the
    gradient a conv returns for its input.  Norm layers are torch's
    batch_norm (training mode, momentum 0.1) and group_norm, eps 1e-5; a
    conv followed by one has no ReLU and the norm's pre-ReLU gradient is
    rounded instead."""
    bf16 = cfg["dtype"] == "bf16"
    rf = _RoundFwd.apply if bf16 else (lambda t: t)
    rb = _RoundBwd.apply if bf16 else (lambda t: t)
    th = torch.tensor(np.asarray(theta, dtype=np.float64), requires_grad=True)
    views = {}
    for i, tag, shp, off in param_layout(cfg):
        n = int(np.prod(shp))
        views.setdefault(i, {})[tag] = th[off:off + n].reshape(shp)
    a = rf(torch.tensor(x).permute(0, 3, 1, 2))
    layers = cfg["layers"]
    running = {}
    for i, spec in enumerate(layers):
        if spec[0] == "conv":
            a_in = rb(a) if i > 0 and layers[i - 1][0] not in ("bnorm", "gnorm") else a
            w = rf(views[i]["w"]).permute(0, 3, 1, 2)
            pre = tF.conv2d(a_in, w, views[i]["b"], padding=1)
            if spec[3]:
                pre = pre + a_in
            if i + 1 < len(layers) and layers[i + 1][0] in ("bnorm", "gnorm"):
                a = rf(rb(pre))  # raw output, normalised next
            else:
                a = rf(torch.relu(rb(pre)))
        elif spec[0] == "bnorm":
            rm = torch.zeros(spec[1], dtype=torch.float64)
            rv = torch.ones(spec[1], dtype=torch.float64)
            u = tF.batch_norm(a, rm, rv, views[i]["w"], views[i]["b"], training=True, momentum=0.1, eps=1e-5)
            running[i] = (rm, rv)
            a = rf(torch.relu(rb(u)))
        elif spec[0] == "gnorm":
            u = tF.group_norm(a, spec[2], views[i]["w"], views[i]["b"], eps=1e-5)
            a = rf(torch.relu(rb(u)))
        elif spec[0] == "block":
            _, cin, cout, stride, groups = spec
            v = views[i]

            def norm(t, sub, v=v, i=i, groups=groups, cout=cout):
                if groups:
                    return tF.group_norm(t, groups, v[sub + "w"], v[sub + "b"], eps=1e-5)
                rm = torch.zeros(cout, dtype=torch.float64)
                rv = torch.ones(cout, dtype=torch.float64)
                running[(i, sub)] = (rm, rv)
                return tF.batch_norm(t, rm, rv, v[sub + "w"], v[sub + "b"], training=True, momentum=0.1, eps=1e-5)

            x_in = rb(a)  # the block's input gradient (main + shortcut) is rounded
            z1 = rf(rb(tF.conv2d(x_in, rf(v["w1"]).permute(0, 3, 1, 2), v["b1"], stride=stride, padding=1)))
            a1 = rf(torch.relu(rb(norm(z1, "n1"))))
            z2 = rf(rb(tF.conv2d(a1, rf(v["w2"]).permute(0, 3, 1, 2), v["b2"], padding=1)))
            if "wp" in v:
                zp = rf(rb(tF.conv2d(rb(x_in), rf(v["wp"]).permute(0, 3, 1, 2), v["bp"], stride=stride)))
                sc = rf(norm(zp, "np"))
            else:
                sc = x_in
            a = rf(torch.relu(rb(norm(z2, "n2") + sc)))
        elif spec[0] == "maxpool":
            a = tF.max_pool2d(a, 2)
        elif spec[0] == "avgpool":
            a = rf(a.mean(dim=(2, 3)))
        elif spec[0] == "linear":
            a = a @ rf(views[i]["w"]).T + views[i]["b"]
    loss = tF.cross_entropy(a, torch.tensor(y), label_smoothing=cfg.get("label_smoothing", 0.0))
    loss.backward()
    if with_running:
        return loss.item(), th.grad.numpy(), {i: (m.numpy(), v.numpy()) for i, (m, v) in running.items()}
    return loss.item(), th.grad.numpy()


@pytest.mark.parametrize("name", ["tiny", "ragged", "ragged_bf16", "tiny_norm", "ragged_norm_bf16", "tiny_recipe",
                                  "ragged_recipe_bf16", "resnet_tiny", "resnet_tiny_bf16"])
def test_split_step_matches_torch_autograd(name):
    cfg = get_config(name)
    theta = init_params(cfg)
    x, y = _batch(cfg)
    loss, grad, _ = split_forward_backward(cfg, theta, x, y)
    tloss, tgrad = torch_split_model_loss(cfg, theta, x, y)
    assert loss == pytest.approx(tloss, rel=1e-12)
    # absolute floor at the gradient's overall scale: the bias of a conv that
    # feeds a BatchNorm has an exactly zero gradient (the batch mean removes
    # it), which both sides produce as rounding noise
    scale = np.abs(tgrad).max()
    for i, tag, shp, off in param_layout(cfg):
        n = int(np.prod(shp))
        a, b = grad[off:off + n], tgrad[off:off + n]
        assert np.allclose(a, b, rtol=1e-9, atol=1e-12 * max(np.abs(b).max(), 1e-3 * scale)), (i, tag)


def test_split_step_matches_torch_autograd_wide_residual_server():
    # the 16-cluster server stack (64->256, three residual 256->256) on a
    # reduced batch and image size
    cfg = get_config("gcpsl16", dtype="f32", H=8, W=8, N_ex=200, B=4)
    theta = init_params(cfg)
    x, y = _batch(cfg)
    loss, grad, _ = split_forward_backward(cfg, theta, x, y)
    tloss, tgrad = torch_split_model_loss(cfg, theta, x, y)
    assert loss == pytest.approx(tloss, rel=1e-12)
    assert np.allclose(grad, tgrad, rtol=1e-9, atol=1e-12 * np.abs(tgrad).max())


def test_split_step_finite_differences():
    cfg = get_config("tiny")
    theta = init_params(cfg).astype(np.float64)
    x, y = _batch(cfg, seed=5)
    loss, grad, rec = split_forward_backward(cfg, theta, x, y, keep=True)
    # guard: no ReLU pre-activation and no max-pool runner-up within reach of
    # the perturbation, so the loss is smooth around theta
    for key, v in rec.items():
        if key.startswith("pre"):
            assert np.abs(v).min() > 1e-6, key
    for i, spec in enumerate(cfg["layers"]):
        if spec[0] == "maxpool":
            a = rec["acts"][i]
            Bt, H, W, C = a.shape
            win = np.sort(a.reshape(Bt, H // 2, 2, W // 2, 2, C).transpose(0, 1, 3, 5, 2, 4)
                          .reshape(-1, 4), axis=1)
            live = win[:, 3] > 0
            assert (win[live, 3] - win[live, 2]).min() > 1e-6
    rng = np.random.default_rng(0)
    coords = rng.choice(len(theta), size=60, replace=False)
    h = 1e-6
    for j in coords:
        tp, tm = theta.copy(), theta.copy()
        tp[j] += h
        tm[j] -= h
        fd = (split_forward_backward(cfg, tp, x, y)[0] - split_forward_backward(cfg, tm, x, y)[0]) / (2 * h)
        assert abs(fd - grad[j]) <= 1e-8 + 1e-6 * abs(grad[j]), (j, fd, grad[j])


@pytest.mark.parametrize("name", ["tiny_norm", "ragged_norm_bf16", "resnet_tiny"])
def test_batchnorm_running_statistics_match_torch(name):
    # one round's running mean / variance update (Sec. IV-B normalisation
    # state) against torch's buffers after one training-mode batch_norm
    from gcpsl_inputs import norm_layout
    from oracle.model import bn_running_update
    cfg = get_config(name)
    theta = init_params(cfg)
    x, y = _batch(cfg)
    _, _, rec = split_forward_backward(cfg, theta, x, y)
    _, _, running = torch_split_model_loss(cfg, theta, x, y, with_running=True)
    assert sorted(rec["bn_batch"], key=str) == sorted(running, key=str)
    for i, (mean, var, n) in rec["bn_batch"].items():
        ch = len(mean)
        rm, rv, cnt = bn_running_update(np.zeros(ch), np.ones(ch), 0.0, mean, var, n)
        assert np.allclose(rm, running[i][0], rtol=1e-12, atol=1e-15)
        assert np.allclose(rv, running[i][1], rtol=1e-12)
        assert cnt == 1.0
    assert [t for _, t, _, _ in norm_layout(cfg)] == ["mean", "var", "count"] * len(running)


def test_norm_closed_forms():
    # batch norm of a constant-shifted, scaled tensor: x_hat is the
    # standardised tensor whatever the shift and scale; group norm with one
    # channel per group and H = W = 1 gives zero (each set has one value)
    from oracle.model import norm_forward
    rng = np.random.default_rng(4)
    z = rng.standard_normal((3, 4, 5, 6))
    _, xh1, _, _, _ = norm_forward(z, np.ones(6), np.zeros(6))
    _, xh2, _, _, _ = norm_forward(7.0 * z - 3.0, np.ones(6), np.zeros(6))
    assert np.allclose(xh1, xh2, atol=1e-4)  # eps = 1e-5 sets the small difference
    assert np.allclose(xh1.mean(axis=(0, 1, 2)), 0.0, atol=1e-12)
    assert np.allclose((xh1 ** 2).mean(axis=(0, 1, 2)), 1.0 / (1.0 + 1e-5 / z.var(axis=(0, 1, 2))), rtol=1e-12)
    u, _, _, _, _ = norm_forward(rng.standard_normal((2, 1, 1, 6)), np.full(6, 2.0), np.full(6, 0.5), groups=6)
    assert np.allclose(u, 0.5)  # x_hat = 0, so u = beta


def test_split_step_finite_differences_with_norm_layers():
    cfg = get_config("tiny_norm")
    theta = init_params(cfg).astype(np.float64)
    theta += np.random.default_rng(1).uniform(-0.1, 0.1, theta.shape)  # gamma, beta off their init
    x, y = _batch(cfg, seed=5)
    loss, grad, rec = split_forward_backward(cfg, theta, x, y, keep=True)
    for i, spec in enumerate(cfg["layers"]):
        if spec[0] in ("bnorm", "gnorm"):  # no ReLU kink within reach
            assert np.abs(rec[f"pre{i}"]).min() > 1e-6
        if spec[0] == "maxpool":
            a = rec["acts"][i]
            Bt, H, W, C = a.shape
            win = np.sort(a.reshape(Bt, H // 2, 2, W // 2, 2, C).transpose(0, 1, 3, 5, 2, 4)
                          .reshape(-1, 4), axis=1)
            live = win[:, 3] > 0
            assert (win[live, 3] - win[live, 2]).min() > 1e-6
    rng = np.random.default_rng(0)
    coords = rng.choice(len(theta), size=60, replace=False)
    h = 1e-6
    for j in coords:
        tp, tm = theta.copy(), theta.copy()
        tp[j] += h
        tm[j] -= h
        fd = (split_forward_backward(cfg, tp, x, y)[0] - split_forward_backward(cfg, tm, x, y)[0]) / (2 * h)
        assert abs(fd - grad[j]) <= 1e-8 + 1e-6 * abs(grad[j]), (j, fd, grad[j])


def test_choose_with_own_decisions_changes_nothing():
    # a decision callback that returns the oracle's own decisions reproduces
    # the plain pass bit for bit (every ReLU and max-pool decision consulted)
    for name in ("ragged_bf16", "tiny_norm"):
        cfg = get_config(name)
        theta = init_params(cfg)
        x, y = _batch(cfg)
        seen = []

        def own(kind, i, decision, values):
            seen.append((kind, i))
            return decision

        l0, g0, r0 = split_forward_backward(cfg, theta, x, y, keep=True)
        l1, g1, r1 = split_forward_backward(cfg, theta, x, y, keep=True, choose=own)
        assert l0 == l1 and np.array_equal(g0, g1)
        for a, b in zip(r0["acts"], r1["acts"]):
            assert np.array_equal(a, b)
        relus = [i for i, sp in enumerate(cfg["layers"])
                 if sp[0] in ("bnorm", "gnorm") or (sp[0] == "conv" and not (
                     i + 1 < len(cfg["layers"]) and cfg["layers"][i + 1][0] in ("bnorm", "gnorm")))]
        pools = [i for i, sp in enumerate(cfg["layers"]) if sp[0] == "maxpool"]
        assert sorted(seen) == sorted([("relu", i) for i in relus] + [("pool", i) for i in pools])


def test_forced_decisions_give_the_gradient_of_the_fixed_decision_network():
    # With every ReLU mask and max-pool index fixed (here: the pass's own
    # decisions at theta with about 5 % of them overturned at random), the
    # pass is a smooth function of theta, and its gradient must be the
    # derivative of that function: central finite differences in fp64, with
    # the same fixed decisions at theta +- h.
    cfg = get_config("tiny")
    theta = init_params(cfg).astype(np.float64)
    x, y = _batch(cfg, seed=5)
    rng = np.random.default_rng(11)
    fixed = {}

    def record(kind, i, decision, values):
        d = decision.copy()
        flip = rng.random(d.shape) < 0.05
        if kind == "relu":
            d[flip] = ~d[flip]
        else:
            d[flip] = (d[flip] + 1 + rng.integers(0, 3, size=int(flip.sum()))) % 4
        fixed[(kind, i)] = d
        return d

    loss, grad, _ = split_forward_backward(cfg, theta, x, y, choose=record)

    def replay(kind, i, decision, values):
        return fixed[(kind, i)]

    assert split_forward_backward(cfg, theta, x, y, choose=replay)[0] == loss
    plain = split_forward_backward(cfg, theta, x, y)[1]
    assert not np.allclose(plain, grad, rtol=1e-3)  # the overturned decisions matter
    coords = rng.choice(len(theta), size=60, replace=False)
    h = 1e-6
    for j in coords:
        tp, tm = theta.copy(), theta.copy()
        tp[j] += h
        tm[j] -= h
        fd = (split_forward_backward(cfg, tp, x, y, choose=replay)[0]
              - split_forward_backward(cfg, tm, x, y, choose=replay)[0]) / (2 * h)
        assert abs(fd - grad[j]) <= 1e-8 + 1e-6 * abs(grad[j]), (j, fd, grad[j])


def test_resnet_block_finite_differences_and_decisions():
    # the ResNet-shaped model (every block kind): with its discrete decisions
    # fixed, the gradient is the derivative of the loss (central differences,
    # fp64); both ReLUs of every block are consulted, the inner one under
    # the key (layer, "n1")
    cfg = get_config("resnet_tiny")
    theta = init_params(cfg).astype(np.float64)
    x, y = _batch(cfg, seed=3)
    fixed = {}

    def record(kind, i, decision, values):
        fixed[(kind, i)] = decision.copy()
        return decision

    loss, grad, _ = split_forward_backward(cfg, theta, x, y, choose=record)
    blocks = [i for i, sp in enumerate(cfg["layers"]) if sp[0] == "block"]
    assert {k for k in fixed if isinstance(k[1], tuple)} == {("relu", (i, "n1")) for i in blocks}
    assert all(("relu", i) in fixed for i in blocks)

    def replay(kind, i, decision, values):
        return fixed[(kind, i)]

    rng = np.random.default_rng(4)
    coords = rng.choice(len(theta), size=50, replace=False)
    h = 1e-6
    for j in coords:
        tp, tm = theta.copy(), theta.copy()
        tp[j] += h
        tm[j] -= h
        fd = (split_forward_backward(cfg, tp, x, y, choose=replay)[0]
              - split_forward_backward(cfg, tm, x, y, choose=replay)[0]) / (2 * h)
        assert abs(fd - grad[j]) <= 1e-8 + 1e-6 * abs(grad[j]), (j, fd, grad[j])


def test_strided_conv_matches_explicit_loops():
    # stride 2, 3x3 pad 1 and 1x1 pad 0, forward and backward, against the
    # definition written as loops on a tiny tensor
    from oracle.model import conv_backward, conv_forward
    rng = np.random.default_rng(9)
    x = rng.standard_normal((2, 6, 6, 3))
    for R, pad in ((3, 1), (1, 0)):
        w = rng.standard_normal((4, R, R, 3))
        b = rng.standard_normal(4)
        out = conv_forward(x, w, b, 2, pad)
        Ho = (6 + 2 * pad - R) // 2 + 1
        assert out.shape == (2, Ho, Ho, 4)
        want = np.zeros_like(out)
        for n in range(2):
            for ho in range(Ho):
                for wo in range(Ho):
                    for o in range(4):
                        acc = b[o]
                        for r in range(R):
                            for s_ in range(R):
                                hh, ww = 2 * ho + r - pad, 2 * wo + s_ - pad
                                if 0 <= hh < 6 and 0 <= ww < 6:
                                    acc += x[n, hh, ww] @ w[o, r, s_]
                        want[n, ho, wo, o] = acc
        assert np.allclose(out, want, rtol=1e-13, atol=1e-13)
        gp = rng.standard_normal(out.shape)
        dx, dw, db = conv_backward(x, w, gp, 2, pad)
        # the gradient of sum(out * gp) is linear: check it against the loops
        dx_want = np.zeros_like(x)
        dw_want = np.zeros_like(w)
        for n in range(2):
            for ho in range(Ho):
                for wo in range(Ho):
                    for r in range(R):
                        for s_ in range(R):
                            hh, ww = 2 * ho + r - pad, 2 * wo + s_ - pad
                            if 0 <= hh < 6 and 0 <= ww < 6:
                                dx_want[n, hh, ww] += gp[n, ho, wo] @ w[:, r, s_]
                                dw_want[:, r, s_] += np.outer(gp[n, ho, wo], x[n, hh, ww])
        assert np.allclose(dx, dx_want, rtol=1e-12, atol=1e-12)
        assert np.allclose(dw, dw_want, rtol=1e-12, atol=1e-12)
        assert np.allclose(db, gp.sum(axis=(0, 1, 2)), rtol=1e-12)
