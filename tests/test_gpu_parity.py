"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Bar: bit-exact on sampled indices, labels, gathered inputs (as values),
cluster assignments, participation counts and fusion of given replicas;
floating point within tol = 1e-4 (fp32 workloads) or 2e-2 (bf16 workloads),
tested per tensor as ||a - b||_2 <= tol ||b||_2 and max|a - b| <= tol max|b|,
and elementwise relative for the per-cluster losses.
"""
import numpy as np
import pytest
import torch

from gcpsl_inputs import param_layout, client_stats, get_config, init_params, make_dataset
from oracle.model import im2col3x3, round_bf16, split_forward_backward
from oracle.sampler import active_clients, batch_indices, cluster_examples
from oracle.train import GCPSLOracle, fuse as oracle_fuse

pytestmark = pytest.mark.gpu

from paper_2609_29395_amd import driver, gcpsl  # noqa: E402

TOL = {"f32": 1e-4, "bf16": 2e-2}


def close(a, b, tol):
    a = np.asarray(a, dtype=np.float64).ravel()
    b = np.asarray(b, dtype=np.float64).ravel()
    assert a.shape == b.shape, (a.shape, b.shape)
    nb = np.linalg.norm(b)
    err = np.linalg.norm(a - b)
    mx = np.abs(b).max() if b.size else 0.0
    ok = err <= tol * nb + 1e-30 and np.abs(a - b).max() <= tol * mx + 1e-30
    return ok, (err / (nb + 1e-30), np.abs(a - b).max() / (mx + 1e-30))


def kink_sensitive(cfg):
    """bf16 workloads with norm layers: a norm centres its output at zero, so
    the ReLU after it cuts at the mode of the distribution and a one-ulp
    difference upstream (fp32 kernels against the fp64 oracle) flips its
    decision for ~0.1 % of the values; each flip changes that gradient entry
    completely and the norm's backward spreads it over the channel.  Losses,
    parameters, normalisation state, forward activations and the parameter
    gradient stay within the bf16 bar; the per-element backward tensors and
    the momentum (the accumulated gradients) are held to the flip check
    below instead.  The same holds for the 16 x 16 residual workload without
    a max pool: its top conv feeds the average pool, which hands every pixel
    of a channel the same gradient, and one ReLU decision at a pre-activation
    within bf16 rounding of zero moves a full-size entry of that layer's
    gradient (0.4 % in norm, 52 % of the maximum at one element of one
    replica, propagating with shrinking size into the layers below).  With a
    2 x 2 max pool between the top conv and the average pool, a window whose
    two largest values are within bf16 rounding of each other can also route
    its gradient to the other pixel (measured: 0.6 % in norm, 2.9 % of the
    maximum in the first layer's gradient of one replica)."""
    norm = any(sp[0] in ("bnorm", "gnorm") for sp in cfg["layers"])
    return cfg["dtype"] == "bf16" and (norm or cfg["name"] in ("halo_res_bf16", "halo_split_bf16",
                                                              "halo_maxhead_bf16"))


def relu_flips_are_near_kinks(act_gpu, act_ref, pre_ref, rel=1e-2):
    """Every ReLU decision where GPU and oracle differ is at a pre-activation
    within rel of the tensor's largest magnitude of zero; returns the count."""
    diff = (np.asarray(act_gpu).ravel() > 0) != (np.asarray(act_ref).ravel() > 0)
    pre = np.asarray(pre_ref).ravel()
    bad = np.abs(pre[diff.ravel()]) > rel * np.abs(pre).max()
    assert not bad.any(), (int(bad.sum()), pre[diff.ravel()][bad][:5])
    return int(diff.sum())


def _np(t):
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy()


# ---------------------------------------------------------------- sampling

@pytest.mark.parametrize("name,window,starts", [
    ("tiny", 4, [0, 20, 97]),
    ("ragged", 3, [0, 21, 500]),
    ("gcpsl4", 2, [0, 195, 196]),
    ("gcpsl16", 2, [0, 1, 87, 999]),
])
def test_sample_and_gather_bit_exact(name, window, starts):
    cfg = get_config(name)
    images, labels, coe = make_dataset(cfg)
    ctx, assignment = driver.setup(cfg, max_steps=1000, max_window=window)
    ids = cluster_examples(coe, assignment, cfg["C"])
    assert ctx.cluster_sizes().tolist() == [len(x) for x in ids]
    C, B = cfg["C"], cfg["B"]
    out = torch.zeros(window, C, B, dtype=torch.int32, device="cuda")
    for s0 in starts:
        ctx.sample(s0, window, out)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        ys = _np(ctx.tensor("y")).reshape(-1, C, B)
        H, W, Cin = cfg["H"], cfg["W"], cfg["Cin"]
        vec = 8 if cfg["dtype"] == "bf16" else 4
        kc = Cin if Cin % vec == 0 else -(-9 * Cin // vec) * vec
        xs = _np(ctx.tensor("x")).reshape(-1, C, B, H, W, kc)
        for j in range(window):
            for n in range(C):
                want = batch_indices(ids[n], B, cfg["seed"], n, s0 + j)
                assert np.array_equal(got[j, n], want), (s0, j, n)
                assert np.array_equal(ys[j, n], labels[want])
                ref = images[want].astype(np.float64)
                if cfg["dtype"] == "bf16":
                    ref = round_bf16(ref)
                if kc != Cin:  # staged as im2col rows of the image layer
                    ref = np.concatenate([im2col3x3(ref).reshape(B, H, W, 9 * Cin),
                                          np.zeros((B, H, W, kc - 9 * Cin))], axis=3)
                assert np.array_equal(xs[j, n].astype(np.float64), ref)
    # per-step |A_{n,t}| of every sampled step
    hits = _np(ctx.tensor("hits")).reshape(-1, C)
    for s0 in starts:
        for j in range(window):
            if s0 + j >= hits.shape[0]:
                continue  # beyond max_steps: not recorded
            for n in range(C):
                want = active_clients(batch_indices(ids[n], B, cfg["seed"], n, s0 + j), coe)
                assert hits[s0 + j, n] == want


# ------------------------------------------------------- multi-step runs

@pytest.mark.parametrize("name", ["tiny", "tiny_jsd", "ragged", "ragged_bf16", "ragged_res_bf16", "tiny_norm",
                                  "ragged_norm_bf16", "tiny_recipe", "ragged_recipe_bf16", "halo_res_bf16",
                                  "halo_split_bf16", "img32_bf16", "col_ragged_bf16", "wide_head_bf16",
                                  "halo_maxhead_bf16"])
def test_run_parity_with_fusion(name):
    cfg = get_config(name)
    T = cfg["T"]
    ctx, assignment = driver.setup(cfg)
    losses = torch.zeros(T, cfg["C"], device="cuda")
    driver.train(ctx, T, losses=losses)
    torch.cuda.synchronize()
    ref = GCPSLOracle(cfg, cluster_of_client=assignment).run(T)
    tol = TOL[cfg["dtype"]]
    got_l, want_l = losses.cpu().numpy(), np.array(ref.losses)
    assert np.all(np.abs(got_l - want_l) <= tol * np.abs(want_l)), (got_l, want_l)
    th, mo = ctx.theta.cpu().numpy(), ctx.mom.cpu().numpy()
    for n in range(cfg["C"]):
        ok, e = close(th[n], ref.theta[n], tol)
        assert ok, ("theta", n, e)
        if not kink_sensitive(cfg):
            ok, e = close(mo[n], ref.mom[n], tol)
            assert ok, ("momentum", n, e)
        if ctx.S:  # batch-norm running statistics, fused with the parameters
            ok, e = close(ctx.norm_state[n].cpu().numpy(), ref.norm[n], tol)
            assert ok, ("norm state", n, e)
    a, t, per = ctx.participation()
    assert t == cfg["K"] * T
    assert np.array_equal(per, np.array(ref.active)) and a == int(np.sum(ref.active))


@pytest.mark.parametrize("name", ["ragged", "ragged_bf16", "ragged_res_bf16", "tiny", "tiny_norm", "ragged_norm_bf16",
                                  "tiny_recipe", "ragged_recipe_bf16", "halo_res_bf16", "halo_split_bf16",
                                  "img32_bf16", "col_ragged_bf16", "wide_head_bf16", "halo_maxhead_bf16"])
def test_intermediates_one_round(name):
    cfg = get_config(name)
    ctx, assignment = driver.setup(cfg)
    ctx.sample(0)
    loss = torch.zeros(cfg["C"], device="cuda")
    ctx.step(0, loss)
    torch.cuda.synchronize()
    o = GCPSLOracle(cfg, cluster_of_client=assignment)
    tol = TOL[cfg["dtype"]]
    C = cfg["C"]
    grads = _np(ctx.tensor("grad")).reshape(C, -1)
    for n in range(C):
        idx, x, y = o.batch(0, n)
        l, g, rec = split_forward_backward(cfg, o.theta[n], x, y, keep=True)
        assert abs(loss[n].item() - l) <= tol * abs(l)
        for i, spec in enumerate(cfg["layers"]):
            name_i = f"act{i}"
            try:
                t = _np(ctx.tensor(name_i)).reshape(C, -1)[n]
            except gcpsl.GCPSLError:
                t = None
            if t is not None and spec[0] != "linear":
                ok, e = close(t, rec["acts"][i + 1], tol)
                assert ok, (name_i, n, e)
            if kink_sensitive(cfg):
                relu_after = spec[0] in ("bnorm", "gnorm") or (
                    spec[0] == "conv" and not (i + 1 < len(cfg["layers"]) and cfg["layers"][i + 1][0] in ("bnorm", "gnorm")))
                if relu_after and t is not None:
                    relu_flips_are_near_kinks(t, rec["acts"][i + 1], rec[f"pre{i}"])
                continue
            if spec[0] in ("conv", "bnorm", "gnorm"):
                ok, e = close(_np(ctx.tensor(f"gpre{i}")).reshape(C, -1)[n], rec[f"gpre{i}"], tol)
                assert ok, (f"gpre{i}", n, e)
                if i > 0 and cfg["layers"][i - 1][0] == "maxpool":
                    ok, e = close(_np(ctx.tensor(f"gin{i}")).reshape(C, -1)[n], rec[f"gin{i}"], tol)
                    assert ok, (f"gin{i}", n, e)
        ok, e = close(grads[n], g, tol)
        assert ok, ("grad", n, e)


@pytest.mark.parametrize("term", [dict(weight_decay=0.05), dict(nesterov=True), dict(label_smoothing=0.3),
                                  dict(weight_decay=0.05, nesterov=True, label_smoothing=0.3)])
def test_recipe_terms_each_change_the_run(term):
    """Each term of the training recipe (Sec. V-A) on its own, at a strength
    that moves the parameters well beyond the parity bar: the GPU run matches
    the oracle run with the term, and differs from the GPU run without it."""
    base = dict(momentum=0.9, nesterov=False, weight_decay=0.0, label_smoothing=0.0)
    runs = {}
    for key, over in (("with", dict(base, **term)), ("without", base)):
        cfg = get_config("tiny", **over)
        ctx, assignment = driver.setup(cfg)
        losses = torch.zeros(cfg["T"], cfg["C"], device="cuda")
        driver.train(ctx, cfg["T"], losses=losses)
        torch.cuda.synchronize()
        runs[key] = (ctx.theta.cpu().numpy(), losses.cpu().numpy(), cfg, assignment)
    th, lo, cfg, assignment = runs["with"]
    ref = GCPSLOracle(cfg, cluster_of_client=assignment).run(cfg["T"])
    tol = TOL["f32"]
    assert np.all(np.abs(lo - np.array(ref.losses)) <= tol * np.abs(np.array(ref.losses)))
    for n in range(cfg["C"]):
        ok, e = close(th[n], ref.theta[n], tol)
        assert ok, ("theta", n, e)
        ok, e = close(runs["without"][0][n], ref.theta[n], tol)
        assert not ok, ("the term left theta unchanged", n, e)


# ------------------------------------------------------------------ fusion

def test_fusion_bit_exact_against_oracle_on_given_replicas():
    cfg = get_config("ragged")
    ctx, assignment = driver.setup(cfg)
    driver.train(ctx, 3, F=0)
    torch.cuda.synchronize()
    before = ctx.theta.cpu().numpy()
    assert not np.array_equal(before[0], before[1])
    ctx.fuse()
    torch.cuda.synchronize()
    after = ctx.theta.cpu().numpy()
    want = oracle_fuse(list(before), ctx.cluster_sizes().tolist())
    for n in range(cfg["C"]):
        assert np.array_equal(after[n], want)
    assert not np.array_equal(ctx.mom[0].cpu().numpy(), ctx.mom[1].cpu().numpy())


def test_fusion_of_identical_replicas_is_identity():
    cfg = get_config("gcpsl16")
    ctx, _ = driver.setup(cfg)
    before = ctx.theta.clone()
    ctx.fuse()
    torch.cuda.synchronize()
    assert torch.equal(ctx.theta, before)


@pytest.mark.parametrize("C,P", [(1, 1), (3, 7), (5, 1001), (4, 1002), (7, 1024), (16, 65538), (64, 333)])
def test_fuse_replicas_bit_exact_against_oracle(C, P):
    """gcpsl_fuse_replicas on caller-given replicas (every kernel width: P
    odd, P = 2 mod 4, P = 0 mod 4) and weights with zeros among them."""
    rng = np.random.default_rng(C * 1000 + P)
    th = (rng.standard_normal((C, P)) * np.exp(rng.uniform(-8, 8, (C, P)))).astype(np.float32)
    w = rng.integers(0, 60000, size=C)
    w[rng.random(C) < 0.2] = 0
    if w.sum() == 0:
        w[0] = 1
    t = torch.tensor(th, device="cuda")
    gcpsl.fuse_replicas(t, w)
    torch.cuda.synchronize()
    want = oracle_fuse(list(th), w.tolist())
    got = t.cpu().numpy()
    for n in range(C):
        assert np.array_equal(got[n], want), n


def test_fuse_replicas_large_sampled_and_identity():
    """The 16-replica, 16M-parameter fusion timed by the benchmark: sampled
    columns against the oracle (fusion is column by column), and identical
    replicas come back unchanged."""
    C, P = 16, 16 * 1024 * 1024 + 2
    g = torch.Generator(device="cuda").manual_seed(5)
    t = torch.randn(C, P, device="cuda", generator=g)
    w = np.arange(1, C + 1, dtype=np.int64) * 3001
    cols = np.sort(np.random.default_rng(6).choice(P, size=4096, replace=False))
    cols = np.concatenate([[0, 1, P - 2, P - 1], cols])
    before = t[:, torch.tensor(cols, device="cuda")].cpu().numpy()
    gcpsl.fuse_replicas(t, w)
    torch.cuda.synchronize()
    after = t[:, torch.tensor(cols, device="cuda")].cpu().numpy()
    want = oracle_fuse(list(before), w.tolist())
    for n in range(C):
        assert np.array_equal(after[n], want), n
    same = t[:1].expand(C, -1).contiguous()
    ref = same[0].clone()
    gcpsl.fuse_replicas(same, w)
    torch.cuda.synchronize()
    assert torch.equal(same, ref.expand(C, -1))


# ------------------------------------------------ full sizes, sampled outputs

def _windows(a, shape):
    Bt, H, W, Ch = shape
    return (np.asarray(a).reshape(Bt, H // 2, 2, W // 2, 2, Ch).transpose(0, 1, 3, 5, 2, 4)
            .reshape(-1, 4))


def routing_flips(act_ref, gpre_gpu, gpre_ref, shape, tie):
    """Windows where the GPU routes a max-pool gradient to another pixel than
    the oracle.  Where rounding decides between two pixels whose values are
    within (rel, abs) = tie of each other -- rel of the window maximum, abs of
    the tensor's largest value, since a one-ulp difference in an upstream
    input moves every later value by an amount set by that scale -- both
    choices are correct; any other difference is a bug.  Returns the number
    of (valid) flips."""
    rel, absolute = tie
    A = _windows(act_ref, shape)
    G = _windows(gpre_gpu, shape) != 0
    R = _windows(gpre_ref, shape) != 0
    bad = np.flatnonzero((G != R).any(axis=1))
    scale = np.abs(A).max()
    for w in bad:
        top = A[w].max()
        chosen = np.flatnonzero(G[w] | R[w])
        # every pixel either side picked is (within rounding) a maximum of its
        # window, or a ReLU-clamped value near zero
        assert np.all(top - A[w][chosen] <= rel * abs(top) + absolute * scale), \
            (w, A[w], G[w], R[w])
    return len(bad)


@pytest.mark.parametrize("name", ["gpsl", "gcpsl4", "gcpsl8", "gcpsl16"])
def test_full_size_round_sampled_replicas(name):
    """One round at the workload's real size; replicas 0 and C-1 recomputed by
    the oracle.  Forward activations, loss and the updated parameters are held
    to the parity bar.  Gradients are held to it too unless a max-pool routing
    decision flipped at a near-tie (checked valid above); one such flip moves
    |dL/dz| / npos to a neighbouring pixel and was measured at 2e-4 relative on
    the 64-example gradient, so the gradient bound then widens to 5e-3 (fp32)."""
    cfg = get_config(name)
    ctx, assignment = driver.setup(cfg)
    C = cfg["C"]
    ctx.sample(0)
    loss = torch.zeros(C, device="cuda")
    ctx.step(0, loss)
    torch.cuda.synchronize()
    tol = TOL[cfg["dtype"]]
    # fp32: a few ulp (2^-23) of the window max plus 1e-6 of the scale;
    # bf16: one ulp is 2^-8 = 3.9e-3, so 2e-2 of the max and 1e-3 of the scale
    tie = (1e-5, 1e-6) if cfg["dtype"] == "f32" else (2e-2, 1e-3)
    o = GCPSLOracle(cfg, cluster_of_client=assignment)
    grads = _np(ctx.tensor("grad")).reshape(C, -1)
    th = ctx.theta.cpu().numpy()
    layers = cfg["layers"]
    for n in sorted({0, C - 1}):
        idx, x, y = o.batch(0, n)
        l, g, rec = split_forward_backward(cfg, o.theta[n], x, y, keep=True)
        assert abs(loss[n].item() - l) <= tol * abs(l), (n, loss[n].item(), l)
        flips = 0
        for i, spec in enumerate(layers):
            if spec[0] != "conv":
                continue
            act = _np(ctx.tensor(f"act{i}")).reshape(C, -1)[n]
            ok, e = close(act, rec["acts"][i + 1], tol)
            assert ok, (f"act{i}", n, e)
            if i + 1 < len(layers) and layers[i + 1][0] == "maxpool":
                shape = rec["acts"][i + 1].shape
                gp = _np(ctx.tensor(f"gpre{i}")).reshape(C, -1)[n]
                flips += routing_flips(rec["acts"][i + 1], gp, rec[f"gpre{i}"], shape, tie)
        gtol = tol if (flips == 0 or cfg["dtype"] == "bf16") else 5e-3
        ok, e = close(grads[n], g, gtol)
        assert ok, ("grad", n, flips, e)
        # and each layer's weight and bias gradient on its own (a mistake in
        # one layer's kernel cannot hide behind the others' magnitudes)
        for li, tag, shp, off in param_layout(cfg):
            size = int(np.prod(shp))
            ok, e = close(grads[n][off:off + size], g[off:off + size], gtol)
            assert ok, ("grad", li, tag, n, flips, e)
        want = o.theta[n].astype(np.float64) - cfg["lr"] * g
        ok, e = close(th[n], want, tol)
        assert ok, ("theta", n, e)
    # participation of the round, every cluster
    a, t, per = ctx.participation()
    coe = make_dataset(cfg)[2]
    ids = cluster_examples(coe, assignment, C)
    assert per.shape == (1, C)
    for n in range(C):
        assert per[0, n] == active_clients(batch_indices(ids[n], cfg["B"], cfg["seed"], n, 0), coe)


# ------------------------------------------------------ invariants, errors

def test_two_runs_are_bit_identical():
    cfg = get_config("ragged_bf16")
    outs = []
    for _ in range(2):
        ctx, _ = driver.setup(cfg)
        driver.train(ctx, 4)
        torch.cuda.synchronize()
        outs.append(ctx.theta.cpu().numpy())
    assert np.array_equal(outs[0], outs[1])


def test_state_errors():
    cfg = get_config("tiny")
    ctx, _ = driver.setup(cfg, max_window=2)
    with pytest.raises(gcpsl.GCPSLError) as e:
        ctx.step(0)
    assert e.value.code == gcpsl.ESTATE
    with pytest.raises(gcpsl.GCPSLError) as e:
        ctx.sample(0, 3)
    assert e.value.code == gcpsl.EINVAL
    ctx.sample(4, 2)
    with pytest.raises(gcpsl.GCPSLError) as e:
        ctx.step(6)
    assert e.value.code == gcpsl.ESTATE
    ctx.step(5)
    ctx.step(4)
    torch.cuda.synchronize()
    with pytest.raises(gcpsl.GCPSLError):
        ctx.tensor("nope")
