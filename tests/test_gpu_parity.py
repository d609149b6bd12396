"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Bar: bit-exact on sampled indices, labels, gathered inputs (as values),
cluster assignments, participation counts and fusion of given replicas;
floating point within tol = 1e-4 (fp32 workloads) or 2e-2 (bf16 workloads),
tested per tensor as ||a - b||_2 <= tol ||b||_2 and max|a - b| <= tol max|b|,
and elementwise relative for the per-cluster losses.  Every round's oracle
runs under the GPU's ReLU and max-pool decisions, each one that differs from
the oracle's own first checked to be a near-tie of the oracle's values
(gpu_match); no tensor is exempt from the comparison.
"""
import numpy as np
import pytest
import torch

from gcpsl_inputs import param_layout, client_stats, get_config, init_params, make_dataset
from oracle.model import im2col3x3, round_bf16, split_forward_backward
from oracle.sampler import active_clients, batch_indices, cluster_examples
from oracle.train import GCPSLOracle, fuse as oracle_fuse, sgd_args, sgd_update

from gpu_match import TOL, bar, deep_bf16, noisy_rounding, GpuChoices, LazyChoices, close, compare_params, layer_shapes, master_ulp, replayed, replica_tensor, routed_gradient, twin_bar
from gpu_match import to_np as _np

pytestmark = pytest.mark.gpu

from paper_2609_29395_amd import driver, gcpsl  # noqa: E402

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
        # staged as the images themselves (kc = Cin) or as the image layer's
        # im2col rows (kc = 9 Cin rounded up to the vector width)
        xt = _np(ctx.tensor("x"))
        kc = xt.size // (window * C * B * H * W)
        vec = 8 if cfg["dtype"] == "bf16" else 4
        assert kc in (Cin, -(-9 * Cin // vec) * vec), kc
        xs = xt.reshape(-1, C, B, H, W, kc)
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

def matched_run(cfg, T, F=None, log=None):
    """T rounds on the GPU, one at a time, fusing after every F-th; the oracle
    runs the same rounds under the GPU's validated decisions.  Returns the
    context, the oracle, the initial parameters, the GPU losses [T][C] and
    the number of decisions that differed."""
    F = cfg["F"] if F is None else F
    C = cfg["C"]
    ctx, assignment = driver.setup(cfg, max_steps=T)
    o = GCPSLOracle(cfg, cluster_of_client=assignment)
    # deep bf16 networks: a twin oracle under accumulation-order noise, which
    # calibrates the bar of the update and momentum comparisons (twin_bar)
    twin = GCPSLOracle(cfg, cluster_of_client=assignment) if deep_bf16(cfg) else None
    noise = noisy_rounding(seed=cfg["seed"] + 1)
    theta0 = ctx.theta[0].cpu().numpy().astype(np.float64)
    losses = torch.zeros(T, C, device="cuda")
    flips, worst = 0, 0.0
    for s in range(T):
        ctx.sample(s)
        ctx.step(s, losses[s])
        torch.cuda.synchronize()
        ch = LazyChoices(ctx, cfg)
        o.round(s, choose=ch)
        flips += sum(sum(c.flips.values()) for c in ch.values())
        worst = max([worst] + [c.worst for c in ch.values()])
        if twin is not None:
            with noise:
                twin.round(s, choose=replayed(ch))
        if F and (s + 1) % F == 0:
            ctx.fuse()
            o.fuse()
            if twin is not None:
                twin.fuse()
        if log:
            log(f"round {s + 1}/{T} done, {flips} decisions at near-ties so far "
                f"(largest distance {worst:.2e} of the tensor's scale)")
    o.twin = twin
    torch.cuda.synchronize()
    return ctx, o, theta0, losses.cpu().numpy(), flips


def check_run(ctx, o, theta0, losses, cfg):
    """Losses of every round (elementwise), then per replica the parameters,
    the update theta_T - theta_0 and the momentum, each layer's weight and bias
    on its own; the normalisation state; participation bit-exact."""
    tol = bar(cfg)
    T, F = len(losses), cfg["F"]
    fusions = T // F if F else 0
    want_l = np.array(o.losses)
    assert np.all(np.abs(losses - want_l) <= tol * np.abs(want_l)), (losses, want_l)
    th, mo = ctx.theta.cpu().numpy(), ctx.mom.cpu().numpy()
    twin = getattr(o, "twin", None)
    ulps = [master_ulp(o.theta[n], len(losses) + fusions) for n in range(cfg["C"])]
    tol_u = tol_m = tol
    if twin is not None:
        tol_u = twin_bar(tol, cfg, [(twin.theta[n] - theta0, o.theta[n] - theta0, ulps[n]) for n in range(cfg["C"])])
        tol_m = twin_bar(tol, cfg, [(twin.mom[n], o.mom[n], None) for n in range(cfg["C"])])
        print(f"bars calibrated by the twin oracle: update {tol_u:.3f}, momentum {tol_m:.3f}", flush=True)
    for n in range(cfg["C"]):
        ok, e = close(th[n], o.theta[n], tol)
        assert ok, ("theta", n, e)
        compare_params(th[n] - theta0, o.theta[n] - theta0, cfg, tol_u, ("update", n), ulp=ulps[n])
        compare_params(mo[n], o.mom[n], cfg, tol_m, ("momentum", n))
        if ctx.S:  # batch-norm running statistics, fused with the parameters
            ok, e = close(ctx.norm_state[n].cpu().numpy(), o.norm[n], tol)
            assert ok, ("norm state", n, e)
    a, t, per = ctx.participation()
    assert t == cfg["K"] * len(losses)
    assert np.array_equal(per, np.array(o.active)) and a == int(np.sum(o.active))
    check_metrics(ctx, o, cfg)


def check_metrics(ctx, o, cfg):
    """Sec. V-E metrics bit-exact: every batch's deviation numerator (-1 where
    a cluster drew none) and the logical payload by category."""
    sn, nb, den, per = ctx.batch_deviation()
    want = np.array(o.deviation, dtype=np.int64)
    assert np.array_equal(per, want), (per, want)
    assert den == cfg["B"] * sum(o.global_hist)
    assert sn == int(want[want >= 0].sum()) and nb == int((want >= 0).sum())
    assert ctx.payload() == o.payload, (ctx.payload(), o.payload)


@pytest.mark.parametrize("name", ["tiny", "tiny_jsd", "ragged", "ragged_bf16", "ragged_res_bf16", "tiny_norm",
                                  "ragged_norm_bf16", "tiny_recipe", "ragged_recipe_bf16", "halo_res_bf16",
                                  "halo_split_bf16", "img32_bf16", "col_ragged_bf16", "wide_head_bf16",
                                  "halo_maxhead_bf16", "halo128_bf16", "resnet_tiny", "resnet_tiny_bf16"])
def test_run_parity_with_fusion(name):
    cfg = get_config(name)
    ctx, o, theta0, losses, flips = matched_run(cfg, cfg["T"])
    print(f"{name}: {flips} decisions at near-ties", flush=True)
    check_run(ctx, o, theta0, losses, cfg)


@pytest.mark.parametrize("name", ["ragged", "ragged_bf16", "ragged_res_bf16", "tiny", "tiny_norm", "ragged_norm_bf16",
                                  "tiny_recipe", "ragged_recipe_bf16", "halo_res_bf16", "halo_split_bf16",
                                  "img32_bf16", "col_ragged_bf16", "wide_head_bf16", "halo_maxhead_bf16",
                                  "halo128_bf16", "resnet_tiny", "resnet_tiny_bf16"])
def test_intermediates_one_round(name):
    cfg = get_config(name)
    ctx, assignment = driver.setup(cfg)
    ctx.sample(0)
    loss = torch.zeros(cfg["C"], device="cuda")
    ctx.step(0, loss)
    torch.cuda.synchronize()
    o = GCPSLOracle(cfg, cluster_of_client=assignment)
    tol = bar(cfg)
    C = cfg["C"]
    layers = cfg["layers"]
    shapes = layer_shapes(cfg)
    grads = _np(ctx.tensor("grad")).reshape(C, -1)
    for n in range(C):
        idx, x, y = o.batch(0, n)
        ch = GpuChoices(ctx, cfg, n)
        l, g, rec = split_forward_backward(cfg, o.theta[n], x, y, keep=True, choose=ch)
        assert abs(loss[n].item() - l) <= tol * abs(l)
        for i, spec in enumerate(layers):
            if spec[0] != "linear":
                t = replica_tensor(ctx, f"act{i}", n, shapes[i])
                if t is not None:
                    ok, e = close(t, rec["acts"][i + 1], tol)
                    assert ok, (f"act{i}", n, e)
                else:  # unstored: a conv whose max pool keeps routing codes, or a pool fused into the head
                    assert i in ch.route or spec[0] == "maxpool", (i, spec)
            if spec[0] in ("conv", "bnorm", "gnorm", "block"):
                got = replica_tensor(ctx, f"gpre{i}", n, rec[f"gpre{i}"].shape)
                if got is None:
                    # the gradient the layer's kernels route from the next
                    # conv's input gradient through the codes
                    assert i in ch.route, i
                    gin = replica_tensor(ctx, f"gin{i + 2}", n, shapes[i + 1])
                    got = routed_gradient(gin, ch.route[i])
                got = got.reshape(-1)
                ok, e = close(got, rec[f"gpre{i}"], tol)
                assert ok, (f"gpre{i}", n, e)
            if spec[0] == "conv" and i > 0 and layers[i - 1][0] == "maxpool":
                ok, e = close(_np(ctx.tensor(f"gin{i}")).reshape(C, -1)[n], rec[f"gin{i}"], tol)
                assert ok, (f"gin{i}", n, e)
            if spec[0] == "block":  # every stored tensor inside the block
                names = [f"z{i}.1", f"act{i}.n1", f"z{i}.2", f"dz{i}.1", f"gpre{i}.n1", f"dz{i}.2"]
                if f"sc{i}" in rec:
                    names += [f"z{i}.p", f"sc{i}", f"dz{i}.p", f"gsc{i}"]
                for nm in names:
                    ok, e = close(_np(ctx.tensor(nm)).reshape(C, -1)[n], rec[nm], tol)
                    assert ok, (nm, n, e)
                if i > 0 and layers[i - 1][0] == "maxpool":
                    ok, e = close(_np(ctx.tensor(f"gin{i}")).reshape(C, -1)[n], rec[f"gin{i}"], tol)
                    assert ok, (f"gin{i}", n, e)
        ok, e = close(grads[n], g, tol)
        assert ok, ("grad", n, e)
        compare_params(grads[n], g, cfg, tol, ("grad", n))
        print(f"{name} replica {n}: decisions at near-ties {ch.flips}, largest distance {ch.worst:.2e}", flush=True)


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


@pytest.mark.parametrize("name", ["ragged", "tiny_norm", "gcpsl4"])
def test_fusion_in_two_halves_equals_fusion(name):
    """gcpsl_fuse_partial then gcpsl_fuse_finalise (the halves a sharded run
    puts an all-reduce between) against gcpsl_fuse on the same trained
    replicas: the fp64 partial equals the oracle's sum_n n_n theta_n bit for
    bit, the result equals gcpsl_fuse's bit for bit (parameters and
    normalisation state), and both count the same fusion payload."""
    cfg = get_config(name)
    ctx, assignment = driver.setup(cfg)
    driver.train(ctx, 3, F=0)
    torch.cuda.synchronize()
    before = ctx.theta.clone()
    ns_before = ctx.norm_state.clone() if ctx.S else None
    assert not torch.equal(before[0], before[1])
    sizes = ctx.cluster_sizes()
    partial = torch.zeros(ctx.P + ctx.S, dtype=torch.float64, device="cuda")
    ctx.fuse_partial(partial)
    torch.cuda.synchronize()
    got = partial.cpu().numpy()
    th = before.cpu().numpy()
    want = np.zeros(ctx.P)
    for n in range(cfg["C"]):
        want += float(sizes[n]) * th[n].astype(np.float64)
    assert np.array_equal(got[:ctx.P], want)
    if ctx.S:
        ns = ns_before.cpu().numpy()
        want_s = np.zeros(ctx.S)
        for n in range(cfg["C"]):
            want_s += float(sizes[n]) * ns[n].astype(np.float64)
        assert np.array_equal(got[ctx.P:], want_s)
    ctx.fuse_finalise(partial, int(sizes.sum()))
    torch.cuda.synchronize()
    halves = ctx.theta.clone()
    halves_ns = ctx.norm_state.clone() if ctx.S else None
    pay_halves = ctx.payload()["fusion"]
    ctx.theta.copy_(before)
    if ctx.S:
        ctx.norm_state.copy_(ns_before)
    ctx.fuse()
    torch.cuda.synchronize()
    assert torch.equal(ctx.theta, halves)
    if ctx.S:
        assert torch.equal(ctx.norm_state, halves_ns)
    assert ctx.payload()["fusion"] == 2 * pay_halves == 4 * 4 * cfg["C"] * (ctx.P + ctx.S)
    # a run whose replicas span other devices divides by the global W
    ctx.fuse_finalise(partial, 2 * int(sizes.sum()))
    torch.cuda.synchronize()
    half = (got[:ctx.P] / (2.0 * sizes.sum())).astype(np.float32)
    for n in range(cfg["C"]):
        assert np.array_equal(ctx.theta[n].cpu().numpy(), half)
    with pytest.raises(gcpsl.GCPSLError) as e:
        ctx.fuse_finalise(partial, 0)
    assert e.value.code == gcpsl.EINVAL


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

@pytest.mark.parametrize("name", ["gpsl", "gcpsl4", "gcpsl8", "gcpsl16", "resnet18", "resnet18_bf16"])
def test_full_size_round_sampled_replicas(name):
    """One round at the workload's real size; replicas 0 and C-1 recomputed by
    the oracle under the GPU's validated decisions: forward activations of
    every conv, loss, each layer's weight and bias gradient and the update."""
    cfg = get_config(name)
    ctx, assignment = driver.setup(cfg)
    C = cfg["C"]
    theta0 = ctx.theta[0].cpu().numpy().astype(np.float64)
    ctx.sample(0)
    loss = torch.zeros(C, device="cuda")
    ctx.step(0, loss)
    torch.cuda.synchronize()
    tol = bar(cfg)
    o = GCPSLOracle(cfg, cluster_of_client=assignment)
    grads = _np(ctx.tensor("grad")).reshape(C, -1)
    th = ctx.theta.cpu().numpy()
    layers = cfg["layers"]
    shapes = layer_shapes(cfg)
    for n in sorted({0, C - 1}):
        idx, x, y = o.batch(0, n)
        ch = GpuChoices(ctx, cfg, n)
        l, g, rec = split_forward_backward(cfg, o.theta[n], x, y, keep=True, choose=ch)
        assert abs(loss[n].item() - l) <= tol * abs(l), (n, loss[n].item(), l)
        for i, spec in enumerate(layers):
            if spec[0] not in ("conv", "block"):
                continue
            act = replica_tensor(ctx, f"act{i}", n, shapes[i])
            if act is None:
                # routing codes: the next stored output is the conv's max pool
                # (or, at the head, the mean over the pool)
                assert i in ch.route, i
                while act is None:
                    i += 1
                    act = replica_tensor(ctx, f"act{i}", n, shapes[i])
            ok, e = close(act, rec["acts"][i + 1], tol)
            assert ok, (f"act{i}", n, e)
        ok, e = close(grads[n], g, tol)
        assert ok, ("grad", n, ch.flips, e)
        compare_params(grads[n], g, cfg, tol, ("grad", n))
        # one update from v = 0 (the workload's SGD terms), stored as an fp32
        # master on both sides
        want32 = o.theta[n].copy()
        sgd_update(want32, np.zeros_like(want32), g, *sgd_args(cfg))
        want = want32.astype(np.float64)
        compare_params(th[n] - theta0, want - theta0, cfg, tol, ("update", n), ulp=master_ulp(want))
        print(f"{name} replica {n}: decisions at near-ties {ch.flips}, largest distance {ch.worst:.2e}", flush=True)
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


def test_create_rejects_labels_outside_the_classes():
    # the sampler counts labels per class for the batch deviation (Sec. V-E):
    # gcpsl_create reads them back and refuses any outside [0, L)
    from gcpsl_inputs import client_stats, init_params
    cfg = get_config("tiny")
    images, labels, coe = make_dataset(cfg)
    counts, hist = client_stats(cfg, labels, coe)
    assignment = gcpsl.assign(cfg["rule"], cfg["K"], cfg["C"], cfg["seed"], counts, hist)
    bad = labels.copy()
    bad[17] = cfg["L"]
    with pytest.raises(gcpsl.GCPSLError) as e:
        gcpsl.Context(cfg, images, bad, coe, assignment, init_params(cfg))
    assert e.value.code == gcpsl.EINVAL and "labels" in str(e.value)
