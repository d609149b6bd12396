"""Pins for the oracle's SGD update, fusion (Eq. 5) and the training loop (Alg. 2)."""
import numpy as np
import pytest
import torch

from gcpsl_inputs import get_config, init_params
from oracle.train import GCPSLOracle, fuse, sgd_update

from conftest import load_golden


def test_sgd_two_steps_closed_form():
    # v1 = g0, theta1 = theta0 - lr g0; v2 = mu g0 + g1, theta2 = theta1 - lr v2
    theta = np.array([1.0, -2.0], dtype=np.float32)
    mom = np.zeros(2, dtype=np.float32)
    sgd_update(theta, mom, np.array([0.5, 0.25]), 0.1, 0.9)
    assert np.allclose(theta, [0.95, -2.025], rtol=1e-7)
    sgd_update(theta, mom, np.array([-1.0, 2.0]), 0.1, 0.9)
    assert np.allclose(mom, [-0.55, 2.225], rtol=1e-7)
    assert np.allclose(theta, [1.005, -2.2475], rtol=1e-7)


def test_sgd_matches_torch_optimizer():
    rng = np.random.default_rng(0)
    t0 = rng.standard_normal(50).astype(np.float32)
    grads = [rng.standard_normal(50) for _ in range(4)]
    theta, mom = t0.copy(), np.zeros(50, dtype=np.float32)
    p = torch.nn.Parameter(torch.tensor(t0, dtype=torch.float64))
    opt = torch.optim.SGD([p], lr=0.05, momentum=0.9)
    for g in grads:
        sgd_update(theta, mom, g, 0.05, 0.9)
        p.grad = torch.tensor(g)
        opt.step()
    assert np.allclose(theta, p.detach().numpy(), rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("mu,wd,nesterov", [(0.9, 5e-4, True), (0.9, 5e-4, False), (0.9, 0.0, True),
                                             (0.0, 5e-4, False), (0.5, 0.1, True)])
def test_sgd_weight_decay_and_nesterov_match_torch_optimizer(mu, wd, nesterov):
    """The paper's recipe (Sec. V-A): momentum 0.9 with the Nesterov term and
    weight decay 5e-4, against torch.optim.SGD in fp64 over several steps."""
    rng = np.random.default_rng(11)
    t0 = rng.standard_normal(64).astype(np.float32)
    grads = [rng.standard_normal(64) for _ in range(5)]
    theta, mom = t0.copy(), np.zeros(64, dtype=np.float32)
    p = torch.nn.Parameter(torch.tensor(t0, dtype=torch.float64))
    opt = torch.optim.SGD([p], lr=0.01, momentum=mu, weight_decay=wd, nesterov=nesterov and mu > 0)
    for g in grads:
        sgd_update(theta, mom, g, 0.01, mu, wd, nesterov)
        p.grad = torch.tensor(g)
        opt.step()
    assert np.allclose(theta, p.detach().numpy(), rtol=1e-6, atol=1e-7)


def test_sgd_nesterov_weight_decay_closed_form():
    # theta0 = 2, wd = 0.5, mu = 0.5, lr = 0.1, g = 1:
    # g' = 1 + 0.5*2 = 2; v1 = 2; step = g' + mu v1 = 3; theta1 = 2 - 0.3 = 1.7
    # g' = 1 + 0.85 = 1.85; v2 = 1 + 1.85 = 2.85; step = 1.85 + 1.425 = 3.275; theta2 = 1.3725
    theta = np.array([2.0], dtype=np.float32)
    mom = np.zeros(1, dtype=np.float32)
    sgd_update(theta, mom, np.array([1.0]), 0.1, 0.5, 0.5, True)
    assert theta[0] == pytest.approx(1.7, rel=1e-7) and mom[0] == 2.0
    sgd_update(theta, mom, np.array([1.0]), 0.1, 0.5, 0.5, True)
    assert mom[0] == pytest.approx(2.85, rel=1e-7)
    assert theta[0] == pytest.approx(1.3725, rel=1e-7)
    # without the extra terms the update is the plain momentum step
    t1, m1 = np.array([2.0], np.float32), np.zeros(1, np.float32)
    sgd_update(t1, m1, np.array([1.0]), 0.1, 0.5, 0.0, False)
    assert t1[0] == pytest.approx(1.9, rel=1e-7)


def test_recipe_rounds_match_torch_training_loop():
    """One cluster, three rounds of the paper's recipe (Nesterov, weight
    decay, label smoothing) against torch autograd + torch.optim.SGD in fp64
    on the same batches."""
    from test_oracle_model import torch_split_model_loss
    cfg = get_config("tiny_recipe", C=1, F=0, dtype="f32")
    o = GCPSLOracle(cfg)
    p = torch.nn.Parameter(torch.tensor(o.theta[0], dtype=torch.float64))
    opt = torch.optim.SGD([p], lr=cfg["lr"], momentum=cfg["momentum"], weight_decay=cfg["weight_decay"],
                          nesterov=True)
    for step in range(3):
        _, x, y = o.batch(step, 0)
        want_loss, g = torch_split_model_loss(cfg, p.detach().numpy(), x, y)
        losses, _ = o.round(step)
        assert losses[0] == pytest.approx(want_loss, rel=1e-6)
        p.grad = torch.tensor(g)
        opt.step()
        assert np.allclose(o.theta[0], p.detach().numpy(), rtol=1e-5, atol=1e-7), step


@pytest.mark.parametrize("name, F, steps", [("ragged", 3, 7), ("tiny_recipe", 2, 5), ("ragged_bf16", 2, 5),
                                           ("resnet_tiny", 2, 3)])
def test_run_across_fusions_matches_torch_training_loops(name, F, steps):
    """Multi-round end-to-end values (Alg. 2, Eq. 5): C replicas, each trained
    by its own torch.optim.SGD (momentum kept local) on torch.autograd
    gradients in fp64 on the same batches, and every F rounds replaced by
    numpy's weighted average of the replicas with the clusters' example counts
    as weights.  Parameters, momenta and the fused parameters are stored in
    fp32 after each update, as the workloads keep them (bf16 rounding happens
    only inside the forward and backward passes).  The oracle's run must give
    the same loss for every cluster and round, and the same parameters and
    momenta at the end (up to one fp32 ulp: torch steps with the momentum
    before it is stored)."""
    from test_oracle_model import torch_split_model_loss
    cfg = get_config(name, F=F)
    C = cfg["C"]
    o = GCPSLOracle(cfg)
    w = np.bincount(o.assignment[o.coe], minlength=C)  # examples per cluster
    assert w.sum() == cfg["N_ex"] and len(set(w.tolist())) == C  # unequal weights
    ps = [torch.nn.Parameter(torch.tensor(o.theta[n], dtype=torch.float64)) for n in range(C)]
    opts = [torch.optim.SGD([p], lr=cfg["lr"], momentum=cfg["momentum"], weight_decay=cfg["weight_decay"],
                            nesterov=cfg["nesterov"]) for p in ps]
    want = []
    for s in range(steps):
        want.append([])
        for n in range(C):
            _, x, y = o.batch(s, n)  # the keyed sampler, pinned on its own
            loss, g = torch_split_model_loss(cfg, ps[n].detach().numpy(), x, y)
            want[-1].append(loss)
            ps[n].grad = torch.tensor(g)
            opts[n].step()
            buf = opts[n].state[ps[n]]["momentum_buffer"]
            for t in (ps[n].data, buf):
                t.copy_(t.float().double())
        if (s + 1) % F == 0:
            avg = np.average(np.stack([p.detach().numpy() for p in ps]), axis=0, weights=w)
            for p in ps:
                p.data = torch.tensor(avg.astype(np.float32).astype(np.float64))
    o.run(steps)
    assert np.allclose(np.array(o.losses), np.array(want), rtol=1e-7, atol=0)
    for n in range(C):
        assert np.allclose(o.theta[n], ps[n].detach().numpy(), rtol=1e-5, atol=1e-7), n
        buf = opts[n].state[ps[n]]["momentum_buffer"].numpy()
        assert np.allclose(o.mom[n], buf, rtol=1e-5, atol=1e-7), n
    # the run ends between fusions: the replicas have trained apart again
    assert not np.array_equal(o.theta[0], o.theta[1])


@pytest.mark.parametrize("name", ["resnet_tiny_bf16", "ragged_recipe_bf16"])
def test_rounds_of_a_run_match_torch_at_the_oracles_parameters(name):
    """bf16 runs with norm layers drift apart from a free-running torch loop
    once a one-ulp difference in an fp32 master weight flips its bf16
    rounding, so each round of a 4-round run with fusions (F = 2) is checked
    from the oracle's own parameters at that point: the loss and gradient it
    takes must be torch.autograd's at the same parameters and batch."""
    from test_oracle_model import torch_split_model_loss
    cfg = get_config(name, F=2)
    o = GCPSLOracle(cfg)
    for s in range(4):
        theta = [t.copy() for t in o.theta]
        losses, grads = o.round(s)
        for n in range(cfg["C"]):
            _, x, y = o.batch(s, n)
            want_loss, g = torch_split_model_loss(cfg, theta[n], x, y)
            assert losses[n] == pytest.approx(want_loss, rel=1e-12), (s, n)
            assert np.allclose(grads[n], g, rtol=1e-9, atol=1e-12 * np.abs(g).max()), (s, n)
        if (s + 1) % 2 == 0:
            o.fuse()
    assert np.array_equal(o.theta[0], o.theta[1])  # fused after the last round


def test_fusion_worked_example():
    # tests/golden: weights 1, 2, 5 (W = 8): (1*[8,0] + 2*[0,4] + 5*[0.8,-1.6]) / 8 = [1.5, 0]
    g = load_golden("fusion_eq5_worked.txt")
    th = [np.array(g[f"theta{n}"], np.float32) for n in range(len(g["weights"]))]
    assert np.allclose(fuse(th, g["weights"]), g["fused"], atol=1e-7)


def test_fusion_of_identical_replicas_is_bit_exact_identity():
    rng = np.random.default_rng(1)
    t = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    for weights in ([12544, 13151, 13337, 10968], [1, 1], [155, 11279, 7, 3, 99991]):
        out = fuse([t.copy() for _ in weights], weights)
        assert out.dtype == np.float32 and np.array_equal(out, t)


def test_fusion_weights_sum_to_one_exactly():
    # constant replicas c_n: the result is the exact weighted mean
    w = [3, 5, 8]
    th = [np.full(4, c, np.float32) for c in (1.0, 2.0, 4.0)]
    assert np.all(fuse(th, w) == np.float32((3 * 1 + 5 * 2 + 8 * 4) / 16))


def test_single_cluster_gcpsl_equals_gpsl():
    # C = 1: fusion over one replica is the identity, so any fusion interval
    # gives the GPSL run bit for bit
    cfg = get_config("tiny", C=1)
    a = GCPSLOracle(cfg).run(6, F=2)
    b = GCPSLOracle(cfg).run(6, F=0)
    assert np.array_equal(a.theta[0], b.theta[0])
    assert a.losses == b.losses


def test_fusion_leaves_momentum_local_and_replicas_equal():
    cfg = get_config("tiny")
    o = GCPSLOracle(cfg).run(5, F=5)
    assert np.array_equal(o.theta[0], o.theta[1])
    assert not np.array_equal(o.mom[0], o.mom[1]) or cfg["momentum"] == 0.0
    cfg = get_config("ragged")
    o = GCPSLOracle(cfg).run(3, F=3)
    assert all(np.array_equal(o.theta[0], t) for t in o.theta)
    assert not np.array_equal(o.mom[0], o.mom[1])


def test_replicas_start_equal_and_train_apart():
    cfg = get_config("ragged")
    o = GCPSLOracle(cfg)
    t0 = init_params(cfg)
    assert all(np.array_equal(t, t0) for t in o.theta)
    o.run(2, F=0)
    assert not np.array_equal(o.theta[0], o.theta[1])
    assert len(o.active) == 2 and all(1 <= a <= cfg["B"] for row in o.active for a in row)


def test_tiny_workload_learns():
    # The class-mean images are separable: 200 rounds must take the mean
    # loss well below the chance level log(4).
    cfg = get_config("tiny")
    o = GCPSLOracle(cfg).run(200)
    L = np.array(o.losses).mean(axis=1)
    assert abs(L[:5].mean() - np.log(4)) < 0.1
    assert L[-20:].mean() < 0.5


def test_normalisation_state_is_fused_with_the_parameter_weights():
    # Sec. IV-B / IV-C: each server replica's BatchNorm running mean, variance
    # and counter evolve locally and are fused with the weights n_n / W
    cfg = get_config("tiny_norm", F=0)
    o = GCPSLOracle(cfg)
    for s in range(3):
        o.round(s)
    assert not np.array_equal(o.norm[0], o.norm[1])
    before = [st.astype(np.float64) for st in o.norm]
    W = sum(o.weights)
    want = (sum(w * st for w, st in zip(o.weights, before)) / W).astype(np.float32)
    o.fuse()
    for st in o.norm:
        assert np.array_equal(st, want)
    # the counter of every replica is 3 rounds, so the fused counter is 3
    from gcpsl_inputs import norm_layout
    counts = [off for _, tag, _, off in norm_layout(cfg) if tag == "count"]
    assert all(o.norm[0][c] == 3.0 for c in counts)
