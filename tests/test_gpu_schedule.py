"""GPU parity of the epoch-barrier schedule (Sec. III-A; Sec. IV-D, Eq. 6)
and of sequential against concurrent execution of the clusters, through the
C ABI.  Floating point within the workload tolerance of the oracle (1e-4
fp32, 2e-2 bf16, per tensor as in test_gpu_parity); participation counts
bit-exact; sequential and concurrent GPU runs bit-identical to each other."""
import numpy as np
import pytest
import torch

from gcpsl_inputs import get_config
from oracle.train import GCPSLOracle, epoch_rounds

pytestmark = pytest.mark.gpu

from paper_2609_29395_amd import driver, gcpsl  # noqa: E402
from gpu_match import TOL, bar, LazyChoices, close, compare_params, master_ulp  # noqa: E402
from test_gpu_parity import check_metrics  # noqa: E402


# the routing-code paths under the epoch schedule (replicas addressed
# through the slot map, a waiting cluster): the image-side layer's codes
# (img32_bf16) and the head's (halo_maxhead_bf16), with data and batch
# sizes that make an epoch a few rounds long
CODES_EPOCH = {"img32_bf16": dict(schedule="epoch", B=48, N_ex=322, T=6),
               "halo_maxhead_bf16": dict(schedule="epoch", B=24, N_ex=203, T=7)}


@pytest.mark.parametrize("name", ["tiny_epoch", "ragged_epoch", "ragged_bf16_epoch", *CODES_EPOCH])
def test_epoch_schedule_parity(name):
    cfg = get_config(name, **CODES_EPOCH.get(name, {}))
    T = cfg["T"]
    print(f"epoch schedule parity: {name} T={T}", flush=True)
    ctx, assignment = driver.setup(cfg)
    ref = GCPSLOracle(cfg, cluster_of_client=assignment)
    rounds, R = ctx.epoch_rounds()
    assert (rounds.tolist(), R) == epoch_rounds(ref.weights, cfg["B"])
    assert T > R  # spans a fusion barrier
    theta0 = ctx.theta[0].cpu().numpy().astype(np.float64)
    losses = torch.full((T, cfg["C"]), float("nan"), device="cuda")
    for s in range(T):  # slot by slot, the oracle under the GPU's validated decisions
        ctx.sample(s)
        ctx.step(s, losses[s])
        torch.cuda.synchronize()
        ref.slot(s, choose=LazyChoices(ctx, cfg))
        if s % R == R - 1:
            ctx.fuse()
    torch.cuda.synchronize()
    tol = bar(cfg)
    got_l, want_l = losses.cpu().numpy(), np.array(ref.losses)
    ran = ~np.isnan(want_l)
    assert np.array_equal(~np.isnan(got_l), ran)  # waiting clusters write no loss
    assert np.all(np.abs(got_l[ran] - want_l[ran]) <= tol * np.abs(want_l[ran])), (got_l, want_l)
    th, mo = ctx.theta.cpu().numpy(), ctx.mom.cpu().numpy()
    for n in range(cfg["C"]):
        ok, e = close(th[n], ref.theta[n], tol)
        assert ok, ("theta", n, e)
        compare_params(th[n] - theta0, ref.theta[n] - theta0, cfg, tol, ("update", n),
                       ulp=master_ulp(ref.theta[n], T + T // R))
        compare_params(mo[n], ref.mom[n], cfg, tol, ("momentum", n))
    a, t, per = ctx.participation()
    assert t == cfg["K"] * T
    assert np.array_equal(per, np.array(ref.active)) and a == int(np.sum(ref.active))
    check_metrics(ctx, ref, cfg)  # waiting clusters: no batch deviation, no payload


def test_epoch_sample_marks_waiting_clusters():
    cfg = get_config("ragged_epoch")
    ctx, _ = driver.setup(cfg, max_window=8)
    rounds, R = ctx.epoch_rounds()
    out = torch.zeros(8, cfg["C"], cfg["B"], dtype=torch.int32, device="cuda")
    ctx.sample(R - 4, 8, out)  # slots across the epoch boundary
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    for j in range(8):
        t = (R - 4 + j) % R
        for n in range(cfg["C"]):
            if t < rounds[n]:
                assert (got[j, n] >= 0).all() and len(np.unique(got[j, n])) == cfg["B"]
            else:
                assert (got[j, n] == -1).all()


def _run(cfg, T, serial):
    ctx, _ = driver.setup(cfg)
    losses = torch.full((T, cfg["C"]), float("nan"), device="cuda")
    driver.train(ctx, T, losses=losses, serial=serial)
    torch.cuda.synchronize()
    return ctx, losses.cpu().numpy()


@pytest.mark.parametrize("name", ["tiny_epoch", "ragged_bf16_epoch", "ragged", "ragged_bf16", "tiny_norm",
                                  *CODES_EPOCH])
def test_sequential_equals_concurrent_bit_for_bit(name):
    # Eq. 6 compares running the cluster workloads one after another with
    # running them side by side: the same rounds, so the same results
    cfg = get_config(name, **CODES_EPOCH.get(name, {}))
    T = cfg["T"]
    print(f"sequential vs concurrent: {name} T={T}", flush=True)
    a, la = _run(cfg, T, serial=False)
    b, lb = _run(cfg, T, serial=True)
    assert np.array_equal(la, lb, equal_nan=True)
    assert torch.equal(a.theta, b.theta) and torch.equal(a.mom, b.mom)
    if a.S:
        assert torch.equal(a.norm_state, b.norm_state)
    assert np.array_equal(a.participation()[2], b.participation()[2])


def test_step_replica_errors():
    cfg = get_config("ragged_epoch")
    ctx, _ = driver.setup(cfg)
    rounds, R = ctx.epoch_rounds()
    with pytest.raises(gcpsl.GCPSLError) as e:
        ctx.step_replica(0, 0)
    assert e.value.code == gcpsl.ESTATE  # nothing sampled yet
    ctx.sample(R - 1)
    waiting = [n for n in range(cfg["C"]) if rounds[n] <= R - 1]
    assert waiting
    with pytest.raises(gcpsl.GCPSLError) as e:
        ctx.step_replica(R - 1, waiting[0])
    assert e.value.code == gcpsl.EINVAL
    with pytest.raises(gcpsl.GCPSLError) as e:
        ctx.step_replica(R - 1, cfg["C"])
    assert e.value.code == gcpsl.EINVAL
    ctx.step_replica(R - 1, int(np.argmax(rounds)))
    torch.cuda.synchronize()


def test_cluster_of_exactly_b_examples():
    # B = the smaller cluster's size: that cluster's epoch is one round whose
    # batch is all of its examples (in permuted order), every round a new epoch
    cfg = get_config("tiny", B=197, T=3, F=0)
    ctx, assignment = driver.setup(cfg, max_window=3)
    sizes = ctx.cluster_sizes()
    small = int(np.argmin(sizes))
    assert sizes[small] == cfg["B"]
    out = torch.zeros(3, cfg["C"], cfg["B"], dtype=torch.int32, device="cuda")
    ctx.sample(0, 3, out)
    torch.cuda.synchronize()
    ref = GCPSLOracle(cfg, cluster_of_client=assignment)
    got = out.cpu().numpy()
    for j in range(3):
        assert np.array_equal(np.sort(got[j, small]), ref.ids[small])
        assert not np.array_equal(got[0, small], got[1, small])  # a fresh permutation per epoch
    losses = torch.zeros(3, cfg["C"], device="cuda")
    for s in range(3):
        ctx.step(s, losses[s])
    torch.cuda.synchronize()
    ref.run(3, F=0)
    assert np.allclose(losses.cpu().numpy(), np.array(ref.losses), rtol=TOL["f32"])
    for n in range(cfg["C"]):
        ok, e = close(ctx.theta[n].cpu().numpy(), ref.theta[n], TOL["f32"])
        assert ok, (n, e)


def test_single_cluster_epoch_schedule_is_gpsl():
    # C = 1: the system epoch is the cluster's epoch and fusing one replica is
    # the identity, so the epoch schedule equals lockstep GPSL bit for bit
    cfg = get_config("tiny_epoch", C=1, B=32)
    ctx_e, _ = driver.setup(cfg, max_steps=20)
    rounds, R = ctx_e.epoch_rounds()
    assert R == rounds[0] == 512 // 32
    T = R + 2
    driver.train(ctx_e, T)
    ctx_l, _ = driver.setup(cfg, max_steps=20, schedule="lockstep")
    driver.train(ctx_l, T, F=0)
    torch.cuda.synchronize()
    assert torch.equal(ctx_e.theta, ctx_l.theta) and torch.equal(ctx_e.mom, ctx_l.mom)
    assert np.array_equal(ctx_e.participation()[2], ctx_l.participation()[2])
