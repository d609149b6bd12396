"""gcpsl_create_static, the allocation-free context: its workspace is the
library's static device array instead of a caller buffer.  Two runs in a row
(the second on a smaller workload, in the array the first one left behind)
against the same runs on contexts with caller-owned workspaces: the same
kernels on the same inputs, so every loss, parameter, momentum, participation
count, batch deviation and payload byte agrees bit for bit."""
import numpy as np
import pytest
import torch

from gcpsl_inputs import get_config

pytestmark = pytest.mark.gpu

from paper_2609_29395_amd import driver, gcpsl  # noqa: E402


def _run(cfg, static):
    T = cfg["T"]
    ctx, _ = driver.setup(cfg, static=static)
    losses = torch.zeros(T, cfg["C"], device="cuda")
    driver.train(ctx, T, losses=losses)
    torch.cuda.synchronize()
    out = dict(losses=losses.cpu().numpy(), theta=ctx.theta.cpu().numpy(), mom=ctx.mom.cpu().numpy(),
               part=ctx.participation(), dev=ctx.batch_deviation(), pay=ctx.payload(),
               norm=ctx.norm_state.cpu().numpy() if ctx.S else None)
    return ctx, out


def _same(a, b):
    assert np.array_equal(a["losses"], b["losses"])
    assert np.array_equal(a["theta"], b["theta"]) and np.array_equal(a["mom"], b["mom"])
    assert a["part"][:2] == b["part"][:2] and np.array_equal(a["part"][2], b["part"][2])
    assert a["dev"][:3] == b["dev"][:3] and np.array_equal(a["dev"][3], b["dev"][3])
    assert a["pay"] == b["pay"]
    if a["norm"] is not None:
        assert np.array_equal(a["norm"], b["norm"])


def test_static_context_matches_caller_workspace_twice_in_a_row():
    # first call: the ragged bf16 workload (about 9 MiB of workspace)
    big = get_config("ragged_bf16")
    ctx_s, got = _run(big, static=True)
    _, want = _run(big, static=False)
    _same(got, want)
    # a second static context on the same device is refused while one lives
    with pytest.raises(gcpsl.GCPSLError) as e:
        driver.setup(get_config("tiny"), static=True)
    assert e.value.code == gcpsl.ESTATE
    ctx_s.close()
    # second call, smaller input (with batch-norm state), in the array the
    # first run left behind
    small = get_config("tiny_norm")
    ctx_s2, got = _run(small, static=True)
    _, want = _run(small, static=False)
    _same(got, want)
    ctx_s2.close()


def test_static_context_rejects_a_workspace_beyond_the_array():
    cfg = get_config("gpsl")  # about 218 MiB of workspace
    with pytest.raises(gcpsl.GCPSLError) as e:
        driver.setup(cfg, static=True)
    assert e.value.code == gcpsl.EINVAL and "static workspace" in str(e.value)
    # the failed call left the device's array free
    ctx, _ = driver.setup(get_config("tiny"), static=True)
    ctx.close()
