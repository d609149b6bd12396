"""Routing codes of the image-side max pool, checked against the GPU's own
state round after round (8-cluster workload, full size).

Each round, from the layer input and the bf16 weights the GPU itself used,
the CPU recomputes (oracle conv helpers, fp64) the 32 -> 64 layer's output,
its 2 x 2 max pool and the pool's routing codes, and from the GPU's cut
gradient and codes the layer's weight gradient and the input gradient of the
layer below.  The GPU's pool, codes and gradients must agree up to rounding
(codes may differ only where the window's two largest values are within
rounding of each other).  Unlike the matched runs this does not depend on
the oracle's own trajectory, so a wrong code in any round shows at once (a
missing LDS wait in the pool epilogue once let a wave read its neighbour's
staged row early and corrupted a few windows every few rounds)."""
import numpy as np
import pytest
import torch

from gcpsl_inputs import get_config
from gcpsl_inputs.configs import param_layout
from gpu_match import pool_windows, routed_gradient, to_np
from oracle.model import conv3x3_backward, conv3x3_forward, round_bf16

pytestmark = pytest.mark.gpu

from paper_2609_29395_amd import driver  # noqa: E402


def test_codes_pool_and_routed_gradients_follow_the_gpu_state():
    cfg = get_config("gcpsl8")
    C, B = cfg["C"], cfg["B"]
    rounds, reps = 4, (0, 3, 7)
    ctx, _ = driver.setup(cfg, max_steps=rounds)
    lay = {(i, t): (shp, off) for i, t, shp, off in param_layout(cfg)}

    def part(theta, i, t):
        shp, off = lay[(i, t)]
        return theta[off:off + int(np.prod(shp))].reshape(shp)

    loss = torch.zeros(C, device="cuda")
    for s in range(rounds):
        theta = ctx.theta.cpu().numpy().astype(np.float64)
        ctx.sample(s)
        ctx.step(s, loss)
        torch.cuda.synchronize()
        a0 = to_np(ctx.tensor("act0")).reshape(C, B, 32, 32, 32).astype(np.float64)
        pool = to_np(ctx.tensor("act2")).reshape(C, B, 16, 16, 64).astype(np.float64)
        route = to_np(ctx.tensor("route2")).reshape(C, B, 16, 16, 64).astype(np.int64)
        gin = to_np(ctx.tensor("gin3")).reshape(C, B, 16, 16, 64).astype(np.float64)
        gpre0 = to_np(ctx.tensor("gpre0")).reshape(C, B, 32, 32, 32).astype(np.float64)
        grad = ctx.tensor("grad").cpu().numpy().reshape(C, -1).astype(np.float64)
        for n in reps:
            w1 = round_bf16(part(theta[n], 1, "w"))
            z = conv3x3_forward(a0[n], w1, part(theta[n], 1, "b"))
            a = round_bf16(np.maximum(z, 0.0))
            win = pool_windows(a)
            mx = win.max(axis=3)
            scale = np.abs(z).max()
            # pool: one bf16 rounding of an fp32 sum apart
            assert np.abs(pool[n] - mx).max() <= 2 ** -7 * scale, (s, n)
            # codes: 0..4; where they differ from the recomputed first maximum,
            # the window value they name is within rounding of the maximum
            assert route[n].min() >= 0 and route[n].max() <= 4, (s, n)
            code = np.where(mx > 0, np.argmax(win, axis=3), 4)
            named = np.where(route[n] < 4, np.take_along_axis(
                win, np.minimum(route[n], 3)[:, :, :, None, :], axis=3)[:, :, :, 0, :], 0.0)
            gap = np.abs(mx - named)[code != route[n]]
            assert gap.size == 0 or gap.max() <= 2 ** -7 * scale, (s, n, int((code != route[n]).sum()), gap.max())
            # the layer's gradients from the GPU's cut gradient and codes
            g = routed_gradient(gin[n], route[n])
            dx, dw, _ = conv3x3_backward(a0[n], w1, g)
            gw = part(grad[n], 1, "w")
            assert np.abs(gw - dw).max() <= 1e-4 * np.abs(dw).max(), (s, n)
            want0 = dx * (a0[n] > 0)
            assert np.abs(gpre0[n] - want0).max() <= 2 ** -7 * np.abs(want0).max(), (s, n)


def test_codes_break_exact_ties_at_the_first_window_position():
    # With the 32 -> 64 layer's weights zero, every pre-activation of a
    # channel is its bias, so all four values of every 2 x 2 window tie: the
    # pool's code is the first position (0) where the bias is positive and 4
    # (no positive value) where it is zero or negative, and the pooled value
    # is the bf16 bias or 0, exactly (Sec. III-A's forward with the stored
    # max pool; the first maximum in row-major window order).
    cfg = get_config("gcpsl8")
    C, B = cfg["C"], cfg["B"]
    ctx, _ = driver.setup(cfg, max_steps=1)
    lay = {(i, t): (shp, off) for i, t, shp, off in param_layout(cfg)}
    (wshp, woff), (bshp, boff) = lay[(1, "w")], lay[(1, "b")]
    co = int(bshp[0])
    pattern = np.array([0.5, -0.25, 0.0, 1e-3])
    bias = pattern[np.arange(co) % 4]
    ctx.theta[:, woff:woff + int(np.prod(wshp))] = 0.0
    ctx.theta[:, boff:boff + co] = torch.tensor(bias, dtype=torch.float32, device="cuda")
    loss = torch.zeros(C, device="cuda")
    ctx.sample(0)
    ctx.step(0, loss)
    torch.cuda.synchronize()
    pool = to_np(ctx.tensor("act2")).reshape(C, B, 16, 16, co).astype(np.float64)
    route = to_np(ctx.tensor("route2")).reshape(C, B, 16, 16, co).astype(np.int64)
    want_code = np.where(bias > 0, 0, 4)
    want_pool = round_bf16(np.maximum(bias, 0.0))
    assert np.array_equal(route, np.broadcast_to(want_code, route.shape)), \
        np.unique(route.reshape(-1, co), axis=0)[:4]
    assert np.array_equal(pool, np.broadcast_to(want_pool, pool.shape))
