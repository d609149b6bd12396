"""The routing codes a 2 x 2 max pool keeps in place of its unpooled input
(the library's "route<j>" tensors: window position 0..3 of the first
row-major maximum, 4 where that maximum is not positive), and the host-side
expansion the GPU parity tests use to compare the gradient routed through
them with the oracle's pre-activation gradient.  Pinned here on the CPU to a
brute-force loop over the windows and to the oracle's own max-pool and ReLU
backward; no GPU involved."""
import numpy as np
import pytest

from gpu_match import pool_windows, routed_gradient, unpool_windows
from oracle.model import maxpool2_backward, maxpool2_forward


def _codes(a):
    """Codes of a post-ReLU activation a [Bt,H,W,C], by brute force."""
    Bt, H, W, C = a.shape
    out = np.empty((Bt, H // 2, W // 2, C), np.int64)
    for b in range(Bt):
        for i in range(H // 2):
            for j in range(W // 2):
                for c in range(C):
                    win = [a[b, 2 * i + k // 2, 2 * j + k % 2, c] for k in range(4)]
                    k = 0
                    for q in range(1, 4):  # first maximum under strict comparison
                        if win[q] > win[k]:
                            k = q
                    out[b, i, j, c] = k if win[k] > 0 else 4
    return out


def test_unpool_inverts_pool_windows():
    x = np.random.default_rng(0).standard_normal((2, 6, 8, 3))
    assert np.array_equal(unpool_windows(pool_windows(x)), x)


@pytest.mark.parametrize("seed", [1, 2])
def test_routed_gradient_is_the_oracle_max_pool_and_relu_backward(seed):
    rng = np.random.default_rng(seed)
    # ties and all-zero windows are frequent after rounding and the ReLU
    a = np.maximum(rng.standard_normal((2, 8, 6, 5)).round(1), 0.0)
    g = rng.standard_normal((2, 4, 3, 5))
    codes = _codes(a)
    assert (codes == 4).any() and (codes < 4).any()
    _, arg = maxpool2_forward(a)
    assert np.array_equal(np.where(codes < 4, codes, arg), arg)  # the same first maximum
    want = maxpool2_backward(g, arg) * (a > 0)
    assert np.array_equal(routed_gradient(g, codes), want)
