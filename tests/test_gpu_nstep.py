"""N-step GPU parity at the workloads' real sizes (Alg. 2 with Eq. 5 fusion).

Each of the four CIFAR-shaped workloads runs N rounds on the GPU through the
C ABI, and the oracle runs the same N rounds, every round under the GPU's
ReLU and max-pool decisions where they are validated near-ties (gpu_match).
N spans a fusion where the workload fuses:

    gpsl     C = 1,  fp32, N = 20 (no fusion: one cluster)
    gcpsl4   C = 4,  fp32, N = 51 (fusion after round 50)
    gcpsl8   C = 8,  bf16, N = 26 (fusion after round 25)
    gcpsl16  C = 16, bf16, N = 3 with fusion every 2 rounds (the workload
             fuses every 50; the interval is shortened so a fusion of trained
             replicas falls inside an N the oracle finishes in minutes)
    resnet18 the paper's ResNet-18 split after stage 2 (Sec. V-A), C = 4,
             fp32 and bf16, N = 2 ending on a fusion (lockstep; the
             workload fuses after each epoch of about 175 rounds); the bf16
             run's updates and momenta take the twin-calibrated bar of deep
             bf16 networks (gpu_match.twin_bar)

Compared: every round's loss of every cluster (elementwise), and for every
replica its parameters, its update theta_N - theta_0 and its momentum, each
layer's weight and bias on its own, at 1e-4 (fp32) or 2e-2 (bf16);
participation per round and cluster bit-exact.
"""
import time

import pytest

from gcpsl_inputs import get_config

from test_gpu_parity import check_run, matched_run

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,N,F", [("gpsl", 20, None), ("gcpsl4", 51, None), ("gcpsl8", 26, None),
                                      ("gcpsl16", 3, 2), ("resnet18", 2, 2), ("resnet18_bf16", 2, 2)])
def test_full_size_n_rounds(name, N, F):
    cfg = get_config(name)
    if F is not None:
        cfg["F"] = F
        cfg["schedule"] = "lockstep"
    t0 = time.time()

    def log(msg):
        print(f"{name}: {msg} ({time.time() - t0:.0f} s)", flush=True)

    ctx, o, theta0, losses, flips = matched_run(cfg, N, log=log)
    check_run(ctx, o, theta0, losses, cfg)
    log(f"N={N} F={cfg['F']} parity ok, {flips} decisions at near-ties")
