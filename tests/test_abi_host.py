"""Host-side checks of the C ABI (no GPU needed).

The library must load, export every function include/gcpsl.h declares, run
Alg. 1 on the host bit-exactly like the oracle, and reject bad arguments with
the documented codes before touching the device.
"""
import ctypes as C
import os
import re

import numpy as np
import pytest

from gcpsl_inputs import client_stats, get_config, make_dataset, param_counts
from oracle.assign import assign as oracle_assign

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
g = pytest.importorskip("paper_2609_29395_amd.gcpsl")

if not os.path.exists(g.LIB_PATH):
    pytest.skip("libgcpsl.so not built", allow_module_level=True)


def header_functions():
    text = open(os.path.join(ROOT, "include", "gcpsl.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gcpsl_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = g.lib()
    names = header_functions()
    assert set(names) == set(g.EXPORTS), names
    for n in names:
        assert hasattr(lib, n), n


def test_library_has_no_cuda_symbols():
    out = os.popen(f"nm -D --defined-only {g.LIB_PATH}").read()
    assert "cuda" not in out.lower()


@pytest.mark.parametrize("name", ["tiny", "gcpsl4", "gcpsl8", "gcpsl16", "ragged", "ragged_bf16"])
def test_assign_matches_oracle_bit_exact(name):
    cfg = get_config(name)
    _, labels, coe = make_dataset(cfg)
    counts, hist = client_stats(cfg, labels, coe)
    for rule in ("random", "size", "label_l1"):
        for seed in (0, 1, 12345):
            want = oracle_assign(rule, cfg["K"], cfg["C"], seed, counts, hist)
            got = g.assign(rule, cfg["K"], cfg["C"], seed, counts, hist)
            assert np.array_equal(got, want), (rule, seed)


def test_assign_random_many_shapes():
    for K, Cc in [(1, 1), (2, 2), (3, 2), (17, 5), (1000, 7), (65536, 64)]:
        for seed in (0, 2**63 + 5):
            assert np.array_equal(g.assign("random", K, Cc, seed), oracle_assign("random", K, Cc, seed))


def test_assign_label_l1_random_histograms():
    rng = np.random.default_rng(7)
    for trial in range(20):
        K, Cc, L = int(rng.integers(2, 60)), int(rng.integers(1, 9)), int(rng.integers(1, 12))
        Cc = min(Cc, K)
        hist = rng.integers(0, 30, size=(K, L)) * (rng.random((K, L)) < 0.5)
        counts = hist.sum(1)
        for rule in ("size", "label_l1"):
            assert np.array_equal(g.assign(rule, K, Cc, 0, counts, hist),
                                  oracle_assign(rule, K, Cc, 0, counts, hist))


def test_assign_errors():
    counts = np.ones(4, dtype=np.int64)
    with pytest.raises(g.GCPSLError) as e:
        g.assign("random", 4, 5, 0)
    assert e.value.code == g.EINVAL
    with pytest.raises(g.GCPSLError) as e:
        g.assign(7, 4, 2, 0, counts)
    assert e.value.code == g.EINVAL
    with pytest.raises(g.GCPSLError) as e:
        g.assign("size", 4, 2, 0)
    assert e.value.code == g.EINVAL
    with pytest.raises(g.GCPSLError) as e:
        g.assign("label_l1", 4, 2, 0, counts)
    assert e.value.code == g.EINVAL
    bad = np.array([[1, 0], [0, 1], [1, 1], [2, 0]])
    with pytest.raises(g.GCPSLError) as e:
        g.assign("label_l1", 4, 2, 0, np.array([1, 1, 1, 1]), bad)  # row 2 sums to 2 != 1
    assert e.value.code == g.EINVAL


@pytest.mark.parametrize("name", ["tiny", "gpsl", "gcpsl16", "ragged", "tiny_norm", "ragged_norm_bf16",
                                  "ragged_recipe_bf16", "resnet_tiny", "resnet_tiny_bf16", "resnet18"])
def test_param_count_matches_layout(name):
    from gcpsl_inputs import norm_layout
    cfg = get_config(name)
    _, labels, coe = make_dataset(cfg)
    d, keep = g.make_desc(cfg, coe, np.zeros(cfg["K"], np.int32))
    P, Pc = g.param_count(d)
    pc, ps = param_counts(cfg)
    assert (P, Pc) == (pc + ps, pc)
    nl = norm_layout(cfg)
    assert g.state_count(d) == (nl[-1][3] + nl[-1][2][0] if nl else 0)
    assert g.workspace_bytes(d) > 0


def test_norm_layer_shapes_are_checked():
    base = get_config("tiny_norm")
    _, labels, coe = make_dataset(base)
    bad = [
        # group norm groups must divide the channels
        [("conv", 3, 8, False), ("gnorm", 8, 3), ("maxpool",), ("conv", 8, 16, False), ("bnorm", 16),
         ("avgpool",), ("linear", 16, 4)],
        # a norm layer needs a conv before it
        [("conv", 3, 8, False), ("maxpool",), ("bnorm", 8), ("conv", 8, 16, False), ("avgpool",),
         ("linear", 16, 4)],
        # a residual conv cannot feed a norm layer
        [("conv", 3, 8, False), ("maxpool",), ("conv", 8, 8, True), ("bnorm", 8), ("avgpool",),
         ("linear", 8, 4)],
        # norm channels must match the conv
        [("conv", 3, 8, False), ("gnorm", 16, 2), ("maxpool",), ("conv", 8, 16, False), ("avgpool",),
         ("linear", 16, 4)],
    ]
    for layers in bad:
        cfg = get_config("tiny_norm", layers=layers)
        d, keep = g.make_desc(cfg, coe, np.zeros(cfg["K"], np.int32))
        with pytest.raises(g.GCPSLError) as e:
            g.param_count(d)
        assert e.value.code in (g.EINVAL, g.EUNSUPPORTED), layers


def test_parameter_counts_of_the_workload_models():
    assert param_counts(get_config("tiny")) == (224, 1236)
    assert param_counts(get_config("gpsl")) == (19392, 222730)
    assert param_counts(get_config("gcpsl16")) == (19392, 1920522)


def _desc(cfg, **over):
    _, labels, coe = make_dataset(cfg)
    d, keep = g.make_desc(cfg, coe, np.arange(cfg["K"], dtype=np.int32) % cfg["C"])
    for k, v in over.items():
        setattr(d, k, v)
    return d, keep


def _create(d):
    h = C.c_void_p()
    rc = g.lib().gcpsl_create(C.byref(d), C.byref(h))
    return rc, g.lib().gcpsl_last_error().decode()


def test_create_rejects_bad_descriptions_before_device_work():
    cfg = get_config("tiny")
    fake = 1 << 20  # never dereferenced: every case fails validation first
    base = dict(images=fake, labels=fake, theta=fake, momentum_buf=fake, workspace=fake,
                workspace_bytes=1 << 40)
    d, k = _desc(cfg, **base)
    d.images = None
    assert _create(d)[0] == g.EINVAL
    d, k = _desc(cfg, **dict(base, workspace_bytes=16))
    rc, msg = _create(d)
    assert rc == g.EINVAL and "workspace" in msg
    d, k = _desc(cfg, **dict(base, workspace=fake + 8))
    assert _create(d)[0] == g.EINVAL
    d, k = _desc(cfg, **dict(base, B=400))  # clusters hold 197 and 315 examples
    rc, msg = _create(d)
    assert rc == g.EINVAL and "< B" in msg
    d, k = _desc(cfg, **dict(base, schedule=2))  # unknown schedule
    assert _create(d)[0] == g.EINVAL
    d, k = _desc(cfg, **dict(base, dtype=9))
    assert _create(d)[0] == g.EINVAL
    for bad in (dict(weight_decay=-1e-4), dict(weight_decay=float("inf")), dict(nesterov=2),
                dict(label_smoothing=1.0), dict(label_smoothing=-0.1), dict(label_smoothing=float("nan"))):
        d, k = _desc(cfg, **dict(base, **bad))
        rc, msg = _create(d)
        assert rc == g.EINVAL, bad


def test_unsupported_models_are_reported():
    cfg = get_config("tiny", layers=[("conv", 3, 12, False), ("maxpool",), ("conv", 12, 16, False),
                                     ("avgpool",), ("linear", 16, 4)])
    d, k = _desc(cfg)
    with pytest.raises(g.GCPSLError) as e:
        g.param_count(d)
    assert e.value.code == g.EUNSUPPORTED
    cfg = get_config("tiny", layers=[("conv", 3, 8, False), ("avgpool",), ("conv", 8, 16, False),
                                     ("linear", 16, 4)])
    d, k = _desc(cfg)
    with pytest.raises(g.GCPSLError) as e:
        g.param_count(d)
    assert e.value.code in (g.EUNSUPPORTED, g.EINVAL)
    cfg = get_config("tiny", layers=[("conv", 3, 8, True), ("maxpool",), ("conv", 8, 16, False),
                                     ("avgpool",), ("linear", 16, 4)])
    d, k = _desc(cfg)
    with pytest.raises(g.GCPSLError) as e:
        g.param_count(d)
    assert e.value.code == g.EINVAL


@pytest.mark.parametrize("name", ["tiny", "gcpsl4", "gcpsl8", "gcpsl16", "ragged"])
def test_assign_label_jsd_matches_oracle_bit_exact(name):
    """The paper's label-aware move search (Eq. 4) on each workload's client
    histograms: same clusters as the oracle, bit for bit."""
    from oracle.assign import assign_label_jsd
    cfg = get_config(name)
    _, labels, coe = make_dataset(cfg)
    counts, hist = client_stats(cfg, labels, coe)
    want = assign_label_jsd(cfg["K"], cfg["C"], counts, hist)[0]
    got = g.assign("label_jsd", cfg["K"], cfg["C"], 0, counts, hist)
    assert np.array_equal(got, want)


def test_assign_label_jsd_random_instances():
    from oracle.assign import assign_label_jsd
    rng = np.random.default_rng(21)
    for trial in range(25):
        K = int(rng.integers(2, 48))
        Cc = int(rng.integers(1, min(K, 7) + 1))
        L = int(rng.integers(1, 9))
        hist = rng.integers(0, 25, size=(K, L)) * (rng.random((K, L)) < 0.4)
        if hist.sum() == 0:
            hist[0, 0] = 1
        counts = hist.sum(1)
        assert np.array_equal(g.assign("label_jsd", K, Cc, 0, counts, hist),
                              assign_label_jsd(K, Cc, counts, hist)[0]), trial
    with pytest.raises(g.GCPSLError) as e:
        g.assign("label_jsd", 4, 2, 0, np.zeros(4, np.int64), np.zeros((4, 3), np.int64))
    assert e.value.code == g.EINVAL


def test_fuse_replicas_rejects_bad_arguments_before_device_work():
    lib = g.lib()
    fake = C.c_void_p(1 << 20)  # never dereferenced: every case fails validation first
    w = np.array([3, 4, 5], dtype=np.int64)
    wp = w.ctypes.data_as(C.POINTER(C.c_int64))
    cases = [(None, 3, 10, wp), (fake, 0, 10, wp), (fake, 65, 10, wp), (fake, 3, 0, wp), (fake, 3, 10, None),
             (C.c_void_p((1 << 20) + 2), 3, 10, wp)]
    for th, Cc, P, ww in cases:
        assert lib.gcpsl_fuse_replicas(th, Cc, P, ww, None) == g.EINVAL, (Cc, P)
    for bad in ([3, -1, 5], [0, 0, 0], [1, 1 << 30, 1]):
        b = np.array(bad, dtype=np.int64)
        rc = lib.gcpsl_fuse_replicas(fake, 3, 10, b.ctypes.data_as(C.POINTER(C.c_int64)), None)
        assert rc == g.EINVAL, bad
        assert "weights" in lib.gcpsl_last_error().decode()


@pytest.mark.parametrize("argv, env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}), ([], {"WORLD_SIZE": "2"})])
def test_bench_refuses_more_than_one_gpu(argv, env):
    """bench.py measures one GPU; asked for more it exits with status 2 and a
    message before touching a device."""
    import subprocess
    import sys
    e = dict(os.environ, **env)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv, "--steps", "1", "--warmup", "0"],
                       capture_output=True, text=True, timeout=120, env=e, cwd=ROOT)
    assert r.returncode == 2 and "one GPU only" in r.stderr and r.stdout == ""
