"""ctypes binding of libgcpsl.so (include/gcpsl.h): argument marshalling only.

Every computation of the hot path runs in the library's HIP kernels.  PyTorch
is used for device memory (the caller-owned buffers the C ABI works in) and
for the stream handle.  If the library has not been built, every entry point
raises; there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgcpsl.so")

OK, EINVAL, ESTATE, EHIP, EUNSUPPORTED = 0, -1, -2, -3, -4
RULES = {"random": 0, "size": 1, "label_l1": 2, "label_jsd": 3}
DTYPES = {"f32": 0, "bf16": 1}
CONV3X3, MAXPOOL2, AVGPOOL, LINEAR, BATCHNORM, GROUPNORM, BLOCK = 1, 2, 3, 4, 5, 6, 7
RESIDUAL, STRIDE2 = 1, 2
SCHEDULES = {"lockstep": 0, "epoch": 1}
PAYLOAD = ("activations", "cut_grads", "client_grads", "client_model", "fusion")  # GCPSL_PAYLOAD_* order

EXPORTS = ["gcpsl_param_count", "gcpsl_state_count", "gcpsl_workspace_bytes", "gcpsl_assign", "gcpsl_create",
           "gcpsl_create_static",
           "gcpsl_sample", "gcpsl_step", "gcpsl_step_replica", "gcpsl_epoch_rounds", "gcpsl_fuse",
           "gcpsl_fuse_replicas", "gcpsl_fuse_partial", "gcpsl_fuse_finalise",
           "gcpsl_participation", "gcpsl_batch_deviation", "gcpsl_payload",
           "gcpsl_cluster_sizes", "gcpsl_tensor", "gcpsl_timing", "gcpsl_timing_read",
           "gcpsl_destroy", "gcpsl_last_error"]


class GCPSLError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"gcpsl error {code}: {msg}")
        self.code = code


class Layer(C.Structure):
    _fields_ = [("kind", C.c_int32), ("cin", C.c_int32), ("cout", C.c_int32), ("flags", C.c_int32),
                ("groups", C.c_int32)]


class Desc(C.Structure):
    _fields_ = [
        ("K", C.c_int32), ("C", C.c_int32), ("B", C.c_int32), ("L", C.c_int32),
        ("H", C.c_int32), ("W", C.c_int32), ("Cin", C.c_int32), ("dtype", C.c_int32),
        ("n_examples", C.c_int64), ("n_layers", C.c_int32), ("cut", C.c_int32),
        ("layers", C.POINTER(Layer)), ("lr", C.c_float), ("momentum", C.c_float),
        ("weight_decay", C.c_float), ("nesterov", C.c_int32), ("label_smoothing", C.c_float),
        ("seed", C.c_uint64), ("max_steps", C.c_int64), ("max_window", C.c_int32),
        ("schedule", C.c_int32), ("client_of_example", C.POINTER(C.c_int32)),
        ("cluster_of_client", C.POINTER(C.c_int32)), ("images", C.c_void_p),
        ("labels", C.c_void_p), ("theta", C.c_void_p), ("momentum_buf", C.c_void_p), ("norm_state", C.c_void_p),
        ("workspace", C.c_void_p), ("workspace_bytes", C.c_size_t),
    ]


class KernelStat(C.Structure):
    _fields_ = [("name", C.c_char * 64), ("launches", C.c_int64), ("ms", C.c_double),
                ("flops", C.c_double), ("bytes", C.c_double)]


_lib = None


def lib():
    """Load libgcpsl.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2609_29395_amd.build`")
    L = C.CDLL(LIB_PATH)
    vp, i32, i64, u64 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64
    P = C.POINTER
    L.gcpsl_param_count.argtypes = [P(Desc), P(i64), P(i64)]
    L.gcpsl_state_count.argtypes = [P(Desc), P(i64)]
    L.gcpsl_workspace_bytes.argtypes = [P(Desc), P(C.c_size_t)]
    L.gcpsl_assign.argtypes = [i32, i32, i32, u64, P(i64), P(i64), i32, P(i32)]
    L.gcpsl_create.argtypes = [P(Desc), P(vp)]
    L.gcpsl_create_static.argtypes = [P(Desc), P(vp)]
    L.gcpsl_sample.argtypes = [vp, i64, i32, vp, vp]
    L.gcpsl_step.argtypes = [vp, i64, vp, vp]
    L.gcpsl_step_replica.argtypes = [vp, i64, i32, vp, vp]
    L.gcpsl_epoch_rounds.argtypes = [vp, P(i64), P(i64)]
    L.gcpsl_fuse.argtypes = [vp, vp]
    L.gcpsl_fuse_replicas.argtypes = [vp, i32, i64, P(i64), vp]
    L.gcpsl_fuse_partial.argtypes = [vp, vp, vp]
    L.gcpsl_fuse_finalise.argtypes = [vp, vp, i64, vp]
    L.gcpsl_participation.argtypes = [vp, P(i64), P(i64), P(i32)]
    L.gcpsl_batch_deviation.argtypes = [vp, P(i64), P(i64), P(i64), P(i64)]
    L.gcpsl_payload.argtypes = [vp, P(i64)]
    L.gcpsl_cluster_sizes.argtypes = [vp, P(i64)]
    L.gcpsl_tensor.argtypes = [vp, C.c_char_p, P(vp), P(i64), P(i32)]
    L.gcpsl_timing.argtypes = [vp, i32]
    L.gcpsl_timing_read.argtypes = [vp, P(KernelStat), i32, P(i32)]
    L.gcpsl_destroy.argtypes = [vp]
    L.gcpsl_destroy.restype = None
    L.gcpsl_last_error.restype = C.c_char_p
    for name in EXPORTS:
        if name not in ("gcpsl_destroy", "gcpsl_last_error"):
            getattr(L, name).restype = C.c_int
    _lib = L
    return L


def _check(rc):
    if rc != OK:
        raise GCPSLError(rc, lib().gcpsl_last_error().decode())


def _i32p(a):
    return a.ctypes.data_as(C.POINTER(C.c_int32))


def _i64p(a):
    return a.ctypes.data_as(C.POINTER(C.c_int64))


def layers_struct(layers):
    arr = (Layer * len(layers))()
    for i, spec in enumerate(layers):
        kind = spec[0]
        if kind == "conv":
            arr[i] = Layer(CONV3X3, spec[1], spec[2], RESIDUAL if spec[3] else 0, 0)
        elif kind == "maxpool":
            arr[i] = Layer(MAXPOOL2, 0, 0, 0, 0)
        elif kind == "avgpool":
            arr[i] = Layer(AVGPOOL, 0, 0, 0, 0)
        elif kind == "linear":
            arr[i] = Layer(LINEAR, spec[1], spec[2], 0, 0)
        elif kind == "bnorm":
            arr[i] = Layer(BATCHNORM, spec[1], spec[1], 0, 0)
        elif kind == "gnorm":
            arr[i] = Layer(GROUPNORM, spec[1], spec[1], 0, spec[2])
        elif kind == "block":
            if spec[3] not in (1, 2):
                raise ValueError("block stride must be 1 or 2")
            arr[i] = Layer(BLOCK, spec[1], spec[2], STRIDE2 if spec[3] == 2 else 0, spec[4])
        else:
            raise ValueError(kind)
    return arr


def assign(rule, K, C_, seed, counts=None, hist=None):
    """gcpsl_assign: Alg. 1 cluster_of_client (host)."""
    out = np.zeros(K, dtype=np.int32)
    cnt = None if counts is None else np.ascontiguousarray(counts, dtype=np.int64)
    h = None if hist is None else np.ascontiguousarray(hist, dtype=np.int64)
    L = 0 if h is None else h.shape[1]
    _check(lib().gcpsl_assign(K, C_, RULES[rule] if isinstance(rule, str) else rule, seed,
                              None if cnt is None else _i64p(cnt), None if h is None else _i64p(h),
                              L, _i32p(out)))
    return out


def fuse_replicas(theta, weights, stream=None):
    """gcpsl_fuse_replicas: Eq. 5 in place on a [C][P] fp32 torch tensor on
    the GPU with host weights [C]."""
    if theta.dim() != 2 or theta.dtype.is_floating_point is False or theta.element_size() != 4:
        raise ValueError("theta must be a [C][P] fp32 tensor")
    if not theta.is_contiguous():
        raise ValueError("theta must be contiguous")
    w = np.ascontiguousarray(weights, dtype=np.int64)
    if w.shape != (theta.shape[0],):
        raise ValueError("weights must have one entry per replica")
    _check(lib().gcpsl_fuse_replicas(C.c_void_p(theta.data_ptr()), theta.shape[0], theta.shape[1], _i64p(w),
                                     _stream(stream)))


def make_desc(cfg, client_of_example, cluster_of_client, max_steps=None, max_window=1, schedule="lockstep"):
    """Host part of gcpsl_desc for a workload (device pointers filled by Context)."""
    d = Desc()
    d.K, d.C, d.B, d.L = cfg["K"], cfg["C"], cfg["B"], cfg["L"]
    d.H, d.W, d.Cin = cfg["H"], cfg["W"], cfg["Cin"]
    d.dtype = DTYPES[cfg["dtype"]]
    d.n_examples = cfg["N_ex"]
    keep = {"layers": layers_struct(cfg["layers"]),
            "coe": np.ascontiguousarray(client_of_example, dtype=np.int32),
            "coc": np.ascontiguousarray(cluster_of_client, dtype=np.int32)}
    d.n_layers = len(cfg["layers"])
    d.cut = cfg["cut"]
    d.layers = C.cast(keep["layers"], C.POINTER(Layer))
    d.lr, d.momentum = cfg["lr"], cfg["momentum"]
    d.weight_decay = cfg.get("weight_decay", 0.0)
    d.nesterov = 1 if cfg.get("nesterov", False) else 0
    d.label_smoothing = cfg.get("label_smoothing", 0.0)
    d.seed = cfg["seed"]
    d.max_steps = max_steps if max_steps is not None else cfg["T"]
    d.max_window = max_window
    d.schedule = SCHEDULES[schedule]
    d.client_of_example = _i32p(keep["coe"])
    d.cluster_of_client = _i32p(keep["coc"])
    return d, keep


def param_count(desc):
    P, Pc = C.c_int64(), C.c_int64()
    _check(lib().gcpsl_param_count(C.byref(desc), C.byref(P), C.byref(Pc)))
    return P.value, Pc.value


def state_count(desc):
    S = C.c_int64()
    _check(lib().gcpsl_state_count(C.byref(desc), C.byref(S)))
    return S.value


def workspace_bytes(desc):
    n = C.c_size_t()
    _check(lib().gcpsl_workspace_bytes(C.byref(desc), C.byref(n)))
    return n.value


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


class Context:
    """One gcpsl_ctx with the caller-owned device buffers it works in."""

    def __init__(self, cfg, images, labels, client_of_example, cluster_of_client, theta0,
                 max_steps=None, max_window=1, device="cuda", schedule="lockstep", norm_state0=None,
                 static=False):
        """static: gcpsl_create_static (the library's own workspace, no
        workspace tensor here; `tensor` is then unavailable)."""
        import torch
        self.cfg = cfg
        self.schedule = schedule
        desc, self._keep = make_desc(cfg, client_of_example, cluster_of_client, max_steps, max_window, schedule)
        self.P, self.P_client = param_count(desc)
        t0 = torch.as_tensor(np.asarray(theta0, dtype=np.float32))
        if t0.numel() != self.P:
            raise ValueError(f"theta0 has {t0.numel()} entries, the model has {self.P}")
        self.images = torch.from_numpy(np.array(images, dtype=np.float32)).to(device)
        self.labels = torch.from_numpy(np.array(labels, dtype=np.int32)).to(device)
        self.theta = t0.to(device).reshape(1, -1).repeat(cfg["C"], 1).contiguous()
        self.mom = torch.zeros_like(self.theta)
        self.S = state_count(desc)
        ns0 = np.zeros(self.S, dtype=np.float32) if norm_state0 is None else np.asarray(norm_state0, np.float32)
        if ns0.size != self.S:
            raise ValueError(f"norm_state0 has {ns0.size} entries, the model has {self.S}")
        self.norm_state = (torch.as_tensor(ns0).to(device).reshape(1, -1).repeat(cfg["C"], 1).contiguous()
                           if self.S else None)
        desc.images = self.images.data_ptr()
        desc.labels = self.labels.data_ptr()
        desc.theta = self.theta.data_ptr()
        desc.momentum_buf = self.mom.data_ptr()
        desc.norm_state = self.norm_state.data_ptr() if self.S else None
        self.static = static
        if static:
            self.workspace = None
            desc.workspace, desc.workspace_bytes = None, 0
        else:
            nbytes = workspace_bytes(desc)
            self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
            base = self.workspace.data_ptr()
            desc.workspace = base + (-base) % 256
            desc.workspace_bytes = nbytes
        self.desc = desc
        h = C.c_void_p()
        create = lib().gcpsl_create_static if static else lib().gcpsl_create
        _check(create(C.byref(desc), C.byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().gcpsl_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def sample(self, step, nsteps=1, idx_out=None, stream=None):
        ptr = None if idx_out is None else C.c_void_p(idx_out.data_ptr())
        _check(lib().gcpsl_sample(self._h, step, nsteps, ptr, _stream(stream)))

    def step(self, step, loss_out=None, stream=None):
        ptr = None if loss_out is None else C.c_void_p(loss_out.data_ptr())
        _check(lib().gcpsl_step(self._h, step, ptr, _stream(stream)))

    def step_replica(self, step, replica, loss_out=None, stream=None):
        ptr = None if loss_out is None else C.c_void_p(loss_out.data_ptr())
        _check(lib().gcpsl_step_replica(self._h, step, replica, ptr, _stream(stream)))

    def epoch_rounds(self):
        """(r_n per cluster, R = slots of a system epoch) of the epoch schedule."""
        out = np.zeros(self.cfg["C"], dtype=np.int64)
        R = C.c_int64()
        _check(lib().gcpsl_epoch_rounds(self._h, _i64p(out), C.byref(R)))
        return out, R.value

    def fuse(self, stream=None):
        _check(lib().gcpsl_fuse(self._h, _stream(stream)))

    def fuse_partial(self, partial, stream=None):
        """gcpsl_fuse_partial into a device fp64 tensor of P + S entries."""
        if partial.numel() != self.P + self.S or partial.element_size() != 8 or not partial.is_contiguous():
            raise ValueError("partial must be a contiguous fp64 tensor of P + S entries")
        _check(lib().gcpsl_fuse_partial(self._h, C.c_void_p(partial.data_ptr()), _stream(stream)))

    def fuse_finalise(self, partial, W, stream=None):
        """gcpsl_fuse_finalise from a device fp64 tensor of P + S entries."""
        if partial.numel() != self.P + self.S or partial.element_size() != 8 or not partial.is_contiguous():
            raise ValueError("partial must be a contiguous fp64 tensor of P + S entries")
        _check(lib().gcpsl_fuse_finalise(self._h, C.c_void_p(partial.data_ptr()), int(W), _stream(stream)))

    def batch_deviation(self):
        """(sum of numerators, batches, denominator B |D|, per-step numerators
        [T_h][C] with -1 where no batch was drawn) of Sec. V-E's batch
        deviation (synchronises)."""
        sn, nb, den = C.c_int64(), C.c_int64(), C.c_int64()
        per = np.zeros((self.desc.max_steps, self.cfg["C"]), dtype=np.int64)
        _check(lib().gcpsl_batch_deviation(self._h, C.byref(sn), C.byref(nb), C.byref(den), _i64p(per)))
        T = self.participation()[1] // self.cfg["K"]
        return sn.value, nb.value, den.value, per[:T]

    def payload(self):
        """{category: bytes} of Sec. V-E's logical payload (synchronises)."""
        out = np.zeros(len(PAYLOAD), dtype=np.int64)
        _check(lib().gcpsl_payload(self._h, _i64p(out)))
        return {k: int(v) for k, v in zip(PAYLOAD, out)}

    def participation(self):
        a, t = C.c_int64(), C.c_int64()
        T = self.desc.max_steps
        per = np.zeros((T, self.cfg["C"]), dtype=np.int32)
        _check(lib().gcpsl_participation(self._h, C.byref(a), C.byref(t), _i32p(per)))
        steps = t.value // self.cfg["K"] if self.cfg["K"] else 0
        return a.value, t.value, per[:steps]

    def cluster_sizes(self):
        out = np.zeros(self.cfg["C"], dtype=np.int64)
        _check(lib().gcpsl_cluster_sizes(self._h, _i64p(out)))
        return out

    def timing(self, on):
        _check(lib().gcpsl_timing(self._h, 1 if on else 0))

    def timing_read(self, cap=64):
        """{kernel: dict(launches, ms, flops, bytes)} of the launches recorded
        since the last read (synchronises)."""
        arr = (KernelStat * cap)()
        n = C.c_int32()
        _check(lib().gcpsl_timing_read(self._h, arr, cap, C.byref(n)))
        return {arr[i].name.decode(): dict(launches=arr[i].launches, ms=arr[i].ms, flops=arr[i].flops,
                                           bytes=arr[i].bytes) for i in range(min(n.value, cap))}

    def tensor(self, name):
        """torch view of a named workspace tensor (gcpsl_tensor)."""
        import torch
        if self.workspace is None:
            raise ValueError("a static context's workspace is the library's own; it has no tensor view")
        ptr, n, dt = C.c_void_p(), C.c_int64(), C.c_int32()
        _check(lib().gcpsl_tensor(self._h, name.encode(), C.byref(ptr), C.byref(n), C.byref(dt)))
        tdt = {0: torch.float32, 1: torch.bfloat16, -1: torch.int32, -2: torch.uint8}[dt.value]
        esz = torch.tensor([], dtype=tdt).element_size()
        off = ptr.value - self.workspace.data_ptr()
        return self.workspace[off:off + n.value * esz].view(tdt)
