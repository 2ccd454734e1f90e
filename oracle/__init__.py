"""TEST INFRASTRUCTURE ONLY: ctypes front end of the CPU oracle.

Only tests/, the smoke check and the benchmark's CPU-baseline leg may import
this package.  The product path (the HIP library and its binding) never does.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# A test may point the oracle at another build of its source (mutation tests).
LIB_PATH = os.environ.get("EPROP_ORACLE_LIB") or os.path.join(HERE, "liboracle.so")


class OracleConfig(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("batch", ctypes.c_int32), ("n_in", ctypes.c_int32),
        ("n_rec", ctypes.c_int32), ("n_out", ctypes.c_int32), ("recurrent", ctypes.c_int32),
        ("n_adaptive", ctypes.c_int32),
        ("alpha", ctypes.c_double), ("rho", ctypes.c_double), ("kappa", ctypes.c_double),
        ("thr", ctypes.c_double), ("beta", ctypes.c_double), ("gamma", ctypes.c_double),
        ("reset", ctypes.c_double),
        ("fwd_fp32", ctypes.c_int32), ("smooth", ctypes.c_int32),
        ("reset_through", ctypes.c_int32),
        ("model", ctypes.c_int32), ("alpha_d", ctypes.c_double), ("coupling", ctypes.c_double),
        ("bap", ctypes.c_double),
    ]


class OracleRecord(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("v", "a", "psi", "L", "z", "y")]


_lib = None


def load(path: str = LIB_PATH):
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        from . import build as _b
        _b.build(out=path)
    lib = ctypes.CDLL(path)
    lib.oracle_eprop_run.restype = ctypes.c_int
    lib.oracle_eprop_run.argtypes = [
        ctypes.POINTER(OracleConfig), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
        ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p,
    ]
    lib.oracle_eprop_run_fb.restype = ctypes.c_int
    lib.oracle_eprop_run_fb.argtypes = [
        ctypes.POINTER(OracleConfig), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p,
    ]
    lib.oracle_eprop_run_online.restype = ctypes.c_int
    lib.oracle_eprop_run_online.argtypes = [
        ctypes.POINTER(OracleConfig), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_int32, ctypes.c_void_p, ctypes.c_double, ctypes.c_int32, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.oracle_eprop_run_online_fb.restype = ctypes.c_int
    lib.oracle_eprop_run_online_fb.argtypes = [
        ctypes.POINTER(OracleConfig), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_double, ctypes.c_int32,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p]
    lib.oracle_state_bytes.restype = ctypes.c_size_t
    lib.oracle_state_bytes.argtypes = [ctypes.POINTER(OracleConfig), ctypes.c_int32]
    if path == LIB_PATH:
        _lib = lib
    return lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def make_config(shape, fwd_fp32: bool = True, smooth: bool = False,
                reset: Optional[float] = None, **over) -> OracleConfig:
    """Oracle config from an EpropShape (any object with the same fields)."""
    c = OracleConfig()
    c.n_layers, c.batch, c.n_in, c.n_rec = shape.n_layers, shape.batch, shape.n_in, shape.n_rec
    c.n_out, c.recurrent, c.n_adaptive = shape.n_out, shape.recurrent, shape.n_adaptive
    c.alpha, c.rho, c.kappa = shape.alpha, shape.rho, shape.kappa
    c.thr, c.beta, c.gamma = shape.thr, shape.beta, shape.gamma
    c.reset = shape.thr if reset is None else reset
    c.fwd_fp32, c.smooth = int(fwd_fp32), int(smooth)
    c.reset_through = int(getattr(shape, "reset_grad", 0))
    c.model = int(getattr(shape, "neuron_model", 0))
    c.alpha_d = float(getattr(shape, "alpha_d", 0.0))
    c.coupling = float(getattr(shape, "coupling", 0.0))
    c.bap = float(getattr(shape, "bap", 0.0))
    for k, v in over.items():
        setattr(c, k, v)
    return c


@dataclass
class OracleResult:
    dW: list            # per layer fp64 [n_rec, n_pre] (all synapses) or [n_sample] (sampled)
    dWout: list         # per layer fp64 [n_out, n_rec]
    loss: float
    spikes: Optional[np.ndarray]  # uint32 [T, L, B, ceil(n_rec/32)]
    record: Optional[dict]


def run(shape, W: Sequence[np.ndarray], Wout: Sequence[np.ndarray], x: np.ndarray,
        labels: np.ndarray, *, T: Optional[int] = None, b_lo: int = 0, b_hi: Optional[int] = None,
        sample: Optional[np.ndarray] = None, want_spikes: bool = True, want_record: bool = False,
        fwd_fp32: bool = True, smooth: bool = False, reset: Optional[float] = None,
        spikes_out: Optional[np.ndarray] = None, lib_path: str = LIB_PATH,
        feedback: Optional[Sequence[np.ndarray]] = None, **over) -> OracleResult:
    """Runs the oracle on batch elements [b_lo, b_hi).  ``sample`` is an int32
    array of (layer, j, i) rows; when given, only those synapses' gradients are
    computed (returned as dW[0] of length len(sample)).  ``spikes_out``, if
    given, is the uint32 [T, L, B, ceil(n_rec/32)] record to write into.
    ``feedback``: per layer the fixed matrix B [n_out, n_rec] of the learning
    signal L = B^T delta (None: W_out)."""
    lib = load(lib_path)
    cfg = make_config(shape, fwd_fp32=fwd_fp32, smooth=smooth, reset=reset, **over)
    T = x.shape[0] if T is None else T
    b_hi = shape.batch if b_hi is None else b_hi
    L, N, K, B = shape.n_layers, shape.n_rec, shape.n_out, shape.batch
    Wc = [np.ascontiguousarray(w, dtype=np.float32) for w in W]
    Woc = [np.ascontiguousarray(w, dtype=np.float32) for w in Wout]
    xc = np.ascontiguousarray(x, dtype=np.uint8)
    lab = np.ascontiguousarray(labels, dtype=np.int32)
    assert xc.shape[0] >= T and xc.shape[1] == B and xc.shape[2] == shape.n_in
    Wp = (ctypes.c_void_p * L)(*[_ptr(w) for w in Wc])
    Wop = (ctypes.c_void_p * L)(*[_ptr(w) for w in Woc])
    if sample is None:
        dW = [np.zeros(w.shape, dtype=np.float64) for w in Wc]
        smp_ptr, n_sample = None, -1
    else:
        smp = np.ascontiguousarray(sample, dtype=np.int32).reshape(-1, 3)
        dW = [np.zeros(len(smp), dtype=np.float64)]
        smp_ptr, n_sample = _ptr(smp), len(smp)
    dWp = (ctypes.c_void_p * len(dW))(*[_ptr(d) for d in dW])
    dWout = [np.zeros((K, N), dtype=np.float64) for _ in range(L)]
    dWop = (ctypes.c_void_p * L)(*[_ptr(d) for d in dWout])
    loss = np.zeros(1, dtype=np.float64)
    spikes = None
    if spikes_out is not None:
        assert spikes_out.shape == (T, L, B, (N + 31) // 32) and spikes_out.dtype == np.uint32
        assert spikes_out.flags.c_contiguous
        spikes = spikes_out
    elif want_spikes:
        spikes = np.zeros((T, L, B, (N + 31) // 32), dtype=np.uint32)
    rec = None
    recs = None
    if want_record:
        recs = {k: np.zeros((T, L, B, N)) for k in ("v", "a", "psi", "L", "z")}
        recs["y"] = np.zeros((T, L, B, K))
        rec = OracleRecord(*[_ptr(recs[k]) for k in ("v", "a", "psi", "L", "z", "y")])
    Fbp = None
    if feedback is not None:
        Fbc = [np.ascontiguousarray(f, dtype=np.float32) for f in feedback]
        assert len(Fbc) == L and all(f.shape == (K, N) for f in Fbc)
        Fbp = (ctypes.c_void_p * L)(*[_ptr(f) for f in Fbc])
    rc = lib.oracle_eprop_run_fb(ctypes.byref(cfg), ctypes.cast(Wp, ctypes.c_void_p),
                                 ctypes.cast(Wop, ctypes.c_void_p),
                                 ctypes.cast(Fbp, ctypes.c_void_p) if Fbp is not None else None,
                                 _ptr(xc), T, _ptr(lab), b_lo, b_hi, smp_ptr, n_sample,
                                 _ptr(spikes) if spikes is not None else None,
                                 ctypes.cast(dWp, ctypes.c_void_p),
                                 ctypes.cast(dWop, ctypes.c_void_p),
                                 _ptr(loss), ctypes.byref(rec) if rec is not None else None)
    if rc != 0:
        raise ValueError(f"oracle_eprop_run returned {rc}")
    return OracleResult(dW=dW, dWout=dWout, loss=float(loss[0]), spikes=spikes, record=recs)


@dataclass
class OnlineResult:
    dW: list            # per layer fp64 [n_rec, n_pre]: the gradient of the whole run
    dWout: list         # per layer fp64 [n_out, n_rec]
    loss: float
    spikes: np.ndarray  # uint32 [T, L, B, ceil(n_rec/32)]
    W: list             # per layer fp32: the drive weights in use at the end
    Wout: list          # per layer fp32: the readout weights in use at the end


def run_online(shape, W: Sequence[np.ndarray], Wout: Sequence[np.ndarray], x: np.ndarray,
               labels: np.ndarray, lr: float, every: int, *, T: Optional[int] = None,
               fwd_fp32: bool = True, lib_path: str = LIB_PATH,
               feedback: Optional[Sequence[np.ndarray]] = None, **over) -> OnlineResult:
    """Every batch element, every synapse, with online weight application:
    every ``every`` steps the weights in use become W0 - lr * (gradient so
    far) on the 2**-14 grid (oracle_eprop_run_online_fb).  ``feedback``: per
    layer a fixed matrix B of the learning signal (None: the readout weights
    in use); it does not change with the weights."""
    lib = load(lib_path)
    cfg = make_config(shape, fwd_fp32=fwd_fp32, **over)
    T = x.shape[0] if T is None else T
    L, N, K, B = shape.n_layers, shape.n_rec, shape.n_out, shape.batch
    Wc = [np.ascontiguousarray(w, dtype=np.float32) for w in W]
    Woc = [np.ascontiguousarray(w, dtype=np.float32) for w in Wout]
    xc = np.ascontiguousarray(x, dtype=np.uint8)
    lab = np.ascontiguousarray(labels, dtype=np.int32)
    assert xc.shape[0] >= T and xc.shape[1] == B and xc.shape[2] == shape.n_in
    dW = [np.zeros(w.shape, dtype=np.float64) for w in Wc]
    dWout = [np.zeros((K, N), dtype=np.float64) for _ in range(L)]
    Wf = [np.empty_like(w) for w in Wc]
    Wof = [np.empty_like(w) for w in Woc]
    loss = np.zeros(1, dtype=np.float64)
    spikes = np.zeros((T, L, B, (N + 31) // 32), dtype=np.uint32)
    arr = lambda xs: ctypes.cast((ctypes.c_void_p * len(xs))(*[_ptr(a) for a in xs]), ctypes.c_void_p)
    fbp = None
    if feedback is not None:
        # a None entry: that layer's learning signal through its readout weights in use
        Fbc = [None if f is None else np.ascontiguousarray(f, dtype=np.float32) for f in feedback]
        assert len(Fbc) == L and all(f is None or f.shape == (K, N) for f in Fbc)
        fbp = ctypes.cast((ctypes.c_void_p * L)(*[None if f is None else _ptr(f) for f in Fbc]),
                          ctypes.c_void_p)
    rc = lib.oracle_eprop_run_online_fb(ctypes.byref(cfg), arr(Wc), arr(Woc), fbp, _ptr(xc), T,
                                        _ptr(lab), float(lr), int(every), _ptr(spikes), arr(dW),
                                        arr(dWout), _ptr(loss), arr(Wf), arr(Wof))
    if rc != 0:
        raise ValueError(f"oracle_eprop_run_online returned {rc}")
    return OnlineResult(dW=dW, dWout=dWout, loss=float(loss[0]), spikes=spikes, W=Wf, Wout=Wof)


def state_bytes(shape, n_sample: int = -1, fwd_fp32: bool = True) -> int:
    return int(load().oracle_state_bytes(ctypes.byref(make_config(shape, fwd_fp32)), n_sample))


_SHARD_ARGS = None


def _shard(bounds):
    lo, hi = bounds
    shape, W, Wout, x, labels, T, sample, spikes, kw = _SHARD_ARGS
    # Each shard writes its own batch rows of the shared spike record.
    res = run(shape, W, Wout, x, labels, T=T, b_lo=lo, b_hi=hi, sample=sample,
              want_spikes=False, spikes_out=spikes, **kw)
    return res.dW, res.dWout, res.loss


def run_sharded(shape, W, Wout, x, labels, *, workers: int, T: Optional[int] = None,
                sample: Optional[np.ndarray] = None, want_spikes: bool = True,
                **kw) -> OracleResult:
    """The same result as ``run`` over the whole batch, computed as independent
    single-threaded oracle runs on contiguous batch shards in forked worker
    processes.  The gradient is a sum over batch elements; the shards' fp64
    partial sums are added in shard order.  Each shard writes its own batch rows
    of a spike record shared between the processes."""
    import mmap
    import multiprocessing as mp
    global _SHARD_ARGS
    B, L, N = shape.batch, shape.n_layers, shape.n_rec
    T = x.shape[0] if T is None else T
    workers = max(1, min(workers, B))
    edges = [B * k // workers for k in range(workers + 1)]
    bounds = [(edges[k], edges[k + 1]) for k in range(workers) if edges[k + 1] > edges[k]]
    spikes = None
    if want_spikes:
        shp = (T, L, B, (N + 31) // 32)
        buf = mmap.mmap(-1, max(1, int(np.prod(shp)) * 4))
        spikes = np.frombuffer(buf, dtype=np.uint32, count=int(np.prod(shp))).reshape(shp)
    _SHARD_ARGS = (shape, W, Wout, x, labels, T, sample, spikes, kw)
    try:
        if len(bounds) == 1:
            parts = [_shard(bounds[0])]
        else:
            ctx = mp.get_context("fork")
            with ctx.Pool(len(bounds)) as pool:
                parts = pool.map(_shard, bounds)
    finally:
        _SHARD_ARGS = None
    dW, dWout, loss = parts[0]
    for pdW, pdWout, ploss in parts[1:]:
        for l in range(len(dW)):
            dW[l] += pdW[l]
        for l in range(len(dWout)):
            dWout[l] += pdWout[l]
        loss += ploss
    return OracleResult(dW=dW, dWout=dWout, loss=loss,
                        spikes=None if spikes is None else np.array(spikes), record=None)
