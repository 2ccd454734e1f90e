"""Thin ctypes binding of the e-prop C ABI (include/eprop.h).

Argument marshalling only: every step of the hot path runs in the HIP kernels
of libeprop.so.  PyTorch supplies device memory (the workspace, inputs and
outputs are CUDA/HIP tensors) and the current stream.  There is no CPU
fallback: without the built library or a GPU the calls raise.  EPROP_LIB
names another build of the same library (for comparing kernel variants).
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence, Tuple

import torch

LIB_PATH = os.environ.get("EPROP_LIB") or \
    os.path.join(os.path.dirname(os.path.abspath(__file__)), "libeprop.so")

EPROP_OK, EPROP_EINVAL, EPROP_ENOSPACE, EPROP_EDEVICE, EPROP_ESTATE = 0, -1, -2, -3, -4
EPROP_SPLIT_AUTO, EPROP_SPLIT_EQUAL = 0, 1

# Every function the header declares, in declaration order.
SYMBOLS = (
    "eprop_neuron_coefficients", "eprop_workspace_bytes", "eprop_init", "eprop_step", "eprop_run_sequence",
    "eprop_set_block_split", "eprop_block_lengths", "eprop_get_grads",
    "eprop_reset", "eprop_status", "eprop_set_feedback", "eprop_set_online", "eprop_get_weights",
    "eprop_destroy", "eprop_sequence_static", "eprop_last_error",
    "eprop_profile_begin", "eprop_profile_end", "eprop_debug_buffer",
)


class eprop_config(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("batch", ctypes.c_int32), ("n_in", ctypes.c_int32),
        ("n_rec", ctypes.c_int32), ("n_out", ctypes.c_int32), ("recurrent", ctypes.c_int32),
        ("n_adaptive", ctypes.c_int32),
        ("alpha", ctypes.c_float), ("rho", ctypes.c_float), ("kappa", ctypes.c_float),
        ("thr", ctypes.c_float), ("beta", ctypes.c_float), ("gamma", ctypes.c_float),
        ("reset_grad", ctypes.c_int32),
        ("neuron_model", ctypes.c_int32), ("alpha_d", ctypes.c_float), ("coupling", ctypes.c_float),
        ("bap", ctypes.c_float),
    ]


class EpropError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"e-prop error {code}: {msg}")
        self.code = code


_lib = None


def load_library(path: str = LIB_PATH):
    """Loads libeprop.so; raises if it was not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2501_11407_amd.build` (hipcc, gfx950)")
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    cfgp = ctypes.POINTER(eprop_config)
    sig = {
        "eprop_neuron_coefficients": (ctypes.c_int, [cfgp, i32, ctypes.POINTER(ctypes.c_float)]),
        "eprop_workspace_bytes": (ctypes.c_size_t, [cfgp]),
        "eprop_init": (ctypes.c_int, [cfgp, vp, ctypes.c_size_t, vp, vp, ctypes.POINTER(vp)]),
        "eprop_step": (ctypes.c_int, [vp, vp, vp, vp]),
        "eprop_run_sequence": (ctypes.c_int, [vp, vp, i32, vp, vp]),
        "eprop_set_block_split": (ctypes.c_int, [vp, i32]),
        "eprop_block_lengths": (ctypes.c_int, [cfgp, i32, i64, i32, i32, ctypes.POINTER(i32), i32]),
        "eprop_get_grads": (ctypes.c_int, [vp, vp, vp]),
        "eprop_reset": (ctypes.c_int, [vp]),
        "eprop_set_feedback": (ctypes.c_int, [vp, vp]),
        "eprop_set_online": (ctypes.c_int, [vp, ctypes.c_float, i32]),
        "eprop_get_weights": (ctypes.c_int, [vp, vp]),
        "eprop_status": (ctypes.c_int, [vp]),
        "eprop_destroy": (None, [vp]),
        "eprop_sequence_static": (ctypes.c_int, [cfgp, vp, vp, i32, vp, vp, vp, vp, vp]),
        "eprop_last_error": (ctypes.c_char_p, [vp]),
        "eprop_profile_begin": (ctypes.c_int, [vp, i32]),
        "eprop_profile_end": (ctypes.c_int, [vp, ctypes.POINTER(ctypes.c_double),
                                             ctypes.POINTER(i32), ctypes.POINTER(i64)]),
        "eprop_debug_buffer": (ctypes.c_int, [vp, i32, i32, ctypes.POINTER(vp),
                                              ctypes.POINTER(i64), ctypes.POINTER(i64)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype, fn.argtypes = res, args
    _lib = lib
    return lib


def make_config(shape) -> eprop_config:
    """C config from an EpropShape (or any object with the same fields)."""
    return eprop_config(shape.n_layers, shape.batch, shape.n_in, shape.n_rec, shape.n_out,
                        shape.recurrent, shape.n_adaptive, shape.alpha, shape.rho, shape.kappa,
                        shape.thr, shape.beta, shape.gamma, int(getattr(shape, "reset_grad", 0)),
                        int(getattr(shape, "neuron_model", 0)), float(getattr(shape, "alpha_d", 0.0)),
                        float(getattr(shape, "coupling", 0.0)), float(getattr(shape, "bap", 0.0)))


def eprop_neuron_coefficients(cfg: eprop_config, cls: int):
    """(A [2x2], b [2], r [2], c [2]) of the configured neuron model, derived
    by the library on the host."""
    out = (ctypes.c_float * 10)()
    _check(load_library().eprop_neuron_coefficients(ctypes.byref(cfg), int(cls), out))
    v = list(out)
    return [[v[0], v[1]], [v[2], v[3]]], v[4:6], v[6:8], v[8:10]


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _ptr_array(ts: Sequence[torch.Tensor]):
    return (ctypes.c_void_p * len(ts))(*[t.data_ptr() for t in ts])


def eprop_workspace_bytes(cfg: eprop_config) -> int:
    return int(load_library().eprop_workspace_bytes(ctypes.byref(cfg)))


def eprop_block_lengths(cfg: eprop_config, T: int, t0: int = 0, online_every: int = 0,
                        mode: int = 0) -> list:
    """Block lengths of a run_sequence call of T steps, t0 steps after the
    last reset (host only)."""
    lib = load_library()
    n = lib.eprop_block_lengths(ctypes.byref(cfg), int(T), int(t0), int(online_every), int(mode), None, 0)
    _check(min(n, 0))
    out = (ctypes.c_int32 * n)()
    lib.eprop_block_lengths(ctypes.byref(cfg), int(T), int(t0), int(online_every), int(mode), out, n)
    return list(out)


def eprop_last_error(ctx=None) -> str:
    return load_library().eprop_last_error(ctx).decode()


def _check(rc: int, ctx=None):
    if rc != EPROP_OK:
        raise EpropError(rc, eprop_last_error(ctx))


def eprop_init(cfg: eprop_config, workspace: torch.Tensor, weights: Sequence[torch.Tensor],
               stream: Optional[torch.cuda.Stream] = None):
    """weights: [W_0, Wout_0, (W_1, Wout_1)] fp32 contiguous device tensors."""
    lib = load_library()
    for w in weights:
        assert w.is_cuda and w.dtype == torch.float32 and w.is_contiguous()
    s = (stream or torch.cuda.current_stream()).cuda_stream
    ctx = ctypes.c_void_p()
    rc = lib.eprop_init(ctypes.byref(cfg), _ptr(workspace), workspace.numel(),
                        _ptr_array(weights), ctypes.c_void_p(s), ctypes.byref(ctx))
    _check(rc)
    return ctx


def eprop_step(ctx, x_t: torch.Tensor, labels: torch.Tensor, spikes_t: Optional[torch.Tensor] = None):
    _check(load_library().eprop_step(ctx, _ptr(x_t), _ptr(labels), _ptr(spikes_t)), ctx)


def eprop_run_sequence(ctx, x: torch.Tensor, T: int, labels: torch.Tensor,
                       spikes: Optional[torch.Tensor] = None):
    _check(load_library().eprop_run_sequence(ctx, _ptr(x), int(T), _ptr(labels), _ptr(spikes)), ctx)


def eprop_get_grads(ctx, grads: Sequence[torch.Tensor], loss: Optional[torch.Tensor] = None):
    _check(load_library().eprop_get_grads(ctx, _ptr_array(grads), _ptr(loss)), ctx)


def eprop_reset(ctx):
    _check(load_library().eprop_reset(ctx), ctx)


def eprop_set_feedback(ctx, feedback: Optional[Sequence[Optional[torch.Tensor]]]):
    """feedback: None, or per layer None or a device fp32 [n_out, n_rec] tensor."""
    arr = None
    if feedback is not None:
        arr = (ctypes.c_void_p * len(feedback))(*[_ptr(f) for f in feedback])
    _check(load_library().eprop_set_feedback(ctx, ctypes.cast(arr, ctypes.c_void_p)
                                             if arr is not None else None), ctx)


def eprop_set_block_split(ctx, mode: int):
    _check(load_library().eprop_set_block_split(ctx, int(mode)), ctx)


def eprop_set_online(ctx, lr: float, every: int):
    _check(load_library().eprop_set_online(ctx, float(lr), int(every)), ctx)


def eprop_get_weights(ctx, weights: Sequence[torch.Tensor]):
    """weights: per layer W then W_out, device fp32 tensors (written)."""
    arr = (ctypes.c_void_p * len(weights))(*[_ptr(w) for w in weights])
    _check(load_library().eprop_get_weights(ctx, ctypes.cast(arr, ctypes.c_void_p)), ctx)


def eprop_status(ctx) -> int:
    return int(load_library().eprop_status(ctx))


def eprop_destroy(ctx):
    load_library().eprop_destroy(ctx)


STATIC_SCRATCH_BYTES = 256 << 20      # EPROP_STATIC_SCRATCH_BYTES


def eprop_sequence_static(cfg: eprop_config, weights: Sequence[torch.Tensor], x: torch.Tensor, T: int,
                          labels: torch.Tensor, spikes: Optional[torch.Tensor],
                          grads: Sequence[torch.Tensor], loss: Optional[torch.Tensor] = None,
                          stream: Optional[torch.cuda.Stream] = None):
    """One sequence in the library's static scratch (no caller workspace):
    weights [W_0, Wout_0, ...] and grads [dW_0, dWout_0, ...] device fp32."""
    s = (stream or torch.cuda.current_stream()).cuda_stream
    rc = load_library().eprop_sequence_static(ctypes.byref(cfg), _ptr_array(weights), _ptr(x), int(T),
                                              _ptr(labels), _ptr(spikes), _ptr_array(grads), _ptr(loss),
                                              ctypes.c_void_p(s))
    _check(rc)


def eprop_profile_begin(ctx, max_launches: int):
    _check(load_library().eprop_profile_begin(ctx, int(max_launches)), ctx)


def eprop_profile_end(ctx) -> Tuple[float, int, int]:
    """(summed eligibility-kernel milliseconds, timed launches, timesteps they covered)"""
    ms, n, steps = ctypes.c_double(), ctypes.c_int32(), ctypes.c_int64()
    _check(load_library().eprop_profile_end(ctx, ctypes.byref(ms), ctypes.byref(n),
                                            ctypes.byref(steps)), ctx)
    return ms.value, n.value, steps.value


def eprop_debug_buffer(ctx, layer: int, which: int) -> Tuple[int, int, int]:
    ptr, cols, ld = ctypes.c_void_p(), ctypes.c_int64(), ctypes.c_int64()
    _check(load_library().eprop_debug_buffer(ctx, layer, which, ctypes.byref(ptr),
                                             ctypes.byref(cols), ctypes.byref(ld)), ctx)
    return ptr.value, cols.value, ld.value


class EpropContext:
    """One network on one GPU: workspace, borrowed weights and the C context.

    All work is queued on the stream that is current at construction.
    """

    DEBUG = {"v": 0, "a": 1, "psi": 2, "L": 3, "y": 4}

    def __init__(self, shape, W: Sequence, Wout: Sequence, device: str = "cuda"):
        if not torch.cuda.is_available():
            raise RuntimeError("no GPU visible: the e-prop library runs only on the GPU")
        self.shape = shape
        self.cfg = make_config(shape)
        self.device = torch.device(device)
        nbytes = eprop_workspace_bytes(self.cfg)
        if nbytes == 0:
            raise EpropError(EPROP_EINVAL, eprop_last_error())
        self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        off = (-self.workspace.data_ptr()) % 256
        self.workspace = self.workspace[off:off + nbytes]
        self.weights: List[torch.Tensor] = []
        for l in range(shape.n_layers):
            w = torch.as_tensor(W[l], dtype=torch.float32).to(self.device).contiguous()
            wo = torch.as_tensor(Wout[l], dtype=torch.float32).to(self.device).contiguous()
            if tuple(w.shape) != (shape.n_rec, shape.n_pre(l)):
                raise ValueError(f"W[{l}] must be {(shape.n_rec, shape.n_pre(l))}, got {tuple(w.shape)}")
            if tuple(wo.shape) != (shape.n_out, shape.n_rec):
                raise ValueError(f"Wout[{l}] must be {(shape.n_out, shape.n_rec)}, got {tuple(wo.shape)}")
            self.weights += [w, wo]
        self.stream = torch.cuda.current_stream(self.device)
        self.ctx = eprop_init(self.cfg, self.workspace, self.weights, self.stream)

    # -- host-side checks: every buffer a kernel touches has the shape it assumes
    def _check_dev(self, t, dtype, shape, what):
        if not (isinstance(t, torch.Tensor) and t.device.type == "cuda" and t.dtype == dtype
                and tuple(t.shape) == tuple(shape) and t.is_contiguous()):
            got = (tuple(t.shape), t.dtype, t.device) if isinstance(t, torch.Tensor) else type(t)
            raise ValueError(f"{what}: expected contiguous {dtype} {tuple(shape)} on the GPU, got {got}")

    def _check_step_args(self, x, T, labels, spikes):
        s = self.shape
        self._check_dev(x, torch.uint8, ((T,) if T is not None else ()) + (s.batch, s.n_in), "x")
        self._check_dev(labels, torch.int32, (s.batch,), "labels")
        if spikes is not None:
            w32 = (s.n_rec + 31) // 32
            self._check_dev(spikes, torch.int32,
                            ((T,) if T is not None else ()) + (s.n_layers, s.batch, w32), "spikes")

    # -- the C calls
    def step(self, x_t, labels, spikes_t=None):
        self._check_step_args(x_t, None, labels, spikes_t)
        eprop_step(self.ctx, x_t, labels, spikes_t)

    def run_sequence(self, x, labels, spikes=None):
        T = x.shape[0] if isinstance(x, torch.Tensor) and x.dim() == 3 else -1
        self._check_step_args(x, T, labels, spikes)
        eprop_run_sequence(self.ctx, x, T, labels, spikes)

    def get_grads(self):
        L, N, K = self.shape.n_layers, self.shape.n_rec, self.shape.n_out
        grads = []
        for l in range(L):
            grads.append(torch.empty(N, self.shape.n_pre(l), dtype=torch.float32, device=self.device))
            grads.append(torch.empty(K, N, dtype=torch.float32, device=self.device))
        loss = torch.empty(1, dtype=torch.float64, device=self.device)
        eprop_get_grads(self.ctx, grads, loss)
        return grads[0::2], grads[1::2], loss

    def reset(self):
        eprop_reset(self.ctx)

    def set_feedback(self, feedback: Optional[Sequence]):
        """Fixed feedback matrices B [n_out, n_rec] per layer for the learning
        signal L = B^T delta (None, or None for a layer: W_out).  The tensors
        are kept here for as long as they are set."""
        s = self.shape
        if feedback is None:
            self.feedback = None
        else:
            if len(feedback) != s.n_layers:
                raise ValueError(f"feedback needs {s.n_layers} entries")
            self.feedback = []
            for l, f in enumerate(feedback):
                if f is None:
                    self.feedback.append(None)
                    continue
                t = torch.as_tensor(f, dtype=torch.float32).to(self.device).contiguous()
                if tuple(t.shape) != (s.n_out, s.n_rec):
                    raise ValueError(f"feedback[{l}] must be {(s.n_out, s.n_rec)}, got {tuple(t.shape)}")
                self.feedback.append(t)
        eprop_set_feedback(self.ctx, self.feedback)

    def set_online(self, lr: float, every: int):
        """Online weight application: every ``every`` steps since the reset
        the weights in use become W0 - lr * G on the 2**-14 grid (0: off)."""
        eprop_set_online(self.ctx, lr, every)

    def set_block_split(self, mode: int):
        """EPROP_SPLIT_AUTO (default) or EPROP_SPLIT_EQUAL for later run_sequence calls."""
        eprop_set_block_split(self.ctx, mode)

    def get_weights(self):
        """The weights in use: (W list, W_out list) as new device tensors."""
        s = self.shape
        W = [torch.empty(s.n_rec, s.n_pre(l), dtype=torch.float32, device=self.device)
             for l in range(s.n_layers)]
        Wo = [torch.empty(s.n_out, s.n_rec, dtype=torch.float32, device=self.device)
              for _ in range(s.n_layers)]
        eprop_get_weights(self.ctx, [t for l in range(s.n_layers) for t in (W[l], Wo[l])])
        return W, Wo

    def status(self) -> int:
        return eprop_status(self.ctx)

    def profile_begin(self, max_launches: int):
        eprop_profile_begin(self.ctx, max_launches)

    def profile_end(self):
        return eprop_profile_end(self.ctx)

    def debug(self, name: str, layer: int = 0) -> torch.Tensor:
        """Copy of an internal per-neuron buffer [B, cols] after the last step."""
        ptr, cols, ld = eprop_debug_buffer(self.ctx, layer, self.DEBUG[name])
        off = ptr - self.workspace.data_ptr()
        rows = self.shape.batch
        flat = self.workspace[off:off + 4 * rows * ld].view(torch.float32)
        return flat.view(rows, ld)[:, :cols].clone()

    def integer_drive(self) -> bool:
        """Whether every drive weight is an int16 multiple of 2**-14, so that
        steps with few enough active inputs sum them as integers (else fp32 in
        ascending input order; both give the same result where the first
        applies)."""
        return self.integer_weights()[0]

    def integer_weights(self):
        """(every weight an int16 multiple of 2**-14, the largest |k|)."""
        ptr, _, _ = eprop_debug_buffer(self.ctx, 0, 5)
        off = ptr - self.workspace.data_ptr()
        torch.cuda.synchronize(self.device)
        v = self.workspace[off:off + 8].view(torch.int32).cpu().tolist()
        return bool(v[0]), int(v[1])

    # -- helpers
    def new_spike_buffer(self, T: Optional[int] = None) -> torch.Tensor:
        w32 = (self.shape.n_rec + 31) // 32
        shp = (self.shape.n_layers, self.shape.batch, w32)
        if T is not None:
            shp = (T,) + shp
        return torch.zeros(shp, dtype=torch.int32, device=self.device)

    def close(self):
        if getattr(self, "ctx", None) is not None:
            eprop_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
