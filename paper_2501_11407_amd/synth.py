"""Seeded synthetic workloads for the online e-prop step.

This module only draws inputs: presynaptic spike trains, weights and labels.
It holds none of the method's arithmetic, so both the HIP path and the CPU
oracle can be fed from it.

The workloads stand in for the spoken-digit spike data the paper trains on
(Sec. IV: 700 input channels, spiking hidden layer, non-spiking readout).
Inputs are Bernoulli spikes with one rate per channel, shared over batch and
time.

Weight quantisation: every weight is put on a grid of 2**-14 and clipped to
+-512/fan_in.  With binary presynaptic inputs, every partial sum of the drive
``sum_i W_ji p_i`` is then an integer multiple of 2**-14 below 2**9 in
magnitude.  Such sums are exact in fp32 in any summation order, so the spike
trains of two implementations that sum in different orders (sequential CPU
loop, MFMA tile) are identical.  The readout weights get the same treatment
with fan-in N_rec.  The change to the Gaussian draws is below 2**-15 and the
clip sits at 4.9 sigma or more.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np

GRID = 2.0 ** -14


def f32(v: float) -> float:
    """Round a Python float to the nearest fp32 value (returned as float)."""
    return float(np.float32(v))


@dataclasses.dataclass(frozen=True)
class EpropShape:
    """Network and sequence shape plus neuron constants.

    n_layers: 1, or 2 for a stack whose second layer is fed by the spikes of
      the first layer in the same step.
    recurrent: 0 means the presynaptic vector is the input alone.
    n_adaptive: neurons j < n_adaptive have an adaptive threshold (ALIF).
    reset_grad: 1 keeps the reset path (own spike -> own membrane) in the
      gradient; 0 (default) stops it.
    neuron_model: 0 LIF/ALIF; 1 a two-compartment neuron (a dendrite with
      decay alpha_d receiving the drive and the own spike times bap, a soma
      with decay alpha driven by the dendrite times coupling); n_adaptive
      must be 0 then.
    Constants are fp32-representable; both implementations use these exact
    values.
    """
    batch: int
    n_in: int
    n_rec: int
    n_out: int
    T: int
    n_layers: int = 1
    recurrent: int = 1
    n_adaptive: int = 0
    alpha: float = f32(math.exp(-1.0 / 20.0))
    rho: float = f32(math.exp(-1.0 / 200.0))
    kappa: float = f32(math.exp(-1.0 / 20.0))
    thr: float = 1.0
    beta: float = f32(1.8)
    gamma: float = f32(0.3)
    reset_grad: int = 0
    neuron_model: int = 0
    alpha_d: float = f32(math.exp(-1.0 / 10.0))
    coupling: float = f32(0.5)
    bap: float = f32(-0.5)
    rate_lo: float = 0.005
    rate_hi: float = 0.05
    rate_const: Optional[float] = None  # one fixed rate for every channel

    def n_pre(self, layer: int = 0) -> int:
        fan_in = self.n_in if layer == 0 else self.n_rec
        return fan_in + (self.n_rec if self.recurrent else 0)

    def layer_in(self, layer: int) -> int:
        return self.n_in if layer == 0 else self.n_rec

    def syn_per_step(self) -> int:
        """Synapse updates per timestep summed over layers: B * N_pre * N_post."""
        return sum(self.batch * self.n_pre(l) * self.n_rec for l in range(self.n_layers))

    def replace(self, **kw) -> "EpropShape":
        return dataclasses.replace(self, **kw)


# The five workloads of the hot path.  Names say what they are.
WORKLOADS = {
    # Feed-forward LIF layer where e-prop equals BPTT: B=4, 16 in, 32 LIF, T=50.
    "ff_lif_b4_n32_t50": EpropShape(batch=4, n_in=16, n_rec=32, n_out=4, T=50,
                                    recurrent=0, n_adaptive=0, rate_const=0.1),
    # Recurrent LIF: B=32, 700 in, 256 LIF, T=250, 20 classes.
    "rlif_b32_n256_t250": EpropShape(batch=32, n_in=700, n_rec=256, n_out=20, T=250,
                                     recurrent=1, n_adaptive=0),
    # Recurrent ALIF, 40% adaptive: B=64, 700 in, 512 neurons, T=500, 20 classes.
    "ralif_b64_n512_t500": EpropShape(batch=64, n_in=700, n_rec=512, n_out=20, T=500,
                                      recurrent=1, n_adaptive=int(0.4 * 512)),
    # Recurrent ALIF at scale, 50% adaptive: B=128, 700 in, 1024 neurons, T=1000, 35 classes.
    "ralif_b128_n1024_t1000": EpropShape(batch=128, n_in=700, n_rec=1024, n_out=35, T=1000,
                                         recurrent=1, n_adaptive=512),
    # Two stacked recurrent ALIF layers: B=256, 700 in, 2048 per layer, T=2000, 35 classes.
    "ralif2_b256_n2048_t2000": EpropShape(batch=256, n_in=700, n_rec=2048, n_out=35, T=2000,
                                          n_layers=2, recurrent=1, n_adaptive=1024),
}
WORKLOAD_ORDER = list(WORKLOADS)
WORKLOAD_SEED = {name: k + 1 for k, name in enumerate(WORKLOAD_ORDER)}


def quantize(w: np.ndarray, fan_in: int) -> np.ndarray:
    clip = 512.0 / fan_in
    q = np.round(w / GRID) * GRID
    return np.clip(q, -clip, clip).astype(np.float32)


@dataclasses.dataclass
class Workload:
    shape: EpropShape
    W: List[np.ndarray]      # per layer, fp32 [N_rec, N_pre] = [W_in | W_rec]
    Wout: List[np.ndarray]   # per layer, fp32 [K, N_rec]
    labels: np.ndarray       # int32 [B]
    x: np.ndarray            # uint8 [T, B, N_in]
    rates: np.ndarray        # fp64 [N_in]


def make_weights(shape: EpropShape, rng: np.random.Generator):
    W, Wout = [], []
    for layer in range(shape.n_layers):
        fan = shape.layer_in(layer)
        w_in = rng.normal(0.0, 1.0 / math.sqrt(fan), size=(shape.n_rec, fan))
        parts = [quantize(w_in, shape.n_pre(layer))]
        if shape.recurrent:
            w_rec = rng.normal(0.0, 1.0 / math.sqrt(shape.n_rec), size=(shape.n_rec, shape.n_rec))
            np.fill_diagonal(w_rec, 0.0)
            parts.append(quantize(w_rec, shape.n_pre(layer)))
        W.append(np.ascontiguousarray(np.concatenate(parts, axis=1), dtype=np.float32))
        w_out = rng.normal(0.0, 1.0 / math.sqrt(shape.n_rec), size=(shape.n_out, shape.n_rec))
        Wout.append(np.ascontiguousarray(quantize(w_out, shape.n_rec)))
    return W, Wout


def make_feedback(shape: EpropShape, seed: int) -> List[np.ndarray]:
    """Fixed random feedback matrices B [K, N_rec] per layer for the
    learning signal L = B^T delta: drawn like W_out (N(0, 1/N_rec), on the
    weight grid) from their own generator."""
    rng = np.random.Generator(np.random.PCG64(10_000 + seed))
    return [np.ascontiguousarray(quantize(rng.normal(0.0, 1.0 / math.sqrt(shape.n_rec),
                                                     size=(shape.n_out, shape.n_rec)), shape.n_rec))
            for _ in range(shape.n_layers)]


def make_workload(shape: EpropShape, seed: int, T: Optional[int] = None,
                  input_scale: float = 1.0) -> Workload:
    """Draw a workload with a fixed draw order: rates, then per layer W_in,
    W_rec (zero diagonal), W_out, then labels, then x one timestep at a time.
    ``input_scale`` multiplies the rates (0 gives silent inputs)."""
    T = shape.T if T is None else T
    rng = np.random.Generator(np.random.PCG64(seed))
    if shape.rate_const is not None:
        rates = np.full(shape.n_in, shape.rate_const)
    else:
        rates = rng.uniform(shape.rate_lo, shape.rate_hi, size=shape.n_in)
    rates = rates * input_scale
    W, Wout = make_weights(shape, rng)
    labels = rng.integers(0, shape.n_out, size=shape.batch).astype(np.int32)
    x = np.empty((T, shape.batch, shape.n_in), dtype=np.uint8)
    for t in range(T):
        x[t] = rng.random((shape.batch, shape.n_in)) < rates[None, :]
    return Workload(shape=shape, W=W, Wout=Wout, labels=labels, x=x, rates=rates)


def named_workload(name: str, T: Optional[int] = None) -> Workload:
    return make_workload(WORKLOADS[name], WORKLOAD_SEED[name], T=T)
