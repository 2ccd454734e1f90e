"""Helpers shared by the GPU tests: run the HIP path through the C ABI and
compare it with the oracle."""
import os

import numpy as np
import torch

import oracle
from paper_2501_11407_amd import eprop, synth
from tests.bptt_torch import rel_l2

GRAD_TOL = 1e-4          # relative L2 per gradient tensor, fp32 path vs fp64 oracle


def workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def to_dev(wl, T=None):
    T = wl.x.shape[0] if T is None else T
    x = torch.from_numpy(np.ascontiguousarray(wl.x[:T])).cuda()
    labels = torch.from_numpy(wl.labels.astype(np.int32)).cuda()
    return x, labels


def gpu_run(wl, T=None, chunks=None, ctx=None, feedback=None):
    """Runs the HIP path over the workload; returns numpy results.
    ``chunks``: split the sequence into run_sequence calls of these lengths.
    ``feedback``: per-layer feedback matrices of the learning signal."""
    shape = wl.shape
    T = wl.x.shape[0] if T is None else T
    own = ctx is None
    if own:
        ctx = eprop.EpropContext(shape, wl.W, wl.Wout)
    if feedback is not None:
        ctx.set_feedback(feedback)
    x, labels = to_dev(wl, T)
    spikes = ctx.new_spike_buffer(T)
    chunks = chunks or [T]
    assert sum(chunks) == T
    t0 = 0
    for n in chunks:
        ctx.run_sequence(x[t0:t0 + n], labels, spikes[t0:t0 + n])
        t0 += n
    dW, dWout, loss = ctx.get_grads()
    torch.cuda.synchronize()
    status = ctx.status()
    out = dict(dW=[d.cpu().numpy() for d in dW], dWout=[d.cpu().numpy() for d in dWout],
               loss=float(loss.cpu()), spikes=spikes.cpu().numpy().view(np.uint32), status=status)
    if own:
        ctx.close()
    return out


def first_spike_mismatch(a, b):
    bad = np.argwhere(a != b)
    if len(bad) == 0:
        return None
    t, l, bb, w = bad[0]
    return dict(t=int(t), layer=int(l), b=int(bb), word=int(w), gpu=hex(int(a[t, l, bb, w])),
                oracle=hex(int(b[t, l, bb, w])), n_words=len(bad))


def sample_synapses(shape, n_random=384, seed=0):
    """Random synapses plus the edges of every index range: first/last input,
    first/last recurrent column, first/last adaptive and LIF neuron."""
    rng = np.random.default_rng(seed)
    rows = []
    for l in range(shape.n_layers):
        n_pre, n_in_l = shape.n_pre(l), shape.layer_in(l)
        js = {0, shape.n_rec - 1, max(shape.n_adaptive - 1, 0), min(shape.n_adaptive, shape.n_rec - 1)}
        is_ = {0, n_in_l - 1, min(n_in_l, n_pre - 1), n_pre - 1}
        rows += [(l, j, i) for j in js for i in is_]
        rows += [(l, int(rng.integers(shape.n_rec)), int(rng.integers(n_pre)))
                 for _ in range(n_random // shape.n_layers)]
    return np.array(rows, dtype=np.int32)


def sample_every_tile(shape, tile=64, seed=0):
    """One random synapse inside every tile x tile block of (i, j) of every
    layer, plus the index-range edges of sample_synapses."""
    rng = np.random.default_rng(seed)
    rows = [tuple(r) for r in sample_synapses(shape, n_random=0)]
    for l in range(shape.n_layers):
        n_pre = shape.n_pre(l)
        for i0 in range(0, n_pre, tile):
            for j0 in range(0, shape.n_rec, tile):
                i = int(rng.integers(i0, min(i0 + tile, n_pre)))
                j = int(rng.integers(j0, min(j0 + tile, shape.n_rec)))
                rows.append((l, j, i))
    return np.array(rows, dtype=np.int32)


def check_against_oracle(wl, gpu, sample=None, T=None, tol=GRAD_TOL, feedback=None):
    """Oracle on the same inputs; spikes must be identical, gradients within tol."""
    shape = wl.shape
    ref = oracle.run_sharded(shape, wl.W, wl.Wout, wl.x, wl.labels, T=T, sample=sample,
                             workers=workers(), feedback=feedback)
    mism = first_spike_mismatch(gpu["spikes"], ref.spikes)
    assert mism is None, f"spike trains differ: {mism}"
    errs = {}
    if sample is None:
        for l in range(shape.n_layers):
            errs[f"dW{l}"] = rel_l2(gpu["dW"][l], ref.dW[l])
    else:
        got = np.array([gpu["dW"][l][j, i] for l, j, i in sample])
        errs["dW_sampled"] = rel_l2(got, ref.dW[0])
        assert np.abs(ref.dW[0]).max() > 0
    for l in range(shape.n_layers):
        errs[f"dWout{l}"] = rel_l2(gpu["dWout"][l], ref.dWout[l])
    errs["loss"] = abs(gpu["loss"] - ref.loss) / max(abs(ref.loss), 1e-300)
    assert gpu["status"] == 0
    for k, v in errs.items():
        assert v <= tol, (k, v, errs)
    return errs, ref
