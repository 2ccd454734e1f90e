"""The entry point that allocates nothing (eprop_sequence_static) against the
context path (eprop_init + eprop_run_sequence + eprop_get_grads) and the
oracle, through the C ABI: two calls in a row, the second on a smaller input,
so the second runs over what the first left in the shared static scratch."""
import math

import numpy as np
import pytest
import torch

from paper_2501_11407_amd import eprop, synth
from tests.bptt_torch import rel_l2
from tests.gpu_util import check_against_oracle, gpu_run, to_dev

pytestmark = pytest.mark.gpu
f32 = synth.f32
DISTINCT = dict(kappa=f32(math.exp(-1 / 7)), rho=f32(math.exp(-1 / 50)))

CASES = [
    # two layers, two blocks (200 + 400 steps), partial tiles
    (synth.EpropShape(batch=5, n_in=21, n_rec=45, n_out=4, T=600, n_layers=2, n_adaptive=22,
                      **DISTINCT), 4),
    # then a smaller one: one layer, fewer elements, neurons and steps
    (synth.EpropShape(batch=3, n_in=37, n_rec=29, n_out=5, T=40, n_adaptive=13, **DISTINCT), 3),
]


def static_run(wl):
    shape = wl.shape
    cfg = eprop.make_config(shape)
    dev = torch.device("cuda")
    weights = []
    for l in range(shape.n_layers):
        weights += [torch.from_numpy(wl.W[l]).to(dev), torch.from_numpy(wl.Wout[l]).to(dev)]
    grads = []
    for l in range(shape.n_layers):
        grads += [torch.full((shape.n_rec, shape.n_pre(l)), float("nan"), device=dev),
                  torch.full((shape.n_out, shape.n_rec), float("nan"), device=dev)]
    x, labels = to_dev(wl)
    W32 = (shape.n_rec + 31) // 32
    spikes = torch.zeros((shape.T, shape.n_layers, shape.batch, W32), dtype=torch.int32, device=dev)
    loss = torch.zeros(1, dtype=torch.float64, device=dev)
    torch.cuda.synchronize()
    before = torch.cuda.memory_allocated()
    eprop.eprop_sequence_static(cfg, weights, x, shape.T, labels, spikes, grads, loss)
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == before
    return dict(dW=[grads[2 * l].cpu().numpy() for l in range(shape.n_layers)],
                dWout=[grads[2 * l + 1].cpu().numpy() for l in range(shape.n_layers)],
                loss=float(loss.cpu()), spikes=spikes.cpu().numpy().view(np.uint32), status=0)


def test_static_entry_matches_the_context_path_twice():
    for shape, seed in CASES:
        print(f"[gpu-test] static entry {shape}", flush=True)
        wl = synth.make_workload(shape, seed, input_scale=4.0)
        assert eprop.eprop_workspace_bytes(eprop.make_config(shape)) <= eprop.STATIC_SCRATCH_BYTES
        got = static_run(wl)
        ref = gpu_run(wl)
        assert np.array_equal(got["spikes"], ref["spikes"])
        for l in range(shape.n_layers):
            assert np.array_equal(got["dW"][l], ref["dW"][l]), rel_l2(got["dW"][l], ref["dW"][l])
            assert np.array_equal(got["dWout"][l], ref["dWout"][l])
        assert got["loss"] == ref["loss"]
        errs, oref = check_against_oracle(wl, got)
        assert oref.spikes.any()
        print(f"[gpu-test] static entry vs oracle: {errs}", flush=True)


def test_static_entry_rejects_a_shape_past_its_scratch():
    shape = synth.WORKLOADS["ralif_b64_n512_t500"]
    with pytest.raises(eprop.EpropError) as e:
        static_run(synth.make_workload(shape.replace(T=2), 1))
    assert e.value.code == eprop.EPROP_ENOSPACE
