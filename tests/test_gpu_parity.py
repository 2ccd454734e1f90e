"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Spike trains must be bit-identical; gradients (fp32 HIP path, fp64 oracle)
within relative L2 1e-4 per tensor; the loss within 1e-4 relative.
"""
import gc
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2501_11407_amd import eprop, synth
from tests.bptt_torch import rel_l2
from tests.gpu_util import (check_against_oracle, first_spike_mismatch, gpu_run, sample_every_tile,
                            sample_synapses, to_dev, workers)

pytestmark = pytest.mark.gpu
f32 = synth.f32


def banner(msg):
    print(f"[gpu-test] {msg}", flush=True)


def small(**kw):
    base = dict(batch=3, n_in=37, n_rec=29, n_out=5, T=40, recurrent=1, n_adaptive=0)
    base.update(kw)
    return synth.EpropShape(**base)


DISTINCT = dict(kappa=f32(math.exp(-1 / 7)), rho=f32(math.exp(-1 / 50)))

# Small shapes the oracle finishes in well under a second: ragged sizes that
# leave partial 64x64 eligibility tiles, partial 16-step chunks and 4-step
# quads, partial spike words, an adaptive/LIF boundary inside a tile, several
# tiles over j, several batch splits, and sequences split into two and three
# blocks (174 + 347 steps; 220 + 440 + 440).
RAGGED = {
    "rlif_ragged": (small(**DISTINCT), 2, 4.0),
    "ralif_ragged_na13": (small(n_adaptive=13, **DISTINCT), 3, 4.0),
    "ralif_all_adaptive": (small(n_adaptive=29, **DISTINCT), 5, 4.0),
    "ff_alif": (small(recurrent=0, n_adaptive=11, **DISTINCT), 6, 4.0),
    "ralif2_two_layers": (small(batch=5, n_in=21, n_rec=45, n_out=4, n_layers=2, n_adaptive=22,
                                **DISTINCT), 4, 4.0),
    "batch1_neuron1": (small(batch=1, n_in=1, n_rec=1, n_out=2, T=30, n_adaptive=1), 7, 20.0),
    "one_class": (small(n_out=1, n_adaptive=5), 8, 4.0),
    "wide_1100": (small(batch=2, n_in=50, n_rec=1100, n_out=7, T=12, n_adaptive=550), 9, 4.0),
    "batch37_k33": (small(batch=37, n_in=70, n_rec=70, n_out=33, T=25, n_adaptive=35), 10, 4.0),
    "single_step": (small(T=1, n_adaptive=13), 11, 8.0),
    "blocks_174_347": (small(n_adaptive=13, T=521, **DISTINCT), 12, 4.0),
    "blocks_220_440_440": (small(batch=6, n_adaptive=29, T=1100, **DISTINCT), 13, 4.0),
    # more classes than one wave's lanes (the readout's second path), up to
    # the largest class count the library accepts
    "classes_100": (small(batch=4, n_out=100, n_adaptive=13, **DISTINCT), 14, 4.0),
    "classes_1024": (small(batch=2, n_in=20, n_rec=70, n_out=1024, T=20, n_adaptive=35), 15, 4.0),
}
# Weight multipliers (powers of two keep the 2**-14 grid): one step needs a
# strong drive to spike.  Partial sums stay far below 2**10, so they are exact.
W_SCALE = {"single_step": 8.0}


@pytest.mark.parametrize("name", list(RAGGED))
def test_ragged_shapes(name):
    shape, seed, scale = RAGGED[name]
    banner(f"ragged {name} {shape}")
    wl = synth.make_workload(shape, seed, input_scale=scale)
    for w in wl.W:
        w *= W_SCALE.get(name, 1.0)
    gpu = gpu_run(wl)
    errs, ref = check_against_oracle(wl, gpu)
    if name not in ("one_class",):
        assert ref.spikes.any()


# ---------------------------------------------------------------- large layers
# 8 and 16 neurons per forward thread, up to the largest accepted layer
# (8192 neurons, recurrent or not); every spike compared, the gradient on
# sampled synapses (with every index-range edge) and the readout gradient in full.
@pytest.mark.parametrize("n_rec,n_in,rec", [(3000, 200, 1), (6000, 100, 1), (8192, 200, 0), (8192, 200, 1)])
def test_large_layers(n_rec, n_in, rec):
    shape = synth.EpropShape(batch=2, n_in=n_in, n_rec=n_rec, n_out=10, T=24, recurrent=rec,
                             n_adaptive=n_rec // 2)
    banner(f"large layer {shape}")
    wl = synth.make_workload(shape, 20 + n_rec, input_scale=4.0)
    gpu = gpu_run(wl)
    smp = sample_synapses(shape, seed=n_rec)
    errs, ref = check_against_oracle(wl, gpu, sample=smp)
    assert ref.spikes.any()
    banner(f"{n_rec}: {errs}")


# ---------------------------------------------------------------- drive paths
# Weights on the 2**-14 grid (within the integer bound) are summed as
# integers; any other weights as fp32 in ascending input order, which the
# oracle's sequential fp32 sums reproduce bit for bit.
def _off_grid(wl, seed):
    rng = np.random.default_rng(seed)
    for w in wl.W:
        m = rng.random(w.shape) < 0.3
        w[m] = (w[m] * f32(1 + 2.0 ** -20)).astype(np.float32)   # no longer a multiple of 2**-14


def test_grid_weights_take_the_integer_drive():
    shape, seed, scale = RAGGED["ralif2_two_layers"]
    wl = synth.make_workload(shape, seed, input_scale=scale)
    ctx = eprop.EpropContext(shape, wl.W, wl.Wout)
    assert ctx.integer_drive()
    ctx.close()


@pytest.mark.parametrize("name", ["rlif_ragged", "ralif2_two_layers", "blocks_220_440_440", "wide_1100",
                                  "classes_100"])
def test_off_grid_weights_take_the_float_drive(name):
    shape, seed, scale = RAGGED[name]
    banner(f"off-grid weights {name} {shape}")
    wl = synth.make_workload(shape, seed, input_scale=scale)
    _off_grid(wl, seed)
    ctx = eprop.EpropContext(shape, wl.W, wl.Wout)
    assert not ctx.integer_drive()
    gpu = gpu_run(wl, ctx=ctx)
    ctx.close()
    errs, ref = check_against_oracle(wl, gpu)
    assert ref.spikes.any()


def test_large_grid_weight_takes_the_float_drive():
    # on the grid but past the integer bound: 4.0 is 2**16 units of 2**-14
    shape, seed, scale = RAGGED["ralif_ragged_na13"]
    wl = synth.make_workload(shape, seed, input_scale=scale)
    wl.W[0][3, 5] = f32(4.0)
    ctx = eprop.EpropContext(shape, wl.W, wl.Wout)
    assert not ctx.integer_drive()
    gpu = gpu_run(wl, ctx=ctx)
    ctx.close()
    check_against_oracle(wl, gpu)


def test_integer_drive_decided_per_step():
    # int16 weights up to |k| = 32767 (2.0): steps with more than 512 active
    # inputs take the fp32 drive, the others the integer drive; both must give
    # the oracle's sequential fp32 sums bit for bit
    shape = small(batch=2, n_in=1000, n_rec=40, n_out=3, T=30, n_adaptive=20, **DISTINCT)
    wl = synth.make_workload(shape, 61)
    rng = np.random.default_rng(61)
    k = rng.integers(-32767, 32768, size=wl.W[0].shape)
    k[0, 0] = 32767
    wl.W[0][:] = (k * 2.0 ** -14).astype(np.float32)
    wl.x[:] = 0
    for t in range(shape.T):
        rate = 0.6 if t % 3 == 0 else 0.01
        wl.x[t] = rng.random((shape.batch, shape.n_in)) < rate
    ctx = eprop.EpropContext(shape, wl.W, wl.Wout)
    assert ctx.integer_weights() == (True, 32767)
    gpu = gpu_run(wl, ctx=ctx)
    ctx.close()
    errs, ref = check_against_oracle(wl, gpu)
    assert ref.spikes.any()
    assert wl.x[0].sum(axis=1).max() > 512 and wl.x[1].sum(axis=1).max() < 512


def test_drive_path_follows_the_weights_over_resets():
    shape, seed, scale = RAGGED["ralif_ragged_na13"]
    wl = synth.make_workload(shape, seed, input_scale=scale)
    ctx = eprop.EpropContext(shape, wl.W, wl.Wout)
    assert ctx.integer_drive()
    a = gpu_run(wl, ctx=ctx)
    keep = ctx.weights[0].clone()
    ctx.weights[0][0, 0] += 2.0 ** -20
    ctx.reset()
    assert not ctx.integer_drive()
    ctx.weights[0].copy_(keep)
    ctx.reset()
    assert ctx.integer_drive()
    b = gpu_run(wl, ctx=ctx)
    ctx.close()
    assert np.array_equal(a["spikes"], b["spikes"]) and np.array_equal(a["dW"][0], b["dW"][0])


# ---------------------------------------------------------------- online weight application
# Every `every` steps the weights in use become W0 - lr * G on the 2**-14 grid.
# Rounding turns the gradient into weights, so the GPU (fp32 traces) and the
# oracle (fp64) agree on every weight only if no value lies near a rounding
# tie: the cases are seeds whose oracle values keep a margin well above the
# GPU's gradient error (about 1e-5 grid units at lr = 2**-12); the test
# asserts that margin from the oracle alone.
ONLINE = {
    "rlif": (small(**DISTINCT), 35, 10),
    "ralif": (small(n_adaptive=13, T=60, **DISTINCT), 38, 10),
    "ff_alif": (small(recurrent=0, n_adaptive=11, **DISTINCT), 30, 10),
    "ralif2": (small(batch=2, n_in=21, n_rec=19, n_out=4, T=60, n_layers=2, n_adaptive=9,
                     **DISTINCT), 31, 10),
    "blocks_300": (small(batch=2, n_in=15, n_rec=20, n_out=3, n_adaptive=10, T=300, **DISTINCT), 30,
                   100),
    "reset_path_kept": (small(n_adaptive=13, **DISTINCT).replace(reset_grad=1), 46, 10),
}
ONLINE_LR = 2.0 ** -12


def _online_margin(shape, wl, lr, every):
    m = np.inf
    for t1 in range(every, wl.x.shape[0], every):
        r = oracle.run_online(shape, wl.W, wl.Wout, wl.x, wl.labels, lr, every, T=t1)
        for l in range(shape.n_layers):
            for W0, G in ((wl.W[l], r.dW[l]), (wl.Wout[l], r.dWout[l])):
                v = (W0.astype(np.float64) - lr * G) * 16384.0
                m = min(m, float(np.min(np.abs(np.abs(v - np.floor(v)) - 0.5))))
    return m


@pytest.mark.parametrize("name", list(ONLINE))
def test_online_weights_match_oracle(name):
    shape, seed, every = ONLINE[name]
    banner(f"online weights {name} {shape} every {every}")
    wl = synth.make_workload(shape, seed, input_scale=4.0)
    assert _online_margin(shape, wl, ONLINE_LR, every) > 1e-4
    ref = oracle.run_online(shape, wl.W, wl.Wout, wl.x, wl.labels, ONLINE_LR, every)
    for chunks in (None, [7, shape.T - 7]):
        ctx = eprop.EpropContext(shape, wl.W, wl.Wout)
        ctx.set_online(ONLINE_LR, every)
        gpu = gpu_run(wl, ctx=ctx, chunks=chunks)
        Wg, Wog = ctx.get_weights()
        torch.cuda.synchronize()
        ctx.close()
        mism = first_spike_mismatch(gpu["spikes"], ref.spikes)
        assert mism is None, f"spike trains differ: {mism}"
        for l in range(shape.n_layers):
            assert np.array_equal(Wg[l].cpu().numpy(), ref.W[l]), f"layer {l} weights differ"
            assert np.array_equal(Wog[l].cpu().numpy(), ref.Wout[l])
            assert rel_l2(gpu["dW"][l], ref.dW[l]) <= 1e-4
            assert rel_l2(gpu["dWout"][l], ref.dWout[l]) <= 1e-4
        assert abs(gpu["loss"] - ref.loss) <= 1e-4 * abs(ref.loss)
        assert any(not np.array_equal(ref.W[l], wl.W[l]) for l in range(shape.n_layers))


ONLINE_FB = {
    "rlif": ONLINE["rlif"],
    "ralif": ONLINE["ralif"],
    "ralif2": ONLINE["ralif2"],
}


def _online_margin_fb(shape, wl, lr, every, fb):
    m = np.inf
    for t1 in range(every, wl.x.shape[0], every):
        r = oracle.run_online(shape, wl.W, wl.Wout, wl.x, wl.labels, lr, every, T=t1, feedback=fb)
        for l in range(shape.n_layers):
            for W0, G in ((wl.W[l], r.dW[l]), (wl.Wout[l], r.dWout[l])):
                v = (W0.astype(np.float64) - lr * G) * 16384.0
                m = min(m, float(np.min(np.abs(np.abs(v - np.floor(v)) - 0.5))))
    return m


@pytest.mark.parametrize("name", list(ONLINE_FB))
def test_online_weights_with_feedback_match_oracle(name):
    # Online weight application with fixed feedback matrices (two layers:
    # on layer 1 only).  The matrices stay while W and W_out change.  Split
    # calls set the same matrices again between the calls, after an update:
    # that must not touch the weights in use.
    shape, seed, every = ONLINE_FB[name]
    banner(f"online weights with feedback {name} {shape} every {every}")
    wl = synth.make_workload(shape, seed, input_scale=4.0)
    fb = synth.make_feedback(shape, seed)
    if shape.n_layers == 2:
        fb[1] = None
    assert _online_margin_fb(shape, wl, ONLINE_LR, every, fb) > 1e-4
    ref = oracle.run_online(shape, wl.W, wl.Wout, wl.x, wl.labels, ONLINE_LR, every, feedback=fb)
    sym = oracle.run_online(shape, wl.W, wl.Wout, wl.x, wl.labels, ONLINE_LR, every)
    assert rel_l2(ref.dW[0], sym.dW[0]) > 1e-2
    for split in (None, 15):
        ctx = eprop.EpropContext(shape, wl.W, wl.Wout)
        ctx.set_online(ONLINE_LR, every)
        ctx.set_feedback(fb)
        x, labels = to_dev(wl)
        spikes = ctx.new_spike_buffer(shape.T)
        if split is None:
            ctx.run_sequence(x, labels, spikes)
        else:
            ctx.run_sequence(x[:split], labels, spikes[:split])
            ctx.set_feedback(fb)
            ctx.run_sequence(x[split:], labels, spikes[split:])
        dW, dWout, loss = ctx.get_grads()
        Wg, Wog = ctx.get_weights()
        torch.cuda.synchronize()
        assert ctx.status() == 0
        ctx.close()
        mism = first_spike_mismatch(spikes.cpu().numpy().view(np.uint32), ref.spikes)
        assert mism is None, f"spike trains differ: {mism}"
        for l in range(shape.n_layers):
            assert np.array_equal(Wg[l].cpu().numpy(), ref.W[l]), f"layer {l} weights differ"
            assert np.array_equal(Wog[l].cpu().numpy(), ref.Wout[l])
            assert rel_l2(dW[l].cpu().numpy(), ref.dW[l]) <= 1e-4
            assert rel_l2(dWout[l].cpu().numpy(), ref.dWout[l]) <= 1e-4
        assert abs(float(loss.cpu()) - ref.loss) <= 1e-4 * abs(ref.loss)


def test_online_off_and_reset_give_the_plain_run():
    shape, seed, every = ONLINE["rlif"]
    wl = synth.make_workload(shape, seed, input_scale=4.0)
    plain = gpu_run(wl)
    ctx = eprop.EpropContext(shape, wl.W, wl.Wout)
    ctx.set_online(ONLINE_LR, every)
    gpu_run(wl, ctx=ctx)
    ctx.set_online(0.0, 0)
    ctx.reset()                              # back to W0, updates off
    b = gpu_run(wl, ctx=ctx)
    Wg, _ = ctx.get_weights()
    torch.cuda.synchronize()
    ctx.close()
    assert np.array_equal(b["spikes"], plain["spikes"]) and np.array_equal(b["dW"][0], plain["dW"][0])
    assert np.array_equal(Wg[0].cpu().numpy(), wl.W[0])


# ---------------------------------------------------------------- random feedback
@pytest.mark.parametrize("name", ["rlif_ragged", "ralif_ragged_na13", "ralif2_two_layers",
                                  "blocks_220_440_440"])
def test_random_feedback_matches_oracle(name):
    # learning signal L = B^T delta with fixed matrices B (two layers: the
    # second layer keeps W_out, so both forms run in one context)
    shape, seed, scale = RAGGED[name]
    banner(f"random feedback {name} {shape}")
    wl = synth.make_workload(shape, seed, input_scale=scale)
    fb = synth.make_feedback(shape, seed)
    if shape.n_layers == 2:
        fb[1] = None
    gpu = gpu_run(wl, feedback=fb)
    ref_fb = [f if f is not None else wl.Wout[l] for l, f in enumerate(fb)]
    errs, _ = check_against_oracle(wl, gpu, feedback=ref_fb)
    banner(f"{name}: {errs}")


def test_random_feedback_full_workload():
    wl = synth.named_workload("rlif_b32_n256_t250")
    fb = synth.make_feedback(wl.shape, 2)
    banner("random feedback rlif_b32_n256_t250, every synapse")
    gpu = gpu_run(wl, feedback=fb)
    errs, _ = check_against_oracle(wl, gpu, feedback=fb)
    banner(f"{errs}")


def test_feedback_kept_over_reset_and_cleared():
    shape, seed, scale = RAGGED["ralif_ragged_na13"]
    wl = synth.make_workload(shape, seed, input_scale=scale)
    fb = synth.make_feedback(shape, seed)
    ctx = eprop.EpropContext(shape, wl.W, wl.Wout)
    ctx.set_feedback(fb)
    a = gpu_run(wl, ctx=ctx)
    ctx.reset()
    b = gpu_run(wl, ctx=ctx)                  # the feedback is read again by the reset
    assert np.array_equal(a["dW"][0], b["dW"][0])
    ctx.set_feedback(None)
    ctx.reset()
    c = gpu_run(wl, ctx=ctx)
    ctx.close()
    check_against_oracle(wl, c)               # back to the symmetric learning signal
    check_against_oracle(wl, a, feedback=fb)
    assert rel_l2(a["dW"][0], c["dW"][0]) > 1e-2


# ---------------------------------------------------------------- reset path kept
@pytest.mark.parametrize("name", ["rlif_ragged", "ralif_ragged_na13", "ralif_all_adaptive", "ff_alif",
                                  "ralif2_two_layers", "blocks_220_440_440", "single_step", "classes_100",
                                  "blocks_174_347", "wide_1100"])
def test_reset_through_matches_oracle(name):
    shape, seed, scale = RAGGED[name]
    shape = shape.replace(reset_grad=1)
    banner(f"reset path kept {name} {shape}")
    wl = synth.make_workload(shape, seed, input_scale=scale)
    for w in wl.W:
        w *= W_SCALE.get(name, 1.0)
    gpu = gpu_run(wl)
    errs, ref = check_against_oracle(wl, gpu)
    assert ref.spikes.any()
    banner(f"{name}: {errs}")


# The eligibility kernel exists once per count of 16-step chunks in a block
# (up to 32: blocks of at most 512 steps).  Under the equal split a call of up
# to 256 steps is one block, one of 257..1024 steps two blocks of equal length
# (eprop_block_lengths says so).  Fed in calls of these lengths, the blocks
# hold 1, 2, ..., 32 chunks (the last chunk partial but for the first).
EVERY_CHUNK_COUNT = [16 * k + 1 for k in range(16)] + [2 * (16 * k + 1) for k in range(16, 32)]


def every_chunk_count_run(wl):
    cfg = eprop.make_config(wl.shape)
    blocks = [n for T in EVERY_CHUNK_COUNT
              for n in eprop.eprop_block_lengths(cfg, T, mode=eprop.EPROP_SPLIT_EQUAL)]
    assert sorted({-(-n // 16) for n in blocks}) == list(range(1, 33))
    ctx = eprop.EpropContext(wl.shape, wl.W, wl.Wout)
    ctx.set_block_split(eprop.EPROP_SPLIT_EQUAL)
    gpu = gpu_run(wl, chunks=EVERY_CHUNK_COUNT, ctx=ctx)
    ctx.close()
    return gpu


@pytest.mark.parametrize("reset_grad", [0, 1])
def test_every_chunk_count(reset_grad):
    shape = small(n_rec=70, n_adaptive=13, T=sum(EVERY_CHUNK_COUNT), reset_grad=reset_grad,
                  **DISTINCT)
    banner(f"every chunk count, reset_grad={reset_grad}, {shape}")
    wl = synth.make_workload(shape, 21, input_scale=4.0)
    gpu = every_chunk_count_run(wl)
    errs, ref = check_against_oracle(wl, gpu)
    assert ref.spikes.any()
    banner(f"every chunk count: {errs}")


@pytest.mark.parametrize("name", ["ralif_ragged_na13", "ralif2_two_layers"])
def test_reset_through_with_random_feedback(name):
    # both variants at once: the learning signal through B, the reset path kept
    shape, seed, scale = RAGGED[name]
    shape = shape.replace(reset_grad=1)
    banner(f"reset path kept with random feedback {name}")
    wl = synth.make_workload(shape, seed, input_scale=scale)
    fb = synth.make_feedback(shape, seed)
    gpu = gpu_run(wl, feedback=fb)
    errs, ref = check_against_oracle(wl, gpu, feedback=fb)
    assert ref.spikes.any()


def test_reset_through_full_workload_and_split_calls():
    wl = synth.named_workload("rlif_b32_n256_t250")
    wl.shape = wl.shape.replace(reset_grad=1)
    banner("reset path kept rlif_b32_n256_t250, every synapse, three calls")
    gpu = gpu_run(wl, chunks=[100, 7, 143])
    errs, _ = check_against_oracle(wl, gpu)
    banner(f"{errs}")


# ---------------------------------------------------------------- two-compartment neuron
# A soma-dendrite neuron whose own spike feeds its dendrite: the forward takes
# the step with the coefficients the library derives on the host, the
# eligibility recursion has a full 2x2 Jacobian block per neuron (generic
# adjoint coefficient pass, three traces per synapse).
TC = dict(neuron_model=1, n_adaptive=0)
TWO_COMP = {
    "tc_ragged": (small(**TC, **DISTINCT), 2, 4.0),
    "tc_ff": (small(recurrent=0, **TC, **DISTINCT), 6, 4.0),
    "tc_two_layers": (small(batch=5, n_in=21, n_rec=45, n_out=4, n_layers=2, **TC, **DISTINCT), 4, 4.0),
    "tc_blocks_220_440_440": (small(batch=6, T=1100, **TC, **DISTINCT), 13, 4.0),
    "tc_wide_1100": (small(batch=2, n_in=50, n_rec=1100, n_out=7, T=12, **TC), 9, 4.0),
    "tc_positive_feedback": (small(bap=0.25, coupling=0.75, **TC, **DISTINCT), 8, 4.0),
    "tc_classes_100": (small(batch=4, n_out=100, **TC, **DISTINCT), 14, 4.0),
}


@pytest.mark.parametrize("reset_grad", [0, 1])
@pytest.mark.parametrize("name", list(TWO_COMP))
def test_two_compartment_matches_oracle(name, reset_grad):
    shape, seed, scale = TWO_COMP[name]
    shape = shape.replace(reset_grad=reset_grad)
    banner(f"two-compartment {name} {shape}")
    wl = synth.make_workload(shape, seed, input_scale=scale)
    gpu = gpu_run(wl)
    errs, ref = check_against_oracle(wl, gpu)
    assert ref.spikes.any()
    banner(f"{name}: {errs}")


def test_two_compartment_full_workload_split_calls_and_state():
    # the recurrent workload's shape (B=32, 700 inputs, 256 neurons, T=250)
    # with two-compartment neurons, every synapse, over three calls; the soma
    # and dendrite state bit for bit
    wl = synth.make_workload(synth.WORKLOADS["rlif_b32_n256_t250"].replace(neuron_model=1), 2)
    banner("two-compartment rlif_b32_n256_t250 shape, every synapse, three calls")
    ctx = eprop.EpropContext(wl.shape, wl.W, wl.Wout)
    gpu = gpu_run(wl, chunks=[100, 7, 143], ctx=ctx)
    errs, _ = check_against_oracle(wl, gpu)
    T = 33
    ref = oracle.run(wl.shape, wl.W, wl.Wout, wl.x, wl.labels, T=T, b_hi=wl.shape.batch,
                     want_record=True)
    ctx.reset()
    x, labels = to_dev(wl, T)
    ctx.run_sequence(x, labels)
    torch.cuda.synchronize()
    assert np.array_equal(ctx.debug("v", 0).cpu().numpy(), ref.record["v"][T - 1, 0].astype(np.float32))
    assert np.array_equal(ctx.debug("a", 0).cpu().numpy(), ref.record["a"][T - 1, 0].astype(np.float32))
    ctx.close()
    banner(f"{errs}")


@pytest.mark.parametrize("reset_grad", [0, 1])
def test_two_compartment_every_chunk_count(reset_grad):
    shape = small(n_rec=70, T=sum(EVERY_CHUNK_COUNT), reset_grad=reset_grad, **TC, **DISTINCT)
    banner(f"two-compartment every chunk count, reset_grad={reset_grad}")
    wl = synth.make_workload(shape, 21, input_scale=4.0)
    gpu = every_chunk_count_run(wl)
    errs, ref = check_against_oracle(wl, gpu)
    assert ref.spikes.any()


def test_two_compartment_with_feedback_and_online_weights():
    # the two variants of the learning-signal row on the new neuron
    shape, seed, scale = TWO_COMP["tc_ragged"]
    wl = synth.make_workload(shape, seed, input_scale=scale)
    fb = synth.make_feedback(shape, seed)
    gpu = gpu_run(wl, feedback=fb)
    check_against_oracle(wl, gpu, feedback=fb)
    sh2 = small(n_adaptive=0, neuron_model=1, T=60, **DISTINCT)
    wl2 = synth.make_workload(sh2, 41, input_scale=4.0)
    every = 10
    assert _online_margin(sh2, wl2, ONLINE_LR, every) > 1e-4
    ref = oracle.run_online(sh2, wl2.W, wl2.Wout, wl2.x, wl2.labels, ONLINE_LR, every)
    ctx = eprop.EpropContext(sh2, wl2.W, wl2.Wout)
    ctx.set_online(ONLINE_LR, every)
    g2 = gpu_run(wl2, ctx=ctx, chunks=[7, sh2.T - 7])
    Wg, Wog = ctx.get_weights()
    torch.cuda.synchronize()
    ctx.close()
    assert first_spike_mismatch(g2["spikes"], ref.spikes) is None
    assert np.array_equal(Wg[0].cpu().numpy(), ref.W[0]) and np.array_equal(Wog[0].cpu().numpy(), ref.Wout[0])
    assert rel_l2(g2["dW"][0], ref.dW[0]) <= 1e-4


def test_silent_input_gives_zero_gradient():
    shape = small(n_adaptive=7)
    wl = synth.make_workload(shape, 4, input_scale=0.0)
    gpu = gpu_run(wl)
    assert not gpu["spikes"].any()
    assert all(not d.any() for d in gpu["dW"]) and all(not d.any() for d in gpu["dWout"])
    assert abs(gpu["loss"] - shape.batch * shape.T * math.log(shape.n_out)) < 1e-3


@pytest.mark.parametrize("name", ["ff_lif_b4_n32_t50", "rlif_b32_n256_t250"])
def test_named_workload_all_synapses(name):
    banner(f"workload {name}, every synapse")
    wl = synth.named_workload(name)
    gpu = gpu_run(wl)
    errs, _ = check_against_oracle(wl, gpu)
    banner(f"{name}: {errs}")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["ralif_b64_n512_t500", "ralif_b128_n1024_t1000"])
def test_named_workload_every_synapse_full_size(name):
    # Full size, every spike and every synapse's gradient (the oracle in
    # single-threaded batch shards on the host's cores).
    banner(f"workload {name}, every synapse")
    wl = synth.named_workload(name)
    gpu = gpu_run(wl)
    errs, _ = check_against_oracle(wl, gpu)
    banner(f"{name}: {errs}")


@pytest.mark.timeout(900)
def test_two_layer_workload_every_tile_sampled():
    # Two layers of 2048, B=256, T=2000: every spike, the readout gradients in
    # full, and one synapse in every 64 x 64 block of (i, j) of both layers
    # (3424 blocks) plus the index-range edges, which the oracle computes one
    # by one.
    name = "ralif2_b256_n2048_t2000"
    banner(f"workload {name}, one synapse per 64x64 block")
    wl = synth.named_workload(name)
    gpu = gpu_run(wl)
    smp = sample_every_tile(wl.shape)
    assert len(smp) > 3400
    errs, _ = check_against_oracle(wl, gpu, sample=smp)
    banner(f"{name}: {errs}")


@pytest.mark.parametrize("reset_grad", [0, 1])
def test_large_batch_uneven_splits(reset_grad):
    # B = 233: the eligibility kernel's batch split count comes from the
    # batch (9 splits of 26 or 25 elements), every synapse compared.
    shape = synth.EpropShape(batch=233, n_in=24, n_rec=40, n_out=5, T=40, n_adaptive=20,
                             reset_grad=reset_grad, **DISTINCT)
    banner(f"large batch {shape}")
    wl = synth.make_workload(shape, 233, input_scale=4.0)
    gpu = gpu_run(wl)
    errs, ref = check_against_oracle(wl, gpu)
    assert ref.spikes.any()
    banner(f"B=233: {errs}")


def adversarial_range_workload(reset_grad=0):
    """Mostly inhibitory inputs with a few strong excitatory channels (the
    pseudo-derivative is zero for most steps of most neurons) and a readout
    that becomes confident in the one label, so that the learning signal of a
    neuron spans many decades within one block."""
    shape = synth.EpropShape(batch=4, n_in=40, n_rec=48, n_out=3, T=300, n_adaptive=24,
                             reset_grad=reset_grad, **DISTINCT)
    wl = synth.make_workload(shape, 77, input_scale=6.0)
    rng = np.random.default_rng(5)
    w_in = rng.normal(-0.35, 0.25, size=(shape.n_rec, shape.n_in))
    exc = rng.random(shape.n_in) < 0.25
    w_in[:, exc] = rng.normal(0.9, 0.2, size=(shape.n_rec, int(exc.sum())))
    wl.W[0][:, :shape.n_in] = synth.quantize(w_in, 8)
    wl.labels[:] = 0
    wl.Wout[0][:] = -0.125
    wl.Wout[0][0] = 0.25
    return wl


@pytest.mark.parametrize("reset_grad", [0, 1])
def test_adversarial_dynamic_range(reset_grad):
    # The contraction operands are scaled fp16 pairs with one scale per
    # (batch element, neuron) row and block: small entries of a row with a
    # wide range keep only the row's absolute precision.  Here the learning
    # signal of every row spans >= 8 decades within each block and the
    # pseudo-derivative is zero for most steps (both checked on the oracle's
    # record); the gradients must still meet the parity bar.
    wl = adversarial_range_workload(reset_grad)
    shape = wl.shape
    banner(f"adversarial dynamic range, reset_grad={reset_grad}")
    rec = oracle.run(shape, wl.W, wl.Wout, wl.x, wl.labels, want_record=True).record
    assert (rec["psi"] == 0).mean() > 0.75
    for t0, t1 in ((0, 256), (256, shape.T)):
        a = np.abs(rec["L"][t0:t1, 0])
        lo = np.where(a > 0, a, np.inf).min(0)
        assert np.all(a.max(0) / lo >= 1e8)
    gpu = gpu_run(wl)
    errs, ref = check_against_oracle(wl, gpu)
    assert ref.spikes.any()
    banner(f"adversarial range: {errs}")


def test_intermediate_state_matches_oracle_record():
    shape, seed, scale = RAGGED["ralif2_two_layers"]
    wl = synth.make_workload(shape, seed, input_scale=scale)
    T = 17
    ref = oracle.run(shape, wl.W, wl.Wout, wl.x, wl.labels, T=T, want_record=True)
    ctx = eprop.EpropContext(shape, wl.W, wl.Wout)
    x, labels = to_dev(wl, T)
    ctx.run_sequence(x, labels)
    torch.cuda.synchronize()
    for l in range(shape.n_layers):
        v = ctx.debug("v", l).cpu().numpy()
        assert np.array_equal(v, ref.record["v"][T - 1, l].astype(np.float32))   # fp32 state, same bits
        a = ctx.debug("a", l).cpu().numpy()
        assert np.array_equal(a, ref.record["a"][T - 1, l].astype(np.float32))
        np.testing.assert_allclose(ctx.debug("psi", l).cpu().numpy(), ref.record["psi"][T - 1, l],
                                   rtol=1e-6, atol=1e-7)
        np.testing.assert_allclose(ctx.debug("L", l).cpu().numpy(), ref.record["L"][T - 1, l],
                                   rtol=1e-5, atol=1e-6)
        np.testing.assert_allclose(ctx.debug("y", l).cpu().numpy(), ref.record["y"][T - 1, l],
                                   rtol=1e-5, atol=1e-5)
    ctx.close()


# ---------------------------------------------------------------- boundary properties
def _wl():
    shape, seed, scale = RAGGED["ralif2_two_layers"]
    return synth.make_workload(shape, seed, input_scale=scale)


def _same_forward_close_grads(x, y, tol=1e-6):
    assert np.array_equal(x["spikes"], y["spikes"])
    for l in range(len(x["dW"])):
        assert rel_l2(x["dW"][l], y["dW"][l]) <= tol
        assert rel_l2(x["dWout"][l], y["dWout"][l]) <= tol
    assert abs(x["loss"] - y["loss"]) <= tol * abs(y["loss"])


def test_sequence_equals_steps():
    # run_sequence works in blocks of steps; T single steps give the same
    # spikes and neuron state, and the gradient up to summation order.
    wl = _wl()
    ctx_a = eprop.EpropContext(wl.shape, wl.W, wl.Wout)
    a = gpu_run(wl, ctx=ctx_a)
    ctx = eprop.EpropContext(wl.shape, wl.W, wl.Wout)
    x, labels = to_dev(wl)
    spikes = ctx.new_spike_buffer(wl.shape.T)
    for t in range(wl.shape.T):
        ctx.step(x[t], labels, spikes[t])
    dW, dWout, loss = ctx.get_grads()
    torch.cuda.synchronize()
    b = dict(spikes=spikes.cpu().numpy().view(np.uint32), dW=[d.cpu().numpy() for d in dW],
             dWout=[d.cpu().numpy() for d in dWout], loss=float(loss.cpu()))
    _same_forward_close_grads(b, a)
    for l in range(wl.shape.n_layers):
        for name in ("v", "a"):
            assert torch.equal(ctx.debug(name, l), ctx_a.debug(name, l))
    ctx.close()
    ctx_a.close()


def test_split_sequence_and_determinism():
    wl = _wl()
    a = gpu_run(wl)
    b = gpu_run(wl, chunks=[7, 1, wl.shape.T - 8])
    c = gpu_run(wl)
    _same_forward_close_grads(b, a)
    assert np.array_equal(c["spikes"], a["spikes"])
    for l in range(wl.shape.n_layers):
        assert np.array_equal(c["dW"][l], a["dW"][l])
        assert np.array_equal(c["dWout"][l], a["dWout"][l])
    assert c["loss"] == a["loss"]


def test_reset_starts_a_new_sequence_and_reads_new_weights():
    wl = _wl()
    a = gpu_run(wl)
    ctx = eprop.EpropContext(wl.shape, wl.W, wl.Wout)
    x, labels = to_dev(wl)
    ctx.run_sequence(x[:9], labels)
    # change the weights in place, then reset: the new values must be used
    for w in ctx.weights:
        w.mul_(0.5)
    ctx.reset()
    half = synth.Workload(wl.shape, [w * 0.5 for w in wl.W], [w * 0.5 for w in wl.Wout],
                          wl.labels, wl.x, wl.rates)
    b = gpu_run(half, ctx=ctx)
    ref_half = gpu_run(half)
    assert np.array_equal(b["spikes"], ref_half["spikes"])
    for l in range(wl.shape.n_layers):
        assert np.array_equal(b["dW"][l], ref_half["dW"][l])
    for w in ctx.weights:
        w.mul_(2.0)
    ctx.reset()
    c = gpu_run(wl, ctx=ctx)
    assert np.array_equal(c["dW"][0], a["dW"][0]) and np.array_equal(c["spikes"], a["spikes"])
    ctx.close()


def test_grads_before_any_step_are_zero():
    wl = _wl()
    ctx = eprop.EpropContext(wl.shape, wl.W, wl.Wout)
    dW, dWout, loss = ctx.get_grads()
    torch.cuda.synchronize()
    assert all(not d.any() for d in dW) and all(not d.any() for d in dWout)
    assert float(loss.cpu()) == 0.0
    ctx.close()


def test_out_of_range_label_is_reported():
    wl = _wl()
    ctx = eprop.EpropContext(wl.shape, wl.W, wl.Wout)
    x, labels = to_dev(wl)
    labels[1] = wl.shape.n_out       # one past the last class
    ctx.run_sequence(x[:3], labels)
    assert ctx.status() == eprop.EPROP_ESTATE
    ctx.reset()
    labels[1] = 0
    ctx.run_sequence(x[:3], labels)
    assert ctx.status() == 0
    ctx.close()


def test_error_codes_on_device():
    wl = _wl()
    cfg = eprop.make_config(wl.shape)
    n = eprop.eprop_workspace_bytes(cfg)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    ws = ws[(-ws.data_ptr()) % 256:]
    weights = []
    for l in range(wl.shape.n_layers):
        weights += [torch.from_numpy(wl.W[l]).cuda(), torch.from_numpy(wl.Wout[l]).cuda()]
    with pytest.raises(eprop.EpropError) as e:
        eprop.eprop_init(cfg, ws[: n - 512], weights)
    assert e.value.code == eprop.EPROP_ENOSPACE
    ctx = eprop.eprop_init(cfg, ws, weights)
    x, labels = to_dev(wl)
    lib = eprop.load_library()
    assert lib.eprop_run_sequence(ctx, x.data_ptr(), 0, labels.data_ptr(), None) == eprop.EPROP_EINVAL
    assert lib.eprop_step(ctx, None, labels.data_ptr(), None) == eprop.EPROP_EINVAL
    assert "NULL" in eprop.eprop_last_error(ctx)
    eprop.eprop_destroy(ctx)


def test_device_memory_does_not_grow_with_sequence_length():
    shape = synth.WORKLOADS["rlif_b32_n256_t250"]
    used = {}
    ws = eprop.eprop_workspace_bytes(eprop.make_config(shape))
    for T in (50, 400):
        wl = synth.make_workload(shape, 2, T=T)
        x, labels = to_dev(wl)
        gc.collect()        # contexts of earlier tests must not be freed mid-measurement
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        ctx = eprop.EpropContext(shape, wl.W, wl.Wout)
        ctx.run_sequence(x, labels)
        ctx.get_grads()
        torch.cuda.synchronize()
        used[T] = torch.cuda.max_memory_allocated() - base
        ctx.close()
        del ctx, x
    assert used[50] == used[400], used
    assert ws <= used[50] <= ws + (8 << 20), (used, ws)
