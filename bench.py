"""Throughput of the online e-prop hot path on one MI355X.

A step is one training sequence of the recurrent ALIF workload (B=128, 700
Bernoulli inputs, 1024 neurons of which 512 adaptive, 35 classes, T=1000):
reset, T online e-prop steps through eprop_run_sequence (drive, neuron step,
readout and learning signal, eligibility update and gradient accumulation at
every timestep), then the gradient read-out.  Inputs and weights are seeded
synthetic data already resident in HBM when the clock starts.

Prints one JSON line: synapse-timestep updates per second
(sum over layers of B * N_pre * N_post * T per second), the roofline of the
eligibility kernel (algorithmic HBM bytes per launch over its measured
duration, from HIP events on its stream) and the CPU oracle timed on a
bounded sample on this host.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

WORKLOAD = "ralif_b128_n1024_t1000"
HBM_PEAK_GBS = 8000.0
COUNTERS = os.path.join(ROOT, "profiles", "trace_kernel_counters.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2501_11407_amd", "csrc", "kernels.hip")


def trace_bytes(shape, layer: int, launches: int, first_launches: int, steps: int) -> int:
    """Algorithmic HBM bytes of eligibility-kernel launches on one layer.
    Per launch: ebar (every synapse) and eps^a (synapses onto adaptive
    neurons) read once and written once, the fp64 accumulator of every (i, j)
    read and written once; the first launch after a reset reads neither.  Per
    timestep covered: the filtered presynaptic vector [N_pre, B] and psi, L
    [B, N_post] read once."""
    B, N, NA = shape.batch, shape.n_rec, shape.n_adaptive
    npre = shape.n_pre(layer)
    trace = 4 * B * npre * (N + NA) + 8 * npre * N      # one direction
    return (2 * launches - first_launches) * trace + steps * 4 * (B * npre + 2 * B * N)


def source_digest() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def stored_traffic(shape):
    """HBM bytes per launch of the eligibility kernel from the committed
    rocprofv3 counter summary, if it was taken on the current kernel source."""
    try:
        with open(COUNTERS) as f:
            c = json.load(f)
    except (OSError, ValueError):
        return None
    if c.get("kernel_source_sha256") != source_digest() or c.get("workload") != WORKLOAD:
        return None
    return c.get("hbm_bytes_per_launch")


def cpu_baseline(wl, seconds_hint: float = 20.0):
    """The oracle (one thread, fp64 traces) on batch element 0, every synapse,
    the first T_s timesteps, T_s chosen to take about seconds_hint."""
    import oracle
    shape = wl.shape
    per_step = shape.n_pre(0) * shape.n_rec
    # probe a few steps to size the sample
    T_probe = 20
    t0 = time.perf_counter()
    oracle.run(shape, wl.W, wl.Wout, wl.x, wl.labels, T=T_probe, b_lo=0, b_hi=1, want_spikes=False)
    dt = time.perf_counter() - t0
    T_s = int(min(shape.T, max(T_probe, T_probe * seconds_hint / max(dt, 1e-6))))
    t0 = time.perf_counter()
    oracle.run(shape, wl.W, wl.Wout, wl.x, wl.labels, T=T_s, b_lo=0, b_hi=1, want_spikes=False)
    dt = time.perf_counter() - t0
    return {"value": per_step * T_s / dt, "unit": "syn-steps/s", "cores": 1, "kind": "oracle",
            "sample": f"batch element 0 of {WORKLOAD}, all {per_step} synapses, first {T_s} of "
                      f"{shape.T} timesteps, {dt:.1f} s, single-threaded fp64 oracle"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the batch-sharded multi-GPU design is not built)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2501_11407_amd import eprop, synth

    wl = synth.named_workload(WORKLOAD)
    shape = wl.shape
    dev = torch.device("cuda:0")
    ctx = eprop.EpropContext(shape, wl.W, wl.Wout, device="cuda:0")
    x = torch.from_numpy(wl.x).to(dev)
    labels = torch.from_numpy(wl.labels).to(dev)

    def one_step():
        ctx.reset()
        ctx.run_sequence(x, labels)
        return ctx.get_grads()

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    max_launch = args.steps * shape.T * shape.n_layers
    ctx.profile_begin(max_launch)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        grads = one_step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    trace_ms, n_timed, timed_steps = ctx.profile_end()
    assert timed_steps == args.steps * shape.T * shape.n_layers
    assert ctx.status() == 0
    assert all(bool(torch.isfinite(g).all()) for g in grads[0] + grads[1])

    syn_steps = shape.syn_per_step() * shape.T * args.steps
    value = syn_steps / elapsed
    per_layer_launches = n_timed // shape.n_layers
    alg_bytes = sum(trace_bytes(shape, l, per_layer_launches, args.steps, args.steps * shape.T)
                    for l in range(shape.n_layers))
    achieved = alg_bytes / (trace_ms * 1e-3) / 1e9
    traffic = stored_traffic(shape)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": "trace_kernel", "avg_launch_us": round(trace_ms * 1e3 / n_timed, 2),
                "steps_per_launch": round(timed_steps / n_timed, 2),
                "alg_bytes_per_launch": round(alg_bytes / n_timed)}
    line = {
        "metric": "synapse-timestep e-prop updates/sec (B*N_pre*N_post*T/s) + % HBM peak",
        "value": value, "unit": "syn-steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded Bernoulli spike inputs, quantised Gaussian weights)",
        "config": {"workload": WORKLOAD, "batch": shape.batch, "n_in": shape.n_in,
                   "n_rec": shape.n_rec, "n_adaptive": shape.n_adaptive, "n_out": shape.n_out,
                   "T": shape.T, "layers": shape.n_layers, "parallelism": "single GPU"},
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl)
    ctx.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
