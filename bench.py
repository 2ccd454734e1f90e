"""Throughput of the online e-prop hot path on one MI355X.

A step is one training sequence of the recurrent ALIF workload (B=128, 700
Bernoulli inputs, 1024 neurons of which 512 adaptive, 35 classes, T=1000):
reset, T online e-prop steps through eprop_run_sequence (drive, neuron step,
readout and learning signal, eligibility update and gradient accumulation at
every timestep), then the gradient read-out.  Inputs and weights are seeded
synthetic data already resident in HBM when the clock starts.

Prints one JSON line: synapse-timestep updates per second
(sum over layers of B * N_pre * N_post * T per second), the roofline of the
eligibility kernel, the largest share of the step's device work (algorithmic
HBM bytes per launch over its measured duration, from HIP events on its
stream, against the HBM peak; its algorithmic matrix operations against the
fp16 MFMA peak alongside), and the CPU oracle timed on a bounded sample on
this host.

Counter runs: `--calibrate-copy MIB` adds device-to-device copies of a known
size after the timed steps, so that FETCH_SIZE/WRITE_SIZE of the eligibility
kernel can be scaled by what the same counters read for a plain copy;
`--summarize-counters FETCH_DIR WRITE_DIR` turns the two rocprofv3 CSV
outputs into profiles/trace_kernel_counters.json.
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
HBM_PEAK_GBS = 8000.0              # MI355X published HBM3E bandwidth
FP16_MATRIX_PEAK_TFLOPS = 2500.0   # MI355X published dense fp16 matrix (MFMA) peak
COPY_KERNEL = "copyBuffer"
COUNTERS = os.path.join(ROOT, "profiles", "trace_kernel_counters.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2501_11407_amd", "csrc", "kernels.hip")


def dims(shape):
    """(B, N, neurons with a second per-synapse state component, three-trace
    recursion): the reset path kept, or the two-compartment neuron (whose
    soma and dendrite eligibilities are both per-synapse)."""
    model = getattr(shape, "neuron_model", 0)
    rt = 1 if (getattr(shape, "reset_grad", 0) or model == 1) else 0
    return shape.batch, shape.n_rec, (shape.n_rec if model == 1 else shape.n_adaptive), rt


def trace_bytes(shape, layer: int, launches: int, first_launches: int, steps: int) -> int:
    """Algorithmic HBM bytes of eligibility-kernel launches on one layer.
    Per launch: ebar (every synapse) and eps^a (synapses onto adaptive
    neurons) read once and written once, one fp64 gradient accumulator of
    every (i, j) read and written once; the first launch after a reset reads
    neither.  Per timestep covered, the operands read once: the binary
    presynaptic vector [B, N_pre] (one bit each), the coefficients U, H
    [B, N] and V [B, N_adaptive] (4-byte pair words); per launch the seven
    scalars c, q, P, D and the three block-start coefficients [B, N], and
    the block-start filter [B, N_pre].  With the reset path kept
    (reset_grad = 1): eps^v (every synapse) as a third trace, a fourth
    coefficient row W [B, N], and nine scalars per (b, j)."""
    B, N, NA, rt = dims(shape)
    npre = shape.n_pre(layer)
    trace = 4 * B * npre * ((2 if rt else 1) * N + NA) + 8 * npre * N      # one direction
    rows = (3 if rt else 2) * N + NA
    scalars = 9 if rt else 7
    operands = (steps * B * (npre / 8 + 4 * rows) + launches * scalars * 4 * B * N
                + (0 if rt else launches * 4 * B * npre))
    return int((2 * launches - first_launches) * trace + operands)


BYTE_MODEL = ("block: per launch (one block of up to 512 steps), every trace read once and "
              "written once (4 B x B x N_pre x (N_post + N_adaptive) each way; the first launch "
              "after a reset reads none), the fp64 gradient accumulator read and written once "
              "(8 B x N_pre x N_post each way), the operands of the block's steps read once "
              "(B x N_pre bits of presynaptic spikes and 4 B x B x (2 N_post + N_adaptive) of "
              "coefficient pairs per step, plus 7 scalars per (b, j) and the block-start filter "
              "per launch)")


def per_step_model_bytes(shape, layer: int) -> int:
    """Bytes per timestep if every trace made a round trip at every step:
    per synapse 8 B of ebar, 8 B of eps^a onto adaptive neurons, and per
    (i, j) the fp64 accumulator read and written and W read (12 B over the
    batch)."""
    B, N, NA, rt = dims(shape)
    npre = shape.n_pre(layer)
    return 8 * B * npre * ((2 if rt else 1) * N + NA) + 12 * npre * N


def trace_flops(shape, layer: int, steps: int) -> int:
    """Algorithmic matrix operations of the eligibility kernel: per
    covered timestep and synapse, one multiply-add (2 operations) in each of
    the contractions over the block's steps -- C_U and C_H for every
    synapse, C_V as well for synapses onto adaptive neurons (and, with the
    reset path kept, C_W for every synapse)."""
    B, N, NA, rt = dims(shape)
    npre = shape.n_pre(layer)
    return steps * B * npre * 2 * ((3 if rt else 2) * N + NA)


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


def summarize_counters(fetch_dir: str, write_dir: str, copy_mib: int) -> dict:
    """Reads the FETCH_SIZE and WRITE_SIZE rocprofv3 CSVs (KiB per dispatch),
    scales each by copy bytes / the counter's reading for the plain copies,
    and writes profiles/trace_kernel_counters.json."""
    import csv
    import glob

    def per_kernel(d, counter):
        rows = []
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            rows += list(csv.DictReader(open(f)))
        trace = [float(r["Counter_Value"]) for r in rows
                 if r["Counter_Name"] == counter and "::trace_kernel<" in r["Kernel_Name"]]
        copies = [r for r in rows if r["Counter_Name"] == counter and COPY_KERNEL in r["Kernel_Name"]]
        big = max(int(r["Grid_Size"]) for r in copies)      # the calibration copies, not small ones
        copy = [float(r["Counter_Value"]) for r in copies if int(r["Grid_Size"]) == big]
        return trace, copy

    fetch_t, fetch_c = per_kernel(fetch_dir, "FETCH_SIZE")
    write_t, write_c = per_kernel(write_dir, "WRITE_SIZE")
    copy_kib = copy_mib * 1024.0
    f_scale = copy_kib / (sum(fetch_c) / len(fetch_c))
    w_scale = copy_kib / (sum(write_c) / len(write_c))
    fetch = sum(fetch_t) / len(fetch_t) * 1024.0 * f_scale
    write = sum(write_t) / len(write_t) * 1024.0 * w_scale
    out = {"workload": WORKLOAD, "kernel": "trace_kernel",
           "kernel_source_sha256": source_digest(),
           "dispatches": len(fetch_t), "fetch_bytes_per_launch": round(fetch),
           "write_bytes_per_launch": round(write), "hbm_bytes_per_launch": round(fetch + write),
           "copy_calibration": {"copy_bytes": copy_mib << 20, "fetch_scale": f_scale,
                                "write_scale": w_scale}}
    with open(COUNTERS, "w") as f:
        json.dump(out, f, indent=1)
    return out


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(wl, name: str, seconds_hint: float = 15.0):
    """The oracle (one thread, fp64 traces) over every synapse and all T
    steps of the first n_b batch elements, n_b chosen so that the run takes
    about seconds_hint on this host.  The process is pinned to one core for
    the measurement (the first core it may run on) and unpinned afterwards."""
    import oracle
    shape = wl.shape
    per_step = shape.syn_per_step() // shape.batch     # synapses of one batch element, all layers
    allowed = sorted(os.sched_getaffinity(0))
    core = allowed[0]
    os.sched_setaffinity(0, {core})
    try:
        t0 = time.perf_counter()
        oracle.run(shape, wl.W, wl.Wout, wl.x, wl.labels, b_lo=0, b_hi=1, want_spikes=False)
        probe = time.perf_counter() - t0
        n_b = int(min(shape.batch, max(1, round(seconds_hint / max(probe, 1e-6)))))
        t0 = time.perf_counter()
        oracle.run(shape, wl.W, wl.Wout, wl.x, wl.labels, b_lo=0, b_hi=n_b, want_spikes=False)
        dt = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, set(allowed))
    return {"value": n_b * per_step * shape.T / dt, "unit": "syn-steps/s", "cores": 1,
            "kind": "oracle", "pinned_core": core, "cpu_model": cpu_model(),
            "nproc": os.cpu_count(), "cores_allowed": len(allowed),
            "sample": f"batch elements 0..{n_b - 1} of {name} (of {shape.batch}), all "
                      f"{per_step} synapses, all {shape.T} timesteps: {dt:.1f} s on one thread "
                      f"pinned to core {core} (fp64 traces)"}


def copy_ceiling_gbs(torch, dev, mib: int = 1024, reps: int = 5) -> float:
    """Measured HBM ceiling: a device-to-device copy of `mib` MiB (read once
    and written once), bytes moved per second, best of `reps`, HIP events on
    the current stream."""
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    best = float("inf")
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        e1.synchronize()
        best = min(best, e0.elapsed_time(e1) * 1e-3)
    del src, dst
    return 2 * n / best / 1e9


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"))
    ap.add_argument("--copy-mib", type=int, default=1024)
    ap.add_argument("--reset-grad", type=int, default=0, choices=(0, 1),
                    help="1: the same workload with the reset path kept in the gradient")
    ap.add_argument("--neuron-model", type=int, default=0, choices=(0, 1),
                    help="1: the same workload with two-compartment neurons (no adaptive ones)")
    ap.add_argument("--online-every", type=int, default=0, metavar="K",
                    help="online weight application every K steps (learning rate --online-lr)")
    ap.add_argument("--online-lr", type=float, default=2.0 ** -12)
    ap.add_argument("--workload", default=WORKLOAD,
                    help="another named synthetic workload (the headline is the default)")
    ap.add_argument("--batch", type=int, default=0, metavar="B",
                    help="the named workload with another batch size (same seed and recipe)")
    args = ap.parse_args()
    if args.summarize_counters:
        print(json.dumps(summarize_counters(*args.summarize_counters, args.copy_mib)))
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the batch-sharded multi-GPU design is not built)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2501_11407_amd import eprop, synth

    if args.workload not in synth.WORKLOADS:
        print(f"unknown workload {args.workload}; one of {sorted(synth.WORKLOADS)}", file=sys.stderr)
        sys.exit(2)
    if args.batch:
        wl = synth.make_workload(synth.WORKLOADS[args.workload].replace(batch=args.batch),
                                 synth.WORKLOAD_SEED[args.workload])
    else:
        wl = synth.named_workload(args.workload)
    if args.reset_grad:
        wl.shape = wl.shape.replace(reset_grad=1)
    if args.neuron_model:
        wl.shape = wl.shape.replace(neuron_model=1, n_adaptive=0)
    shape = wl.shape
    workload = args.workload + (f"_batch{args.batch}" if args.batch else "") + \
        ("_reset_grad" if args.reset_grad else "") + \
        ("_two_compartment" if args.neuron_model else "") + \
        (f"_online{args.online_every}" if args.online_every else "")
    dev = torch.device("cuda:0")
    ctx = eprop.EpropContext(shape, wl.W, wl.Wout, device="cuda:0")
    if args.online_every:
        ctx.set_online(args.online_lr, args.online_every)
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
    alg_flops = sum(trace_flops(shape, l, args.steps * shape.T) for l in range(shape.n_layers))
    sec = trace_ms * 1e-3
    # Roofline of the eligibility kernel: its algorithmic HBM bytes take
    # longer at peak bandwidth than its algorithmic matrix operations at the
    # fp16 MFMA peak (the operands are fp16 hi/lo pairs), so it is bounded by
    # HBM; the matrix rate is reported beside it.
    achieved = alg_bytes / sec / 1e9
    tflops = alg_flops / sec / 1e12
    copy_gbs = copy_ceiling_gbs(torch, dev)
    # the same launches priced with the per-step byte model (every trace read
    # and written at every timestep): what an unblocked kernel would move
    per_step_bytes = sum(per_step_model_bytes(shape, l) for l in range(shape.n_layers)) * args.steps * shape.T
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "byte_model": BYTE_MODEL,
                "copy_ceiling_gbs": round(copy_gbs, 1),
                "frac_of_copy_ceiling": round(achieved / copy_gbs, 4),
                "per_step_model_bytes_per_launch": round(per_step_bytes / n_timed),
                "per_step_model_gbs": round(per_step_bytes / sec / 1e9, 1),
                "traffic": (None if (args.reset_grad or args.neuron_model or args.online_every or args.batch
                                     or args.workload != WORKLOAD)
                            else stored_traffic(shape)),
                "kernel": "trace_kernel", "avg_launch_us": round(trace_ms * 1e3 / n_timed, 2),
                "steps_per_launch": round(timed_steps / n_timed, 2),
                "alg_hbm_bytes_per_launch": round(alg_bytes / n_timed),
                "alg_flops_per_launch": round(alg_flops / n_timed),
                "alg_tflops": round(tflops, 2),
                "alg_tflops_frac_fp16_peak": round(tflops / FP16_MATRIX_PEAK_TFLOPS, 4)}
    line = {
        "metric": "synapse-timestep e-prop updates/sec (B*N_pre*N_post*T/s) + % HBM peak",
        "value": value, "unit": "syn-steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32 (contraction operands f16 hi/lo pairs)",
        "precision": "fp32 neuron state, traces and per-launch sums; fp64 gradient accumulators; "
                     "the eligibility contractions take their coefficient operands as scaled "
                     "fp16 hi/lo pairs (about 22 significant bits) against the exact binary "
                     "presynaptic values, with fp32 accumulation",
        "data": "synthetic (seeded Bernoulli spike inputs, quantised Gaussian weights)",
        "config": {"workload": workload, "batch": shape.batch, "n_in": shape.n_in,
                   "n_rec": shape.n_rec, "n_adaptive": shape.n_adaptive, "n_out": shape.n_out,
                   "T": shape.T, "layers": shape.n_layers, "reset_grad": args.reset_grad,
                   "neuron_model": args.neuron_model,
                   "parallelism": "single GPU"},
        "roofline": roofline,
    }
    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, workload)
    ctx.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
