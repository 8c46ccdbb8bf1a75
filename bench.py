"""Throughput of BCPNN hidden-layer training on one MI355X.

Workload: the MNIST-shaped unsupervised layer -- 60000 synthetic 28x28 images encoded as 784
input HCUs of 2 MCUs (x, 1 - x), a hidden layer of 30 HCUs x 100 MCUs with 10% receptive
fields, batch 128, alpha 1e-3, structural plasticity before every 100th batch of an epoch
(1-based), a fresh shuffle per epoch, the last batch of an epoch partial (96 samples).

A step is one batch of that schedule: the structural update when it is due (MI score + greedy
swap), then support, per-HCU softmax, trace, weight and bias updates.  The whole dataset, one
shuffled copy per epoch touched, is staged in HBM before timing.  W warm-up steps run first;
then exactly K steps are timed between two device synchronisations.  The timed region ends
with bcpnn_flush, so the silent-block trace updates of every timed batch (which the library
queues and applies a few batches at a time) are inside it, and no kernel in it carries
profiling events.

After the timed region, an untimed profiling pass continues the same schedule with every
kernel launch timed: the sweep, the weight pass and the structural update by HIP events
recorded on their stream right before and after them, the support and active-block kernels
(short launches on the caller's stream) by the device clock, stamped when their first
workgroup starts and their last one ends.  The kernel durations of the JSON line come from it:
the roofline position of the dominant kernel (the one with the most time per batch on the
caller's stream, which carries the schedule: the support, the active-block trace kernel, or,
where it runs on that stream, the sweep over the silent elements of Pij, per batch of its
launch), the sweep against the HBM roofline and the support against the fp64 matrix cores
(both reported, whichever dominates), the caller's stream per batch, and the structural update.  The line also
carries the whole-matrix weight pass, the STL-shaped layer (a short run of the same schedule on
the first images of that workload, with its weight pass), the forward-pass throughput by batch
size, and the CPU oracle on a bounded sample of the MNIST-shaped schedule on this host's cores
(all threads, and one).
"""
from __future__ import annotations

import argparse
import faulthandler
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "train samples/s, MNIST-shaped 30x100 BCPNN layer; % MFMA peak, HBM GB/s"
PEAK_HBM_GBS = 8000.0
PEAK_F64_MFMA_TFS = 78.6
PEAK_BF16_MFMA_TFS = 2500.0
PEAK_F32_MFMA_TFS = 157.3
# Batches whose silent-element updates one sweep applies (the library's kMaxSweepBatches).
SWEEP_BATCHES = 8
# In the profiling pass after the timed region, every PROFILE_PERIOD-th launch of each kernel
# is timed.
PROFILE_PERIOD = 1
PROFILE_SYNC = 64             # steps of the profiling pass between two reads of the timers
# Launches of the whole-matrix weight pass timed after the training run.
WEIGHT_PASSES = 20
# Structural updates timed after the profiling pass.
STRUCTURAL_TIMED = 3
# Forward-pass batch sizes of the inference sweep.
INFERENCE_BATCHES = [1, 8, 32, 128, 512, 2048, 8192]
# STL-shaped leg of the default line: warm-up and timed batches (the first images of the set).
STL_WARMUP, STL_STEPS = 2, 16

# Memory traffic per launch (bytes between the L2 caches and the memory side: HBM and the
# Infinity Cache) of the support, the sweep and the weight pass, from two rocprofv3 counter runs
# of the same command, FETCH_SIZE and then WRITE_SIZE (KiB per dispatch), each scaled by what
# it reads for a plain 256 MiB device copy (`bench.py --calibrate-copy`: FETCH_SIZE 131084.5
# KiB, WRITE_SIZE 262144 KiB, so factors 1.99981 and 1).  The request counters (128 RDREQ_128B
# + 64 RDREQ_64B + 32 RDREQ_32B read, 64 WRREQ_64B + 32 (WRREQ - WRREQ_64B) written, exact for
# the copy with no factor) give the same within 1.2%.  Keyed by workload and the SHA-256 of the
# kernel's sources (kernel_digest); a changed source reports null until measured again.  The
# sweep's figure is for the counter run's average launch (MNIST shape: 7.65 batches per launch;
# STL shape: 5.56), the others' for every launch (the support's for its training launches).
_SWEEP_DIGEST = "09b18091e61eed64d84faad69563bb73b5ee4fdc99dcee19b7fe35fa7b268136"
_WEIGHT_DIGEST = "329f407e0161ecbbac0607fb9d21c5a0a53d6248efd521244ed72615f3c0d97b"
_SUPPORT_DIGEST = "c8dcdc430cafc6230ea9f8fbd0acd4e435d1500db73bd5e3a89819fd5bb6df6e"
MEASURED_TRAFFIC = {("mnist", _SWEEP_DIGEST): 92.71e6, ("stl", _SWEEP_DIGEST): 9855.62e6}
MEASURED_WEIGHT_TRAFFIC = {("mnist", _WEIGHT_DIGEST): 21.90e6, ("stl", _WEIGHT_DIGEST): 2406.11e6}
MEASURED_SUPPORT_TRAFFIC = {("mnist", _SUPPORT_DIGEST): 11.65e6, ("stl", _SUPPORT_DIGEST): 2692.97e6}


def kernel_digest(csrc, files):
    """SHA-256 over the named source files of one kernel (its .hip file and the headers it
    includes): a measured traffic figure holds only for the sources it was taken with."""
    h = hashlib.sha256()
    for name in files:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


SWEEP_SOURCES = ("k_trace.hip", "bcpnn_internal.h", "device_common.h")
WEIGHT_SOURCES = ("k_weights.hip", "bcpnn_internal.h", "device_common.h")
SUPPORT_SOURCES = ("k_support.hip", "bcpnn_internal.h", "device_common.h")


def sweep_sizes(sched, first, last):
    """Batches per sweep launch over steps [first, last), mirroring the library: the pending
    batches are swept once SWEEP_BATCHES have accumulated and before every structural update;
    the sweeps start from an empty queue (the previous pass ended with a flush) and the rest is
    flushed at the end."""
    sizes, pend = [], 0
    for s in range(first, last):
        if sched[s][4] and pend:
            sizes.append(pend)
            pend = 0
        pend += 1
        if pend == SWEEP_BATCHES:
            sizes.append(pend)
            pend = 0
    if pend:
        sizes.append(pend)
    return sizes


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2345, help="timed batches (5 epochs = 2345)")
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="mnist",
                    choices=["mnist", "stl", "stl_shard8", "mnist_pipeline"],
                    help="mnist / stl: hidden-layer training (the metric); stl_shard8: one GPU's "
                         "share of the STL-shaped layer sharded by hidden HCU over eight GPUs; "
                         "mnist_pipeline: the hidden layer plus a supervised readout, then "
                         "held-out inference")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="time budget of the all-threads CPU-oracle sample (0 = skip); the "
                         "one-thread sample gets half of it")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--launch", choices=["eager", "graph"], default="eager",
                    help="how the steps of the timed region are issued: eager, one library call "
                         "per step; graph, the steps' calls captured once into a HIP graph before "
                         "the timed region and replayed once inside it.  The other way is timed "
                         "on the following steps and reported beside it")
    ap.add_argument("--no-extras", action="store_true",
                    help="only the MNIST-shaped line: no STL-shaped leg, no inference sweep")
    ap.add_argument("--no-pairs", action="store_true",
                    help="contract every input unit instead of exploiting the (x, 1 - x) pixel "
                         "pairs (complement_pairs = 0)")
    ap.add_argument("--precision-report", action="store_true",
                    help="reduced-precision storage (bf16, 10-bit mantissa) on the MNIST-shaped "
                         "layer against the fp32 oracle: trace and weight errors, masks, codes")
    ap.add_argument("--inference-sweep", action="store_true",
                    help="only the forward-pass throughput of the MNIST-shaped layer by batch size")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 256 MiB device copy (HBM counter calibration)")
    return ap.parse_args()


def schedule(n_train, batch, period, n_steps):
    """(epoch, batch index within epoch (0-based), start, size, plasticity-before?) per step."""
    per_epoch = (n_train + batch - 1) // batch
    out = []
    for s in range(n_steps):
        e, k = divmod(s, per_epoch)
        start = k * batch
        size = min(batch, n_train - start)
        out.append((e, k, start, size, period > 0 and (k + 1) % period == 0))
    return out


def stage(msg):
    """A progress line on stderr (the JSON line alone goes to stdout)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def main():
    faulthandler.enable()          # a native crash prints the Python stack of every thread
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU only (got --gpus {args.gpus}); the "
              "multi-GPU design is described in DESIGN.md and not run.", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.calibrate_copy:
        # A plain copy of known size: 256 MiB read + 256 MiB written per launch.
        src = torch.ones(64 << 20, device="cuda", dtype=torch.float32)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "copy", "bytes_read": src.numel() * 4,
                          "bytes_written": dst.numel() * 4, "launches": 5}))
        return

    if args.workload == "mnist_pipeline":
        return run_pipeline(args)
    if args.precision_report:
        return run_precision_report(args)
    if args.inference_sweep:
        print(json.dumps(run_inference_sweep()), flush=True)
        return

    from paper_2106_05373_amd import synth
    w = synth.WORKLOADS[args.workload]
    pairs = 0 if args.no_pairs else int(w.complement_pairs)
    # (the STL-shaped layers stage 1.1 GB per epoch the schedule touches: a short profiling pass)
    res = measure_training(w, args.warmup, args.steps, pairs,
                           profile_steps=None if args.workload == "mnist" else args.steps,
                           launch=args.launch,
                           profile_period=PROFILE_PERIOD if args.workload == "mnist" else 1)

    out = {
        "metric": METRIC, "value": res["value"], "unit": "samples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": res["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic", "config": res["config"], "roofline": res["roofline"],
        "sweep": res["sweep"], "mfma": res["mfma"], "contraction": res["contraction"],
        "critical_path": res["critical_path"], "structural_update": res["structural_update"],
        "weight_pass": res["weight_pass"],
    }
    if not args.no_extras and args.workload == "mnist":
        stl = synth.WORKLOADS["stl"]
        r = measure_training(stl, STL_WARMUP, STL_STEPS, int(stl.complement_pairs),
                             profile_steps=STL_STEPS, launch=args.launch, profile_period=1)
        out["stl"] = {"value": r["value"], "unit": "samples/s", "ms_per_step": r["ms_per_step"],
                      "steps": STL_STEPS, "warmup": STL_WARMUP, "config": r["config"],
                      "roofline": r["roofline"], "sweep": r["sweep"], "mfma": r["mfma"],
                      "contraction": r["contraction"],
                      "critical_path": r["critical_path"],
                      "structural_update": r["structural_update"],
                      "weight_pass": r["weight_pass"]}
        stage("inference sweep")
        out["inference_sweep"] = run_inference_sweep()["sweep"]
    if not args.no_cpu_baseline and args.cpu_seconds > 0 and args.workload == "mnist":
        stage("CPU oracle baseline")
        out["cpu_baseline"] = cpu_baseline(w, res["mask"], args.cpu_seconds)
    print(json.dumps(out), flush=True)


def measure_training(w, warmup, steps, pairs, profile_steps=None, n_images=None,
                     launch="eager", profile_period=PROFILE_PERIOD):
    """Trains the workload's layer on its schedule: `warmup` untimed steps, `steps` timed
    between two synchronisations (ending with bcpnn_flush), then an untimed profiling pass of
    the following steps with every kernel launch timed (events around the sweep, device-clock
    stamps in the support and active-block kernels), structural updates and weight passes
    timed by events.  Returns the fields of the JSON line."""
    import torch
    from paper_2106_05373_amd import bcpnn, synth

    L = w.layer
    B = w.batch
    if profile_steps is None:
        profile_steps = min(max(steps, 64), 512)
    n_train = n_images if n_images is not None else w.n_train
    n_other = steps                  # the other launch mode, timed on the following steps
    n_steps = warmup + steps + n_other + profile_steps
    sched = schedule(n_train, B, w.period, n_steps)
    epochs = sorted({s[0] for s in sched})

    # ---- data staged on the device (not timed) -----------------------------------------
    stage(f"{w.name}: staging {len(epochs)} epoch copies of the inputs ({n_steps} steps)")
    t0 = time.time()
    px, _ = synth.dataset(w, n=n_images)
    X = torch.from_numpy(synth.encode_pixels(px))
    del px
    dev = torch.device("cuda", 0)
    shuffled = {}
    for e in epochs:
        perm = torch.from_numpy(synth.epoch_permutation(n_train, w.seed_shuffle, e))
        shuffled[e] = X[perm].to(dev).contiguous()
    del X
    k_act = synth.active_count(L.in_hcu, w.mask_frac)
    mask = synth.random_mask(L.in_hcu, L.out_hcu, k_act, w.seed_mask)
    prep_s = time.time() - t0

    stream = torch.cuda.Stream(device=dev)
    cfg = bcpnn.default_config(L.in_hcu, L.in_mcu, L.out_hcu, L.out_mcu, B, alpha=w.alpha,
                               gain=w.gain, bias_gain=w.bias_gain, init_noise=w.init_noise,
                               seed=w.seed_noise, complement_pairs=pairs)
    stage(f"{w.name}: layer {L.in_hcu}x{L.in_mcu} -> {L.out_hcu}x{L.out_mcu}, batch {B}, "
          f"complement pairs {pairs}")
    layer = bcpnn.Layer(cfg, mask, stream=stream)

    def step(s):
        e, k, start, size, plastic = sched[s]
        if plastic:
            layer.structural_update(count=False)
        layer.train_batch(shuffled[e][start:start + size])

    torch.cuda.synchronize()
    for s in range(warmup):
        step(s)
    layer.flush()
    torch.cuda.synchronize()

    # ---- the timed region: exactly `steps` steps, no profiling events ----------------------
    def timed(a, b, how):
        """Steps [a, b) then the flush, between two synchronisations; seconds."""
        graph = None
        if how == "graph":
            # the same library calls, recorded once (nothing runs during capture)
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=stream):
                for s in range(a, b):
                    step(s)
                layer.flush()
            torch.cuda.synchronize()
        t_start = time.perf_counter()
        if graph is not None:
            with torch.cuda.stream(stream):
                graph.replay()
        else:
            for s in range(a, b):
                step(s)
            layer.flush()          # the queued silent-block updates of the timed batches
        torch.cuda.synchronize()
        return time.perf_counter() - t_start

    first, last = warmup, warmup + steps
    stage(f"{w.name}: {warmup} warm-up steps done; timing {steps} steps ({launch})")
    wall_s = timed(first, last, launch)
    samples = sum(sched[s][3] for s in range(first, last))
    plastic_steps = sum(sched[s][4] for s in range(first, last))
    other = "graph" if launch == "eager" else "eager"
    stage(f"{w.name}: timing the next {n_other} steps ({other})")
    el = timed(last, last + n_other, other)
    other_fig = {"launch": other,
                 "value": round(sum(sched[s][3] for s in range(last, last + n_other)) / el, 1),
                 "ms_per_step": round(el * 1e3 / n_other, 5),
                 "steps": f"the {n_other} steps after the timed ones, timed the same way"}
    last += n_other

    # ---- untimed profiling pass: the following steps, every profile_period-th launch of each
    # kernel timed (sampled, so that the stream keeps the schedule's pace) ------------------
    stage(f"{w.name}: profiling pass of {profile_steps} steps")
    for k in bcpnn.KERNELS:
        layer.profile_read_kernel(k)                             # discard older records
    layer.profile_enable(profile_period)
    prof = {k: (0.0, 0) for k in ("sweep", "support", "active")}

    def collect():
        # reading waits for the stream and returns the layer's event pairs for reuse: every
        # PROFILE_SYNC steps, so that few timed launches are queued and few event
        # pairs exist at any time (the runtime has aborted with thousands of both)
        for k in prof:
            ms, n = layer.profile_read_kernel(k)
            prof[k] = (prof[k][0] + ms, prof[k][1] + n)

    for s in range(last, n_steps):
        step(s)
        if (s - last) % PROFILE_SYNC == PROFILE_SYNC - 1:
            collect()
    layer.flush()
    collect()
    layer.profile_read_kernel("structural")                      # any due inside the pass
    layer.profile_enable(1)
    stage(f"{w.name}: structural updates and weight passes")
    for _ in range(STRUCTURAL_TIMED):
        layer.structural_update(count=False)
    su_ms, su_n = layer.profile_read_kernel("structural")
    # the whole-matrix log-weight pass (recompute_weights), timed the same way
    for _ in range(WEIGHT_PASSES):
        layer.recompute_weights()
    wp_ms, wp_n = layer.profile_read_kernel("weights")
    layer.profile_enable(0)
    layer.close()

    csrc = os.path.join(ROOT, "paper_2106_05373_amd", "csrc")
    traffic_key = w.name if pairs else w.name + ":unpaired"
    prof_samples = sum(sched[s][3] for s in range(last, n_steps))
    avg_b = prof_samples / max(profile_steps, 1)
    b_pad = 16 * ((B + 15) // 16)
    active = k_act * L.in_mcu * L.n_out
    E = L.n_in * L.n_out

    # ---- the silent-element sweep against the HBM roofline ---------------------------------
    # Per launch it must read every Pij and write those of silent blocks (4 + 4 bytes per silent
    # element, 4 per active one), and read the split operands of each batch it applies once
    # (bf16 hi and lo of x and t, 4 bytes per element per padded batch row; with complement
    # pairs x covers the first unit of each input HCU only, and the column sums of t per
    # 16-row tile are read as well).
    every = "every launch" if profile_period == 1 else f"one launch in {profile_period}"
    sizes = sweep_sizes(sched, last, n_steps)
    # the library's choice of sweep: one workgroup per CU when the matrix has at most 64
    # 32 x 32 blocks per CU, LDS-staged tiles otherwise
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    small_sweep = ((L.n_in + 31) // 32) * ((L.n_out + 31) // 32) <= 64 * n_cu
    per_sweep = sum(sizes) / len(sizes)
    pij_bytes = 4.0 * E + 4.0 * (E - active)
    n_x = L.in_hcu if pairs else L.n_in            # input units the contraction covers
    ops_bytes = 4.0 * (n_x + L.n_out) * b_pad + (4.0 * L.n_out * (b_pad // 16) if pairs else 0.0)
    bytes_per_launch = pij_bytes + per_sweep * ops_bytes
    sweep_ms, sweep_n = prof["sweep"]
    if sweep_n == 0 or sweep_ms <= 0:
        raise RuntimeError("no sweep launch was timed")
    avg_sweep_s = sweep_ms / 1e3 / sweep_n
    achieved_gbs = bytes_per_launch / avg_sweep_s / 1e9
    traffic = MEASURED_TRAFFIC.get((traffic_key, kernel_digest(csrc, SWEEP_SOURCES)))
    sweep = {
        "bound": "hbm", "achieved": round(achieved_gbs, 1), "peak": PEAK_HBM_GBS,
        "unit": "GB/s", "frac": round(achieved_gbs / PEAK_HBM_GBS, 4), "traffic": traffic,
        "kernel": ("trace_sweep_pair" if pairs else "trace_sweep") +
                  ("_kernel" if small_sweep else
                   ("_tile_sum_kernel" if pairs and w.storage == "f32" else "_tile_kernel")) +
                  " (silent-block trace sweep: one read and one write of Pij for up to "
                  f"{SWEEP_BATCHES} queued batches, their x^T t contractions on split-bf16 MFMA; "
                  + ("one workgroup per CU on the layer's second stream beside later batches)"
                     if small_sweep else "LDS-staged tiles on the caller's stream; with pairs "
                     "and fp32 storage the batches' updates regrouped as c1^n P + R)"),
        "avg_us": round(avg_sweep_s * 1e6, 3), "timed_launches": sweep_n,
        "batches_per_launch": round(per_sweep, 3),
        "algorithmic_bytes_per_launch": bytes_per_launch,
        "timing": f"profiling pass of {profile_steps} steps after the timed region, "
                  f"{every} bracketed by events on its stream",
    }

    # ---- the joint-trace contraction against the bf16 matrix cores it runs on --------------
    # Algorithmic flops of X^T T over the units the sweep contracts (2 per multiply-add);
    # executed: three split-bf16 products per multiply-add.
    flops_alg = 2.0 * n_x * L.n_out * avg_b * per_sweep
    contraction = {
        "kernel": sweep["kernel"].split(" ")[0], "dtype": "bf16 (hi/lo split, 3 products)",
        "algorithmic_tflops": round(flops_alg / avg_sweep_s / 1e12, 3),
        "executed_tflops": round(3 * flops_alg / avg_sweep_s / 1e12, 3),
        "peak": PEAK_BF16_MFMA_TFS, "unit": "TFLOP/s",
        "frac_algorithmic": round(flops_alg / avg_sweep_s / 1e12 / PEAK_BF16_MFMA_TFS, 4),
        "frac_executed": round(3 * flops_alg / avg_sweep_s / 1e12 / PEAK_BF16_MFMA_TFS, 4),
        # the fp32-accurate contraction's rate against the fp32 matrix cores it would otherwise
        # run on (157.3 TFLOP/s dense)
        "algorithmic_over_fp32_mfma_peak": round(flops_alg / avg_sweep_s / 1e12 /
                                                 PEAK_F32_MFMA_TFS, 4),
    }

    # ---- the support GEMM on the fp64 matrix cores, and the caller's stream per batch --------
    sup_ms, sup_n = prof["support"]
    act_ms, act_n = prof["active"]
    avg_sup_s = sup_ms / 1e3 / max(sup_n, 1)
    sup_flops = 2.0 * avg_b * k_act * L.in_mcu * L.n_out
    mfma = {
        "kernel": "support_kernel (masked support on fp64 MFMA, per-HCU softmax, split operands)",
        "dtype": "f64", "achieved": round(sup_flops / avg_sup_s / 1e12, 3) if sup_n else None,
        "peak": PEAK_F64_MFMA_TFS, "unit": "TFLOP/s",
        "frac": round(sup_flops / avg_sup_s / 1e12 / PEAK_F64_MFMA_TFS, 4) if sup_n else None,
        "algorithmic_flops_per_launch": sup_flops, "avg_us": round(avg_sup_s * 1e6, 3),
        "timed_launches": sup_n,
    }
    avg_act_s = act_ms / 1e3 / max(act_n, 1)
    critical_path = {
        "stream": "caller's: support then active-block trace kernel, every batch",
        "support_us": round(avg_sup_s * 1e6, 3),
        "active_us": round(avg_act_s * 1e6, 3),
        "batch_us": round(wall_s * 1e6 / max(steps, 1), 3),
    }

    # ---- roofline of the dominant kernel: the one with the most time per batch on the caller's
    # stream, which carries the schedule (a small layer's sweep runs on the layer's second
    # stream beside the following batches, off that stream; a large layer's on it) -----------
    per_batch_us = {"support": avg_sup_s * 1e6, "active": avg_act_s * 1e6,
                    "sweep": avg_sweep_s * 1e6 / per_sweep}
    on_stream = [k for k in per_batch_us if k != "sweep" or not small_sweep]
    dominant = max(on_stream, key=per_batch_us.get)
    share = {"dominant": dominant,
             "us_per_batch": {k: round(v, 3) for k, v in per_batch_us.items()},
             "sweep_stream": "the layer's second stream, beside the following batches"
                             if small_sweep else "the caller's"}
    if dominant == "sweep":
        roofline = dict(sweep, **share)
    else:
        if dominant == "support":
            name, flops, avg_s, n, dtype, peak = (
                mfma["kernel"], sup_flops, avg_sup_s, sup_n, "f64", PEAK_F64_MFMA_TFS)
            traffic_s = MEASURED_SUPPORT_TRAFFIC.get(
                (traffic_key, kernel_digest(csrc, SUPPORT_SOURCES)))
        else:
            # the active blocks' joint-trace contraction, one product per multiply-add
            name = ("trace_active_pair_kernel" if pairs else "trace_active_kernel") + \
                   " (active-block trace, weight and marginal update, split-bf16 MFMA)"
            flops = 2.0 * avg_b * k_act * (1 if pairs else L.in_mcu) * L.n_out
            avg_s, n, dtype, peak, traffic_s = (avg_act_s, act_n, "bf16", PEAK_BF16_MFMA_TFS,
                                                None)
        achieved = flops / avg_s / 1e12
        roofline = {
            "bound": "mfma", "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4), "traffic": traffic_s, "kernel": name,
            "dtype": dtype, "avg_us": round(avg_s * 1e6, 3), "timed_launches": n,
            "algorithmic_flops_per_launch": flops,
            "timing": f"profiling pass of {profile_steps} steps after the timed region, "
                      f"{every} stamped by the kernel with the device clock "
                      "(first workgroup start to last workgroup end)", **share}
    su_s = su_ms / 1e3 / max(su_n, 1)
    structural_update = {
        "kernels": "mi_kernel + swap_kernel", "avg_us": round(su_s * 1e6, 3),
        "timed": su_n, "period_batches": w.period,
        "amortized_us_per_batch": round(su_s * 1e6 / w.period, 3) if w.period else 0.0,
        "in_timed_region": plastic_steps,
    }

    # ---- the log-weight pass over the whole matrix (recompute_weights) ----------------------
    # Per launch it writes every w and reads the Pij of active blocks (a silent weight is 0
    # whatever its trace), plus Pi, Pj and the mask.
    wp_bytes = 4.0 * E + 4.0 * active + 4.0 * (L.n_in + L.n_out) + L.in_hcu * L.out_hcu
    wp_s = wp_ms / 1e3 / max(wp_n, 1)
    weight_pass = {
        "kernel": "recompute_weights_vec_kernel (w = mask ? log(Pij / (Pi Pj)) : 0 over the "
                  "whole matrix, Pij read for active blocks only)",
        "bound": "hbm", "achieved": round(wp_bytes / wp_s / 1e9, 1) if wp_n else None,
        "peak": PEAK_HBM_GBS, "unit": "GB/s",
        "frac": round(wp_bytes / wp_s / 1e9 / PEAK_HBM_GBS, 4) if wp_n else None,
        "traffic": MEASURED_WEIGHT_TRAFFIC.get((traffic_key,
                                                kernel_digest(csrc, WEIGHT_SOURCES))),
        "algorithmic_bytes_per_launch": wp_bytes, "avg_us": round(wp_s * 1e6, 3),
        "timed_launches": wp_n,
    }
    config = {
        "workload": f"{w.name}: {n_train} synthetic images -> {L.in_hcu}x{L.in_mcu} inputs, "
                    f"hidden {L.out_hcu} HCUs x {L.out_mcu} MCUs, "
                    f"{int(round(w.mask_frac * 100))}% receptive fields, plasticity every "
                    f"{w.period} batches, alpha {w.alpha}",
        "global_batch": B, "samples_timed": samples, "structural_updates_timed": plastic_steps,
        "wall_s": round(wall_s, 6), "support_accumulation": "f64",
        "complement_pairs": bool(pairs), "data_staging_s": round(prep_s, 2),
        "timed_region": "K steps then bcpnn_flush (every queued silent-block update of the "
                        "timed batches applied), between two device synchronisations; no "
                        "profiling events",
        "launch": ("HIP graph: the K steps' library calls captured once before the timed "
                   "region, replayed once inside it" if launch == "graph" else
                   "eager: one library call per step inside the timed region"),
        "other_launch": other_fig,
        "parallelism": "single GPU",
    }
    return {"value": round(samples / wall_s, 1), "ms_per_step": round(wall_s * 1e3 / steps, 5),
            "config": config, "roofline": roofline, "sweep": sweep, "contraction": contraction,
            "mfma": mfma,
            "critical_path": critical_path, "structural_update": structural_update,
            "weight_pass": weight_pass, "mask": mask}


def run_pipeline(args):
    """Hidden layer (3 epochs, plasticity) + supervised 1 x 10 readout (1 epoch), then inference
    on 10000 held-out samples.  Prints one JSON line: training and inference throughput, held-out
    accuracy, and the argmax agreement with the oracle given the same trained states."""
    import torch
    import oracle
    from paper_2106_05373_amd import bcpnn, synth
    from paper_2106_05373_amd.pipeline import Network

    w = synth.WORKLOADS["mnist_pipeline"]
    L = w.layer
    B = w.batch
    dev = torch.device("cuda", 0)
    px, labels = synth.dataset(w)
    tx, tlabels = synth.dataset(w, split="test")
    X = synth.encode_pixels(px)
    Xt = torch.from_numpy(synth.encode_pixels(tx)).to(dev)
    onehot = synth.one_hot(labels, w.readout_mcu)
    mask = synth.random_mask(L.in_hcu, L.out_hcu, synth.active_count(L.in_hcu, w.mask_frac),
                             w.seed_mask)
    cfg = bcpnn.default_config(L.in_hcu, L.in_mcu, L.out_hcu, L.out_mcu, B, alpha=w.alpha,
                               gain=w.gain, bias_gain=w.bias_gain, init_noise=w.init_noise,
                               seed=w.seed_noise, complement_pairs=int(w.complement_pairs))
    net = Network(cfg, mask, w.readout_mcu)
    per_epoch = (w.n_train + B - 1) // B

    def epoch_data(e):
        perm = synth.epoch_permutation(w.n_train, w.seed_shuffle, e)
        return (torch.from_numpy(X[perm]).to(dev), torch.from_numpy(onehot[perm]).to(dev))

    # hidden layer: unsupervised, structural plasticity before every period-th batch
    t_hidden = 0.0
    for e in range(w.epochs):
        xe, _ = epoch_data(e)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(per_epoch):
            if w.period > 0 and (k + 1) % w.period == 0:
                net.hidden.structural_update(count=False)
            net.train_hidden(xe[k * B:(k + 1) * B])
        torch.cuda.synchronize()
        t_hidden += time.perf_counter() - t0
    # readout: supervised, hidden layer frozen
    t_read = 0.0
    for e in range(w.epochs, w.epochs + w.readout_epochs):
        xe, te = epoch_data(e)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(per_epoch):
            net.train_readout(xe[k * B:(k + 1) * B], te[k * B:(k + 1) * B])
        torch.cuda.synchronize()
        t_read += time.perf_counter() - t0
    # held-out inference
    pred = torch.empty(len(tlabels), device=dev, dtype=torch.int32)
    for k in range(0, len(tlabels), B):                      # warm-up pass
        net.predict(Xt[k:k + B], out=pred[k:k + B])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(0, len(tlabels), B):
        net.predict(Xt[k:k + B], out=pred[k:k + B])
    torch.cuda.synchronize()
    t_inf = time.perf_counter() - t0
    pred = pred.cpu().numpy()

    # the oracle's inference from the same trained states
    hs, rs = net.hidden.get_state(), net.readout.get_state()
    ho = oracle.OracleLayer(oracle.make_params(L.in_hcu, L.in_mcu, L.out_hcu, L.out_mcu,
                                               gain=w.gain, bias_gain=w.bias_gain), hs["mask"])
    ho.set_state(hs)
    ro = oracle.OracleLayer(oracle.make_params(L.out_hcu, L.out_mcu, 1, w.readout_mcu), rs["mask"])
    ro.set_state(rs)
    t0 = time.perf_counter()
    xt_host = Xt.cpu().numpy()
    ora = np.concatenate([ro.readout(ho.forward(xt_host[k:k + 1000])[1])[:, 0]
                          for k in range(0, len(tlabels), 1000)])
    t_ora = time.perf_counter() - t0
    n_train = per_epoch * B
    out = {
        "metric": "C2 pipeline: held-out inference samples/s (hidden forward + readout argmax)",
        "value": round(len(tlabels) / t_inf, 1), "unit": "samples/s", "n_gpus": 1,
        "higher_is_better": True, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{w.name}: hidden {L.in_hcu}x{L.in_mcu} -> {L.out_hcu}x{L.out_mcu} "
                               f"for {w.epochs} epochs (alpha {w.alpha}, gain {w.gain}, k_B "
                               f"{w.bias_gain}, plasticity every {w.period} batches), "
                               f"readout {L.out_hcu}x{L.out_mcu} -> 1x{w.readout_mcu} for "
                               f"{w.readout_epochs} epoch, {len(tlabels)} held-out samples",
                   "global_batch": B},
        "hidden_train_samples_per_s": round(w.epochs * w.n_train / t_hidden, 1),
        "readout_train_samples_per_s": round(w.readout_epochs * w.n_train / t_read, 1),
        "heldout_accuracy": round(float(np.mean(pred == tlabels)), 4),
        "oracle_heldout_accuracy": round(float(np.mean(ora == tlabels)), 4),
        "oracle_argmax_agreement": round(float(np.mean(pred == ora)), 6),
        "oracle_inference_samples_per_s": round(len(tlabels) / t_ora, 1),
        "oracle_cores": oracle.threads(),
    }
    print(json.dumps(out), flush=True)
    net.close()


def adjusted_rand_index(a, b):
    """Adjusted Rand index of two labelings of the same items (Hubert and Arabie, 1985): 1 for
    identical partitions up to renaming, about 0 for independent ones."""
    a = np.unique(a, return_inverse=True)[1]
    b = np.unique(b, return_inverse=True)[1]
    n = len(a)
    table = np.zeros((a.max() + 1, b.max() + 1), np.int64)
    np.add.at(table, (a, b), 1)
    pairs = lambda m: (m * (m - 1) // 2).sum()
    sum_ij = pairs(table)
    sum_a, sum_b = pairs(table.sum(1)), pairs(table.sum(0))
    expected = sum_a * sum_b / (n * (n - 1) / 2)
    top = 0.5 * (sum_a + sum_b) - expected
    return 1.0 if top == 0 else float((sum_ij - expected) / top)


def run_precision_report(args):
    """Reduced-precision storage on the MNIST-shaped layer as configured for the throughput
    workload (alpha 1e-3, k_B 1, batch 128, 5 epochs of its schedule): Pij and w stored in fp32,
    bf16 or the 10-bit mantissa format on the GPU, each against the fp32 oracle's run on the same
    batches (free runs: neither is re-synchronised).  Per format and epoch: max-abs error of Pi,
    Pj and Pij, the largest scaled weight error, mask entries that differ, and over the last
    epoch the share of Pij elements left unchanged and that decreased (the expected bf16
    stagnation: at alpha 1e-3 a decay step is below half a bf16 ulp); then the hidden code of
    10000 held-out samples against the oracle's (winner identity per sample and hidden HCU, and
    the adjusted Rand index of the winner partitions).  Also, as in the paper's own precision
    study, what the readout pipeline learns per format."""
    import torch
    import oracle
    from paper_2106_05373_amd import bcpnn, synth

    w = synth.WORKLOADS["mnist"]
    L = w.layer
    B = w.batch
    dev = torch.device("cuda", 0)
    px, _ = synth.dataset(w)
    X = synth.encode_pixels(px)
    del px
    tx, _ = synth.dataset(w, split="test", n=10000)
    Xt = synth.encode_pixels(tx)
    mask = synth.random_mask(L.in_hcu, L.out_hcu, synth.active_count(L.in_hcu, w.mask_frac),
                             w.seed_mask)
    per_epoch = (w.n_train + B - 1) // B
    kw = dict(alpha=w.alpha, gain=w.gain, bias_gain=w.bias_gain, init_noise=w.init_noise,
              seed=w.seed_noise)

    def code(y):                                     # winning MCU of every hidden HCU
        return np.asarray(y).reshape(len(y), L.out_hcu, L.out_mcu).argmax(-1)

    def say(msg):
        print(f"[precision report] {msg}", file=sys.stderr, flush=True)

    # the fp32 oracle, states at the end of every epoch
    t0 = time.perf_counter()
    ora = oracle.OracleLayer(oracle.make_params(L.in_hcu, L.in_mcu, L.out_hcu, L.out_mcu, **kw),
                             mask)
    ora_states = []
    for e in range(w.epochs):
        Xe = X[synth.epoch_permutation(w.n_train, w.seed_shuffle, e)]
        for k in range(per_epoch):
            if w.period > 0 and (k + 1) % w.period == 0:
                ora.structural_update()
            ora.train_batch(Xe[k * B:(k + 1) * B])
        ora_states.append(ora.get_state())
        say(f"oracle epoch {e + 1} of {w.epochs} ({time.perf_counter() - t0:.0f} s)")
    code_o = code(ora.forward(Xt)[1])
    t_oracle = time.perf_counter() - t0

    formats = {}
    for st in ("f32", "bf16", "m10"):
        cfg = bcpnn.default_config(L.in_hcu, L.in_mcu, L.out_hcu, L.out_mcu, B, storage=st,
                                   complement_pairs=int(w.complement_pairs), **kw)
        layer = bcpnn.Layer(cfg, mask)
        epochs = []
        prev = None
        for e in range(w.epochs):
            xe = torch.from_numpy(X[synth.epoch_permutation(w.n_train, w.seed_shuffle, e)]).to(dev)
            for k in range(per_epoch):
                if w.period > 0 and (k + 1) % w.period == 0:
                    layer.structural_update(count=False)
                layer.train_batch(xe[k * B:(k + 1) * B])
            sg, so = layer.get_state(), ora_states[e]
            werr = np.abs(sg["w"].astype(np.float64) - so["w"]) / np.maximum(1.0, np.abs(so["w"]))
            row = {"epoch": e + 1}
            for key in ("pi", "pj", "pij"):
                row[f"{key}_max_abs_err"] = float(np.max(np.abs(sg[key].astype(np.float64) - so[key])))
            row["w_max_scaled_err"] = float(werr.max())
            row["mask_entries_differing"] = int(np.sum(sg["mask"] != so["mask"]))
            if prev is not None:
                d = sg["pij"].astype(np.float64) - prev
                row["pij_unchanged_over_epoch"] = round(float(np.mean(d == 0.0)), 4)
                row["pij_decreased_over_epoch"] = round(float(np.mean(d < 0.0)), 4)
            prev = sg["pij"].astype(np.float64)
            epochs.append(row)
        y = torch.empty((len(Xt), L.n_out), device=dev, dtype=torch.float32)
        xt = torch.from_numpy(Xt).to(dev)
        for k in range(0, len(Xt), B):
            n = min(B, len(Xt) - k)
            layer.forward(xt[k:k + n], y[k:k + n])
        code_g = code(y.cpu().numpy())
        layer.close()
        formats[st] = {
            "epochs": epochs,
            "hidden_code_winner_agreement": round(float(np.mean(code_g == code_o)), 4),
            "hidden_code_ari_vs_oracle": round(float(np.mean(
                [adjusted_rand_index(code_g[:, h], code_o[:, h]) for h in range(L.out_hcu)])), 4),
            "distinct_winners_per_hcu": round(float(np.mean(
                [len(np.unique(code_g[:, h])) for h in range(L.out_hcu)])), 2),
        }
        say(f"{st}: {formats[st]['epochs'][-1]}")
    out = {
        "metric": "reduced-precision storage of Pij and w against the fp32 oracle (free runs on "
                  "the same batches): trace and weight errors, masks, stagnation, hidden code",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {L.in_hcu}x{L.in_mcu} -> {L.out_hcu}x{L.out_mcu}, "
                               f"{int(w.mask_frac * 100)}% receptive fields, alpha {w.alpha}, "
                               f"gain {w.gain}, k_B {w.bias_gain}, {w.epochs} epochs of "
                               f"{per_epoch} batches of {B}, plasticity every {w.period}; "
                               f"hidden code on {len(Xt)} held-out samples",
                   "storage_rounding": "round to nearest even of the fp32 result after every "
                                       "update (bf16: 7 stored mantissa bits; m10: 10)"},
        "oracle_distinct_winners_per_hcu": round(float(np.mean(
            [len(np.unique(code_o[:, h])) for h in range(L.out_hcu)])), 2),
        "oracle_wall_s": round(t_oracle, 1), "oracle_cores": oracle.threads(),
        "formats": formats,
        "pipeline": precision_pipeline(say),
    }
    print(json.dumps(out), flush=True)


def precision_pipeline(say):
    """The readout pipeline (3 hidden epochs + 1 readout epoch, its own learning settings) with
    Pij and w of both layers stored in fp32, bf16 or the 10-bit format: held-out accuracy, and
    the hidden code against the fp32 oracle's free run on the same batches (adjusted Rand index
    of the winner partitions, mean over hidden HCUs; free runs permute the MCUs)."""
    import torch
    import oracle
    from paper_2106_05373_amd import bcpnn, synth
    from paper_2106_05373_amd.pipeline import Network

    w = synth.WORKLOADS["mnist_pipeline"]
    L = w.layer
    B = w.batch
    dev = torch.device("cuda", 0)
    px, labels = synth.dataset(w)
    tx, tlabels = synth.dataset(w, split="test")
    X = synth.encode_pixels(px)
    Xt = torch.from_numpy(synth.encode_pixels(tx)).to(dev)
    onehot = synth.one_hot(labels, w.readout_mcu)
    mask = synth.random_mask(L.in_hcu, L.out_hcu, synth.active_count(L.in_hcu, w.mask_frac),
                             w.seed_mask)
    kw = dict(alpha=w.alpha, gain=w.gain, bias_gain=w.bias_gain, init_noise=w.init_noise,
              seed=w.seed_noise)
    per_epoch = (w.n_train + B - 1) // B
    n_code = 2000

    def code(y):
        return np.asarray(y).reshape(len(y), L.out_hcu, L.out_mcu).argmax(-1)

    ora = oracle.OracleLayer(oracle.make_params(L.in_hcu, L.in_mcu, L.out_hcu, L.out_mcu, **kw),
                             mask)
    for e in range(w.epochs):
        Xe = X[synth.epoch_permutation(w.n_train, w.seed_shuffle, e)]
        for k in range(per_epoch):
            if w.period > 0 and (k + 1) % w.period == 0:
                ora.structural_update()
            ora.train_batch(Xe[k * B:(k + 1) * B])
        say(f"pipeline oracle epoch {e + 1} of {w.epochs}")
    code_o = code(ora.forward(Xt[:n_code].cpu().numpy())[1])

    rows = {}
    for st in ("f32", "bf16", "m10"):
        cfg = bcpnn.default_config(L.in_hcu, L.in_mcu, L.out_hcu, L.out_mcu, B, storage=st,
                                   complement_pairs=int(w.complement_pairs), **kw)
        net = Network(cfg, mask, w.readout_mcu)
        for e in range(w.epochs + w.readout_epochs):
            perm = synth.epoch_permutation(w.n_train, w.seed_shuffle, e)
            xe = torch.from_numpy(X[perm]).to(dev)
            te = torch.from_numpy(onehot[perm]).to(dev)
            for k in range(per_epoch):
                if e < w.epochs:
                    if w.period > 0 and (k + 1) % w.period == 0:
                        net.hidden.structural_update(count=False)
                    net.train_hidden(xe[k * B:(k + 1) * B])
                else:
                    net.train_readout(xe[k * B:(k + 1) * B], te[k * B:(k + 1) * B])
        pred = net.predict(Xt).cpu().numpy()
        y = torch.empty((n_code, L.out_hcu * L.out_mcu), device=dev, dtype=torch.float32)
        for k in range(0, n_code, B):
            n = min(B, n_code - k)
            net.hidden.forward(Xt[k:k + n], y[k:k + n])
        code_g = code(y.cpu().numpy())
        rows[st] = {
            "heldout_accuracy": round(float(np.mean(pred == tlabels)), 4),
            "hidden_code_ari_vs_oracle": round(float(np.mean(
                [adjusted_rand_index(code_g[:, h], code_o[:, h]) for h in range(L.out_hcu)])), 4),
            "distinct_winners_per_hcu": round(float(np.mean(
                [len(np.unique(code_g[:, h])) for h in range(L.out_hcu)])), 1),
        }
        net.close()
        say(f"pipeline {st}: {rows[st]}")
    return {"config": f"{w.name}: alpha {w.alpha}, gain {w.gain}, k_B {w.bias_gain}, "
                      f"{w.epochs} hidden + {w.readout_epochs} readout epochs; "
                      f"{len(tlabels)} held-out samples (code on the first {n_code})",
            "oracle_distinct_winners_per_hcu": round(float(np.mean(
                [len(np.unique(code_o[:, h])) for h in range(L.out_hcu)])), 1),
            "storage": rows}


def run_inference_sweep():
    """Forward-pass (support + softmax) throughput of the MNIST-shaped layer by batch size: one
    launch per batch, timed over repeated launches between two synchronisations."""
    import torch
    from paper_2106_05373_amd import bcpnn, synth

    w = synth.WORKLOADS["mnist"]
    L = w.layer
    sizes = INFERENCE_BATCHES
    dev = torch.device("cuda", 0)
    px, _ = synth.dataset(w, split="test", n=max(sizes))
    X = torch.from_numpy(synth.encode_pixels(px)).to(dev)
    mask = synth.random_mask(L.in_hcu, L.out_hcu, synth.active_count(L.in_hcu, w.mask_frac),
                             w.seed_mask)
    stream = torch.cuda.Stream(device=dev)
    layer = bcpnn.Layer(bcpnn.default_config(L.in_hcu, L.in_mcu, L.out_hcu, L.out_mcu,
                                             max(sizes), alpha=w.alpha), mask, stream=stream)
    Y = torch.empty((max(sizes), L.out_hcu * L.out_mcu), device=dev, dtype=torch.float32)
    rows = []
    for B in sizes:
        reps = max(20, min(2000, 200000 // B))
        for _ in range(10):
            layer.forward(X[:B], Y[:B])
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            layer.forward(X[:B], Y[:B])
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / reps
        rows.append({"batch": B, "us_per_batch": round(dt * 1e6, 2),
                     "samples_per_s": round(B / dt, 1)})
    layer.close()
    return {"metric": "inference samples/s by batch size (support + per-HCU softmax)",
            "config": {"workload": f"mnist layer {L.in_hcu}x{L.in_mcu} -> "
                                   f"{L.out_hcu}x{L.out_mcu}, 10% receptive fields"},
            "data": "synthetic", "dtype": "f32 (fp64 accumulation)", "sweep": rows}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, mask, budget_s, n_batches=200):
    """The CPU oracle (as it stands) on this host's cores, on the MNIST-shaped schedule's first
    batches (the same images, shuffle and mask as the GPU run; structural updates before the
    100th and 200th).  All threads: the first n_batches batches, or as many as fit the budget.
    One thread: as many batches as fit half the budget, plus one structural update timed on the
    state they reach, amortised over its period."""
    import oracle
    from paper_2106_05373_amd import synth
    L = w.layer
    B = w.batch
    sched = schedule(w.n_train, B, w.period, n_batches)
    px, _ = synth.dataset(w)
    Xe = synth.encode_pixels(px)[synth.epoch_permutation(w.n_train, w.seed_shuffle, 0)]
    del px
    p = oracle.make_params(L.in_hcu, L.in_mcu, L.out_hcu, L.out_mcu, alpha=w.alpha, gain=w.gain,
                           bias_gain=w.bias_gain, init_noise=w.init_noise, seed=w.seed_noise)
    all_threads = oracle.threads()

    def run(budget):
        ora = oracle.OracleLayer(p, mask)
        done = samples = plastic = 0
        t0 = time.perf_counter()
        for (e, k, start, size, is_plastic) in sched:
            if is_plastic:
                ora.structural_update()
                plastic += 1
            ora.train_batch(Xe[start:start + size])
            done += 1
            samples += size
            if time.perf_counter() - t0 >= budget:
                break
        return ora, done, samples, plastic, time.perf_counter() - t0

    _, done, samples, plastic, el = run(budget_s)
    out = {"value": round(samples / el, 2), "unit": "samples/s", "cores": all_threads,
           "kind": "oracle", "cpu_model": cpu_model(),
           "sample": f"first {done} batches ({samples} samples, {plastic} structural updates, "
                     f"period {w.period}) of the MNIST-shaped schedule in {el:.1f} s, "
                     f"{all_threads} OpenMP threads"}
    oracle.set_threads(1)
    try:
        ora, done1, samples1, plastic1, el1 = run(budget_s / 2)
        t0 = time.perf_counter()
        ora.structural_update()
        su = time.perf_counter() - t0
    finally:
        oracle.set_threads(all_threads)
    per_batch = el1 / done1 + (su / w.period if plastic1 == 0 else 0.0)
    out["single_thread"] = {
        "value": round(B / per_batch, 2), "unit": "samples/s", "cores": 1,
        "sample": f"first {done1} batches ({samples1} samples) in {el1:.1f} s, plus one "
                  f"structural update timed on the state they reach ({su:.2f} s) amortised "
                  f"over its period of {w.period} batches" if plastic1 == 0 else
                  f"first {done1} batches ({samples1} samples, {plastic1} structural updates) "
                  f"in {el1:.1f} s"}
    return out


if __name__ == "__main__":
    main()
