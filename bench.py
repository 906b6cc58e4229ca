#!/usr/bin/env python3
"""Throughput of the spiking-conv hot path on one MI355X.

A step is one pass of the whole path over one batch of seeded synthetic input:
per conv layer conv + fire, and for a learning layer inhibition + k-WTA +
STDP, with DoG filtering, rank-order coding and pooling around them where the
workload has them.  Default workload: the fp16 spike-input layer (128 maps
3x3 over 64 x 64 x 64 spike inputs, batch 128, T = 30) at 5 % input density,
the largest single-GPU configuration; its 2 % and 10 % densities are reported
beside it.

Prints ONE JSON line: whole-job samples/s, per-layer samples/s and synaptic
events/s, per-stage kernel times, the roofline position of the dominant
kernel (timed live with HIP events on the stream it runs on), measured peaks,
and the CPU oracle timed on the host's cores (one thread, then all of them).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import subprocess
import sys
import time
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X datasheet peaks
PEAK_HBM_GBS = 8000.0
PEAK_F16_MFMA_TFLOPS = 2500.0

# worker threads of the CPU baseline: the host share of one GPU
MAX_CPU_THREADS = 16

# HBM traffic of a conv kernel, from rocprofv3 FETCH_SIZE / WRITE_SIZE passes
# scaled by a plain copy of known size; valid only while the kernel source
# hashes to the value recorded with the counters.
PROFILES = os.path.join(ROOT, "profiles")
CONV_SOURCES = [os.path.join(ROOT, "paper_2301_13659_amd", "csrc", f)
                for f in ("spk_conv.hip", "spk_conv_pt.hip", "spk_conv_fast.hip", "spk_conv_mfma.hip", "spk_internal.h")]


def conv_source_hash():
    h = hashlib.sha256()
    for f in CONV_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=5, help="1..7 (default: the spike-input layer)")
    ap.add_argument("--density", type=int, default=1,
                    help="input-density index of workload 5 (0: 2 %%, 1: 5 %%, 2: 10 %%)")
    ap.add_argument("--hbm-passes", action="store_true",
                    help="also time the standalone HBM passes of the first conv layer "
                         "(inhibition, fire over its dense potentials); on for workload 5")
    ap.add_argument("--sparse", action="store_true",
                    help="spike-input workloads: take the input as a spike list (sparse interface)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="CPU budget of each oracle baseline run (0 disables it)")
    ap.add_argument("--no-breakdown", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the density sweep, HBM passes and measured peaks")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="run one plain device copy of this size before the steps "
                         "(calibrates HBM byte counters under a profiler)")
    return ap.parse_args()


def measured_traffic(wl, layer):
    """HBM bytes per launch of a conv layer's kernels as recorded under
    profiles/, or None if absent or taken on a different kernel source."""
    path = os.path.join(PROFILES, f"traffic_conv{layer}_{wl.name}.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if ":" in line:
            k, v = line.split(":", 1)
            rec[k.strip()] = v.strip()
    if rec.get("kernel_source_sha256") != conv_source_hash():
        return None
    try:
        return float(rec["fetch_bytes_per_launch"]) + float(rec["write_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def dtype_label(wl):
    """The arithmetic the conv layers compute in."""
    kinds = {s.w_dtype for s in wl.convs}
    if kinds == {"f16"}:
        return "f16", "fp16 weights x binary spikes on fp16 MFMA (exact products), fp32 accumulation"
    return ("f32", "fp32 master weights carried as two fp16 halves (hi + lo) on fp16 MFMA, "
                   "fp32 accumulation")


def pipe_call(wl, li):
    """The entry point a pipeline step calls for conv layer li (0-based): the
    pooling in front of a layer runs inside its call."""
    convs = [i for i, (kind, _) in enumerate(wl.stages) if kind == "conv"]
    si = convs[li]
    pooled = si > 0 and wl.stages[si - 1][0] == "pool" and wl.coding == "rank"
    return "spk_pool_conv_fire" if pooled else "spk_conv_fire"


def hbm_stages(wl, pipe, kept, stage_ms):
    """Algorithmic HBM bytes of the memory-bound stages (each input read once,
    each output written once) and the rate they reach at the measured times."""
    res = {}

    def put(name, nbytes):
        if name in stage_ms:
            gbs = nbytes / (stage_ms[name] * 1e-3) / 1e9
            res[name] = {"bytes": int(nbytes), "GB/s": round(gbs, 1),
                         "frac": round(gbs / PEAK_HBM_GBS, 4)}

    rate = wl.coding == "rate"
    if kept.dog is not None and "dog" not in stage_ms and not rate:
        # filter bank and coding in one call: image read, times written
        put("code", pipe.images.numel() + kept.times0.numel())
    elif kept.dog is not None:
        put("dog", pipe.images.numel() + kept.dog.numel() * 4)
        put("threshold", kept.dog.numel() * 8)
        if rate:  # values, then one draw read and one frame byte written per step
            put("code", kept.dog.numel() * 4 + kept.times0.numel() * 5)
        else:
            put("code", kept.dog.numel() * 4 + kept.times0.numel())
    if rate:
        for i, (f, c) in enumerate(kept.pooled, start=1):
            src = kept.layer_out[i - 1]
            put(f"pool{i}", src[0].numel() + src[1].numel() * 4 + f.numel() + c.numel() * 4)
        if kept.features is not None:
            put("gather", kept.features.numel() * 8)
        return res
    if pipe.spike_list is not None:
        # time map written once, the list and its offsets read once
        nsp = int(pipe.spike_list[1][:, -1].sum().item())
        put("unpack", pipe.spike_input.numel() + 4 * nsp + pipe.spike_list[1].numel() * 4)
    pi = 0
    li = 0
    t = kept.times0 if kept.times0 is not None else pipe.spike_input
    for kind, s in wl.stages:
        if kind == "gather":
            put("gather", t.numel() * 5)
            continue
        if kind == "pool":
            out = kept.pooled[pi]
            pi += 1
            put(f"pool{pi}", t.numel() + out.numel())
            t = out
            continue
        tf, vk = kept.layer_out[li]
        n = li + 1
        if s.stdp or s.readout:
            # times + potentials read once, winner records written
            put(f"wta{n}", tf.numel() * 5 + wl.batch * s.k_win * 20)
        if s.stdp:
            w = pipe.layers[li].w
            patch = w[0].numel()
            # weights read and written, each winner's pre-time patch and record read
            put(f"stdp{n}", w.numel() * 8 + wl.batch * s.k_win * (patch + 20))
        t = tf
        li += 1
    return res


def timed_reps(torch, fn, reps):
    """Average ms of fn over reps back-to-back calls, HIP events on the current
    stream, after one untimed call."""
    fn()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    e = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        fn()
    e.record()
    torch.cuda.synchronize()
    return a.elapsed_time(e) / reps


def hbm_passes(pipe, kept, torch, spk):
    """The streaming passes the HBM bar is judged on, on the first conv layer's
    outputs: pointwise inhibition alone (times + potentials read, inhibited map
    written) and the fire step over the layer's dense potentials (every step
    read, times + V_key written).  HIP events around several repetitions,
    outside the timed steps."""
    wl = pipe.wl
    spec = wl.convs[0]
    t_in = kept.layer_in[0]
    tf, vk = kept.layer_out[0]
    layer = pipe.layers[0]
    w_op = layer.w16 if layer.w16 is not None else layer.w
    res = {}
    out = torch.empty_like(tf)
    ms = timed_reps(torch, lambda: spk.spk_inhibit(tf, vk, out=out), 10)
    nbytes = tf.numel() * 6
    res["inhibit"] = {"bytes": nbytes, "ms": ms, "GB/s": nbytes / (ms * 1e-3) / 1e9,
                      "frac": nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS}
    _, _, V = spk.spk_conv_fire(t_in, w_op, wl.T, spec.stride, spec.pad, spec.theta, potentials=True)
    ms = timed_reps(torch, lambda: spk.spk_fire(V, spec.theta), 5)
    nbytes = V.numel() * 4 + tf.numel() * 5
    res["fire_sweep"] = {"bytes": nbytes, "ms": ms, "GB/s": nbytes / (ms * 1e-3) / 1e9,
                         "frac": nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
                         "mode": "standalone fire over the dense-interface potentials"}
    del V
    torch.cuda.empty_cache()
    return res


def measured_peaks(torch, dev):
    """What this part reaches on plain library work, beside the datasheet:
    an fp16 GEMM (8192^3, torch.matmul -> hipBLASLt, MFMA-bound) and a
    device-to-device copy of 2 GiB (HBM-bound, bytes read + written)."""
    n = 8192
    a = torch.randn((n, n), device=dev, dtype=torch.float16)
    b = torch.randn((n, n), device=dev, dtype=torch.float16)
    c = torch.empty((n, n), device=dev, dtype=torch.float16)
    ms = timed_reps(torch, lambda: torch.matmul(a, b, out=c), 10)
    gemm = 2 * n ** 3 / (ms * 1e-3) / 1e12
    del a, b, c
    src = torch.empty(1 << 31, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    ms = timed_reps(torch, lambda: dst.copy_(src), 10)
    copy = 2 * src.numel() / (ms * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return {"f16_gemm_tflops": round(gemm, 1), "f16_gemm_frac_of_datasheet": round(gemm / PEAK_F16_MFMA_TFLOPS, 3),
            "copy_GBs": round(copy, 1), "copy_frac_of_datasheet": round(copy / PEAK_HBM_GBS, 3),
            "how": "torch.matmul fp16 8192^3 (hipBLASLt); tensor copy of 2 GiB, read + write bytes"}


def fanout_events(t_in, spec, torch):
    """Synaptic events of a conv layer: every input spike counted once times its fan-out
    (number of output neurons whose window holds it).  t_in is a time map
    B x C x H x W, or rate-coded frames B x T x C x H x W (every spike of every step)."""
    import torch.nn.functional as F
    if t_in.dim() == 5:
        fired = t_in.to(torch.float64).sum(dim=(0, 1, 2))
        t_in = t_in[:, 0]
    else:
        fired = (t_in != 255).to(torch.float64).sum(dim=(0, 1))
    B, C, H, W = t_in.shape
    Ho = (H + 2 * spec.pad - spec.k) // spec.stride + 1
    Wo = (W + 2 * spec.pad - spec.k) // spec.stride + 1
    cover = F.conv_transpose2d(torch.ones((1, 1, Ho, Wo), device=t_in.device),
                               torch.ones((1, 1, spec.k, spec.k), device=t_in.device),
                               stride=spec.stride, padding=spec.pad)
    cover = F.pad(cover, (0, W - cover.shape[-1], 0, H - cover.shape[-2]))[0, 0]
    return float((fired * cover.to(torch.float64)).sum().item()) * spec.co


# ------------------------------------------------------------- CPU baseline

def host_info():
    model = platform.processor() or "unknown"
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                model = line.split(":", 1)[1].strip()
                break
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        nproc = int(subprocess.run(["nproc"], capture_output=True, text=True, timeout=10).stdout)
    except (OSError, subprocess.SubprocessError, ValueError):
        nproc = os.cpu_count() or 1
    return nproc, model


class OracleStep:
    """The oracle running the workload's step on a subset of the batch: each
    sample's forward pass (filtering, coding, every conv layer in the
    oracle's event form, pooling, inhibition and k-WTA of learning layers) is
    independent, so chunks of samples run on threads (the C calls release the
    GIL); then each learning layer's batch STDP over those samples, from the
    weights before the step."""

    def __init__(self, wl, density_index, sparse):
        import oracle
        from paper_2301_13659_amd import workloads as wls
        self.o, self.wl = oracle, wl
        self.imgs = wls.make_images(wl) if wl.image_hw is not None else None
        self.spikes = wls.make_spike_times(wl, density_index) if wl.image_hw is None else None
        self.draws = wls.make_rate_draws(wl) if wl.coding == "rate" else None
        self.ws = [wls.make_weights(wl, i + 1) for i in range(len(wl.convs))]
        self.labels = wls.make_labels(wl)
        self.cfgs = [(c.a_causal, c.a_anticausal, c.lower, c.upper, c.stabilize) for c in wl.stdp]
        self.filters = [(f.ksize, f.sigma1, f.sigma2) for f in wl.dog]
        if wl.log_stds:
            self.filters = oracle.log_filters(wl.log_stds, wl.log_ksize)

    def forward(self, lo, hi):
        o, wl = self.o, self.wl
        rec = []  # per learning layer: (layer index, input times, winners, counts)
        if self.imgs is not None:
            x = o.dog_filter(self.imgs[lo:hi], self.filters)
            if wl.pre_threshold is not None:
                x = o.threshold(x, wl.pre_threshold, 0.0)
            if wl.coding == "rate":
                return self._rate_forward(x, lo, hi)
            t = o.latency_code(x, wl.T, wl.min_value)
        else:
            t = self.spikes[lo:hi]
        li = 0
        for kind, s in wl.stages:
            if kind == "gather":
                o.gather(t, wl.T)
                continue
            if kind == "pool":
                t = o.pool(t, s.k, s.stride, s.pad)
                continue
            sp, off = o.times_to_spikes(t, wl.T)
            tf, vk = o.conv_fire_spikes(sp, off, t.shape[1:], self.ws[li], wl.T, s.stride, s.pad, s.theta)
            if s.stdp or s.readout:
                cand = tf if s.readout else o.inhibit(tf, vk)
                win, n = o.kwta(cand, vk, wl.T, s.k_win, s.radius, s.readout)
                if s.stdp:
                    rec.append((li, t, win, n))
            t = tf
            li += 1
        return rec

    def _rate_forward(self, x, lo, hi):
        o, wl = self.o, self.wl
        f = o.rate_code(x, self.draws[lo:hi], wl.T, wl.min_value)
        c = None
        li = 0
        for kind, s in wl.stages:
            if kind == "gather":
                continue
            if kind == "pool":
                f, c = o.rate_pool(f, c, s.k, s.stride, s.pad)
                continue
            f, c = o.conv_if_rate(f, self.ws[li], s.stride, s.pad, s.theta)
            li += 1
        return []

    def run(self, n_samples, threads):
        import numpy as np
        chunks = [c for c in np.array_split(np.arange(n_samples), threads) if len(c)]
        with ThreadPoolExecutor(len(chunks)) as ex:
            recs = list(ex.map(lambda c: self.forward(int(c[0]), int(c[-1]) + 1), chunks))
        for per_layer in zip(*recs) if recs and recs[0] else []:
            li = per_layer[0][0]
            s = self.wl.convs[li]
            t = np.concatenate([r[1] for r in per_layer])
            win = np.concatenate([r[2] for r in per_layer])
            n = np.concatenate([r[3] for r in per_layer])
            wc = (self.o.rstdp_select(win, n, self.labels[:n_samples], self.wl.rstdp_group)
                  if self.wl.rstdp_group else None)
            self.o.stdp_update(self.ws[li], t, win, n, self.cfgs, s.stride, s.pad, winner_cfg=wc)


def cpu_baseline(wl, budget_s, density_index, sparse):
    """The oracle on the host's cores, twice: one thread, then all the cores
    this GPU's share allows (at most 16).  Each run covers as many samples of
    one batch as fit the budget (estimated from a first timed sample)."""
    nproc, model = host_info()
    threads = max(1, min(MAX_CPU_THREADS, nproc))
    step = OracleStep(wl, density_index, sparse)
    t0 = time.perf_counter()
    step.run(1, 1)
    per_sample = time.perf_counter() - t0
    n1 = max(1, min(wl.batch, int(budget_s / per_sample)))
    t0 = time.perf_counter()
    step.run(n1, 1)
    el1 = time.perf_counter() - t0
    nall = max(threads, min(wl.batch, int(budget_s * threads / per_sample)))
    nall = min(nall, wl.batch)
    t0 = time.perf_counter()
    step.run(nall, threads)
    elall = time.perf_counter() - t0
    conv_form = "event form (arrivals scattered, running sum over steps)" if wl.coding == "rank" else \
        "per-step integrate-and-fire"
    return {
        "value": nall / elall, "unit": "samples/s", "cores": threads, "kind": "oracle",
        "sample": f"{nall} of the {wl.batch} samples of one batch, whole step (forward on "
                  f"{threads} threads over samples, then batch STDP), {elall:.1f} s; plain C, "
                  f"conv in the {conv_form}",
        "single_thread": {"value": n1 / el1, "unit": "samples/s", "cores": 1,
                          "sample": f"{n1} samples, {el1:.1f} s"},
        "host": {"nproc": nproc, "model": model},
    }


# -------------------------------------------------------------------- main

def time_steps(torch, pipe, steps, dom_name):
    """Time `steps` whole steps; HIP events around the dominant conv call."""
    timers = {}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        pipe.step(timers=timers, only={dom_name})
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ev = timers[dom_name]
    dom_ms = sum(a.elapsed_time(b) for a, b, _ in ev) / sum(r for _, _, r in ev)
    return elapsed, dom_ms


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); "
              "the path shards over the batch, as the design notes describe", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2301_13659_amd import spk
    from paper_2301_13659_amd import workloads as wls
    from paper_2301_13659_amd.pipeline import Pipeline, RatePipeline, conv_flops, conv_work, stage_ms

    dev = torch.device("cuda:0")
    wl = wls.get(args.workload)
    spike_input = wl.image_hw is None

    def make_pipe(density_index):
        if wl.coding == "rate":
            return RatePipeline(wl, dev)
        return Pipeline(wl, dev, density_index=density_index, sparse=args.sparse)

    pipe = make_pipe(args.density)
    work = conv_work(wl)
    flops_dense = conv_flops(wl)

    if args.copy_mib > 0:
        # one elementwise kernel that reads and writes copy_mib MiB each
        n = (args.copy_mib << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    # a GPU delay before each timed stage of the breakdown, long enough for
    # the host to enqueue the stage's launches (about 1 ms at the shader clock)
    def gate():
        torch.cuda._sleep(2_000_000)

    # warm-up; the last warm-up step times every conv layer (gated) to find
    # the dominant kernel, the one with the longest launch
    nwarm = max(args.warmup, 2)
    for _ in range(nwarm - 1):
        pipe.step()
    warm = {}
    conv_names = {f"conv{li + 1}" for li in range(len(work))}
    pipe.step(timers=warm, only=conv_names, gate=gate)
    torch.cuda.synchronize()
    conv_ms = stage_ms(warm)
    dom = max(range(len(work)), key=lambda li: conv_ms[f"conv{li + 1}"])
    dom_name = f"conv{dom + 1}"

    elapsed, dom_ms = time_steps(torch, pipe, args.steps, dom_name)
    ms_per_step = elapsed * 1e3 / args.steps
    value = wl.batch * args.steps / elapsed

    # per-stage kernel times: a separate pass in which every stage runs 5
    # times back to back behind a GPU delay (so host launch overhead is not
    # counted), weights restored afterwards; per-layer events
    per_layer = []
    st_ms = {}
    kept = None
    if not args.no_breakdown:
        snap = pipe.snapshot_weights() if hasattr(pipe, "snapshot_weights") else None
        kept = pipe.step(keep=True)
        br = {}
        for _ in range(3):
            pipe.step(timers=br, gate=gate, reps=5)
        torch.cuda.synchronize()
        if snap is not None:
            pipe.restore_weights(snap)
        st_ms = stage_ms(br)
        for li, spec in enumerate(wl.convs):
            n = li + 1
            ev = fanout_events(kept.layer_in[li], spec, torch)
            names = [f"conv{n}", f"wta{n}", f"select{n}", f"stdp{n}", f"pack{n}"]
            lay_ms = sum(st_ms.get(k, 0.0) for k in names)
            c_ms = st_ms[f"conv{n}"]
            per_layer.append({
                "layer": f"conv{n}", "ms": round(lay_ms, 4), "conv_ms": round(c_ms, 4),
                "samples_per_s": wl.batch / (lay_ms * 1e-3),
                "events": ev, "events_per_s": ev / (c_ms * 1e-3),
                "work_flop": work[li][0], "work": work[li][1],
                "tflops": work[li][0] / (c_ms * 1e-3) / 1e12,
                "mfma_frac": work[li][0] / (c_ms * 1e-3) / 1e12 / PEAK_F16_MFMA_TFLOPS,
                "dense_interface_tflops": flops_dense[li] / (c_ms * 1e-3) / 1e12})

    hbm = hbm_stages(wl, pipe, kept, st_ms) if per_layer else {}

    achieved = work[dom][0] / (dom_ms * 1e-3) / 1e12
    sparse_dom = args.sparse and dom == 0
    roofline = {"bound": "mfma", "achieved": achieved, "peak": PEAK_F16_MFMA_TFLOPS,
                "unit": "TFLOP/s", "frac": achieved / PEAK_F16_MFMA_TFLOPS,
                "traffic": None if sparse_dom else measured_traffic(wl, dom + 1),
                "kernel": (f"spk_conv_fire_sparse ({dom_name})" if sparse_dom else
                           f"{pipe_call(wl, dom)} ({dom_name})"),
                "kernel_ms": dom_ms,
                "work": f"{work[dom][1]} = {work[dom][0]:.4g} flop per launch"}
    if sparse_dom:
        # the event conv does not compute the dense product: its frac is the
        # dense-equivalent rate, above 1 where the skipped work outweighs
        roofline["effective"] = True
        if per_layer:
            roofline["events_per_s"] = per_layer[0]["events_per_s"]
    dtype, arith = dtype_label(wl)
    config = {"workload": wl.name, "description": wl.description, "batch": wl.batch,
              "T": wl.T, "parallelism": "single GPU"}
    if spike_input:
        config["input_density"] = wl.densities[args.density]
    if args.sparse:
        config["interface"] = "sparse (spike-list input)"
    line = {
        "metric": "samples/sec and synaptic events/sec per layer; % fp16 MFMA / HBM peak",
        "value": value, "unit": "samples/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": dtype, "arith": arith, "data": "synthetic",
        "config": config, "per_layer": per_layer, "stage_ms": st_ms, "hbm_stages": hbm,
        "roofline": roofline, "library": spk.version(),
    }

    if not args.no_extras:
        if spike_input and wl.coding == "rank":
            # the other input densities of the sweep, whole steps timed the same way
            sweep = {}
            for di, rho in enumerate(wl.densities):
                if di == args.density:
                    continue
                p2 = make_pipe(di)
                for _ in range(2):
                    p2.step()
                n2 = max(5, args.steps // 2)
                el2, dms2 = time_steps(torch, p2, n2, dom_name)
                sweep[f"{rho:g}"] = {"samples_per_s": wl.batch * n2 / el2, "ms_per_step": el2 * 1e3 / n2,
                                     "conv_ms": dms2,
                                     "mfma_frac": work[dom][0] / (dms2 * 1e-3) / 1e12 / PEAK_F16_MFMA_TFLOPS}
                del p2
            torch.cuda.empty_cache()
            line["density_sweep"] = sweep
        if per_layer and wl.coding == "rank" and (args.hbm_passes or wl.index == 5):
            line["hbm_passes"] = hbm_passes(pipe, kept, torch, spk)
        line["measured_peaks"] = measured_peaks(torch, dev)
        mp = line["measured_peaks"]
        roofline["frac_of_measured_gemm"] = achieved / mp["f16_gemm_tflops"]

    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds, args.density, args.sparse)
    print(json.dumps(line))


if __name__ == "__main__":
    main()
