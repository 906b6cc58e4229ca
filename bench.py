#!/usr/bin/env python3
"""Throughput of the spiking-conv hot path on one MI355X.

A step is one pass of the whole path over one batch of seeded synthetic input
(DoG filtering, rank-order coding, and per conv layer conv + fire, inhibition
+ k-WTA + STDP for learning layers, pooling between layers).  Default
workload: the three-layer network at batch 64, T = 15.

Prints ONE JSON line: whole-job samples/s, per-layer samples/s and synaptic
events/s, the roofline position of the dominant kernel (timed live with HIP
events on the stream it runs on) and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X datasheet peaks
PEAK_HBM_GBS = 8000.0
PEAK_F16_MFMA_TFLOPS = 2500.0

# HBM traffic of a conv kernel, from rocprofv3 FETCH_SIZE / WRITE_SIZE passes
# scaled by a plain copy of known size; valid only while the kernel source
# hashes to the value recorded with the counters.
PROFILES = os.path.join(ROOT, "profiles")
CONV_SOURCES = [os.path.join(ROOT, "paper_2301_13659_amd", "csrc", f)
                for f in ("spk_conv.hip", "spk_conv_pt.hip", "spk_conv_fast.hip", "spk_conv_mfma.hip")]


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
    ap.add_argument("--workload", type=int, default=2, help="1..7 (default: three-layer net)")
    ap.add_argument("--density", type=int, default=1, help="spike-density index of workload 5")
    ap.add_argument("--hbm-passes", action="store_true",
                    help="also time the standalone HBM passes of the first conv layer "
                         "(inhibition, fire over its dense potentials); on for workload 5")
    ap.add_argument("--sparse", action="store_true",
                    help="spike-input workloads: take the input as a spike list (sparse interface)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="CPU budget of the oracle baseline (0 disables it)")
    ap.add_argument("--no-breakdown", action="store_true")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="run one plain device copy of this size before the steps "
                         "(calibrates HBM byte counters under a profiler)")
    return ap.parse_args()


def measured_traffic(wl, layer):
    """HBM bytes per launch of a conv layer's kernel as recorded under profiles/,
    or None if absent or taken on a different kernel source."""
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
    if kept.dog is not None:
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


def hbm_passes(pipe, kept, torch, spk):
    """The streaming passes the HBM bar is judged on, on the first conv layer's
    outputs: pointwise inhibition alone (times + potentials read, inhibited map
    written) and the fire step over the layer's dense potentials (every step
    read, times + V_key written).  HIP events around each call, several
    repetitions, outside the timed steps."""
    wl = pipe.wl
    spec = wl.convs[0]
    t_in = kept.layer_in[0]
    tf, vk = kept.layer_out[0]
    layer = pipe.layers[0]
    w_op = layer.w16 if layer.w16 is not None else layer.w

    def timed(fn, reps):
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

    res = {}
    out = torch.empty_like(tf)
    ms = timed(lambda: spk.spk_inhibit(tf, vk, out=out), 10)
    nbytes = tf.numel() * 6
    res["inhibit"] = {"bytes": nbytes, "ms": ms, "GB/s": nbytes / (ms * 1e-3) / 1e9,
                      "frac": nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS}
    _, _, V = spk.spk_conv_fire(t_in, w_op, wl.T, spec.stride, spec.pad, spec.theta, potentials=True)
    ms = timed(lambda: spk.spk_fire(V, spec.theta), 5)
    nbytes = V.numel() * 4 + tf.numel() * 5
    res["fire_sweep"] = {"bytes": nbytes, "ms": ms, "GB/s": nbytes / (ms * 1e-3) / 1e9,
                         "frac": nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
                         "mode": "standalone fire over the dense-interface potentials"}
    del V
    torch.cuda.empty_cache()
    return res


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


def cpu_baseline_rate(wl, budget_s):
    """Rate-coded inference through the oracle, sample by sample; samples/s."""
    import oracle
    from paper_2301_13659_amd import workloads as wls

    imgs = wls.make_images(wl)
    draws = wls.make_rate_draws(wl)
    ws = [wls.make_weights(wl, i + 1) for i in range(len(wl.convs))]
    filters = oracle.log_filters(wl.log_stds, wl.log_ksize)
    done = 0
    t0 = time.perf_counter()
    while done < wl.batch and time.perf_counter() - t0 < budget_s:
        b = done
        x = oracle.dog_filter(imgs[b:b + 1], filters)
        if wl.pre_threshold is not None:
            x = oracle.threshold(x, wl.pre_threshold, 0.0)
        f = oracle.rate_code(x, draws[b:b + 1], wl.T, wl.min_value)
        c = None
        li = 0
        for kind, s in wl.stages:
            if kind == "gather":
                continue
            if kind == "pool":
                f, c = oracle.rate_pool(f, c, s.k, s.stride, s.pad)
                continue
            f, c = oracle.conv_if_rate(f, ws[li], s.stride, s.pad, s.theta)
            li += 1
        done += 1
    el = time.perf_counter() - t0
    return {"value": done / el, "unit": "samples/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} of the {wl.batch} samples of one batch, whole inference, "
                      f"{el:.1f} s single-threaded C"}


def cpu_baseline(wl, budget_s, sparse=False):
    """The oracle (plain C, one thread) on whole samples of the same workload until the
    budget is spent; samples/s."""
    import numpy as np

    import oracle
    from paper_2301_13659_amd import workloads as wls

    if wl.coding == "rate":
        return cpu_baseline_rate(wl, budget_s)

    imgs = wls.make_images(wl) if wl.image_hw is not None else None
    spikes = wls.make_spike_times(wl, 1) if wl.image_hw is None else None
    ws = [wls.make_weights(wl, i + 1) for i in range(len(wl.convs))]
    labels = wls.make_labels(wl)
    cfgs = [(c.a_causal, c.a_anticausal, c.lower, c.upper, c.stabilize) for c in wl.stdp]
    filters = [(f.ksize, f.sigma1, f.sigma2) for f in wl.dog]
    if wl.log_stds:
        filters = oracle.log_filters(wl.log_stds, wl.log_ksize)
    done = 0
    t0 = time.perf_counter()
    while done < wl.batch and time.perf_counter() - t0 < budget_s:
        b = done
        if imgs is not None:
            x = oracle.dog_filter(imgs[b:b + 1], filters)
            if wl.pre_threshold is not None:
                x = oracle.threshold(x, wl.pre_threshold, 0.0)
            t = oracle.latency_code(x, wl.T, wl.min_value)
        else:
            t = spikes[b:b + 1]
        li = 0
        for kind, s in wl.stages:
            if kind == "gather":
                oracle.gather(t, wl.T)
                continue
            if kind == "pool":
                t = oracle.pool(t, s.k, s.stride, s.pad)
                continue
            if sparse and li == 0:
                sp, off = oracle.times_to_spikes(t, wl.T)
                tf, vk = oracle.conv_fire_spikes(sp, off, t.shape[1:], ws[li], wl.T, s.stride, s.pad,
                                                 s.theta)
            else:
                tf, vk = oracle.conv_fire(t, ws[li], wl.T, s.stride, s.pad, s.theta)
            if s.stdp or s.readout:
                cand = tf if s.readout else oracle.inhibit(tf, vk)
                win, n = oracle.kwta(cand, vk, wl.T, s.k_win, s.radius, s.readout)
                if s.stdp:
                    wc = (oracle.rstdp_select(win, n, labels[b:b + 1], wl.rstdp_group)
                          if wl.rstdp_group else None)
                    ws[li] = oracle.stdp_update(ws[li], t, win, n, cfgs, s.stride, s.pad, winner_cfg=wc)
            t = tf
            li += 1
        done += 1
    el = time.perf_counter() - t0
    return {"value": done / el, "unit": "samples/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} of the {wl.batch} samples of one batch, whole step, "
                      f"{el:.1f} s single-threaded C"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); "
              "the path shards over the batch, see the design notes", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2301_13659_amd import spk
    from paper_2301_13659_amd import workloads as wls
    from paper_2301_13659_amd.pipeline import Pipeline, RatePipeline, conv_flops, conv_work

    dev = torch.device("cuda:0")
    wl = wls.get(args.workload)
    if wl.coding == "rate":
        pipe = RatePipeline(wl, dev)
    else:
        pipe = Pipeline(wl, dev, density_index=args.density, sparse=args.sparse)
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

    # warm-up; every step after the first also times the conv layers, to find
    # the dominant kernel (the one with the longest launch)
    warm = {}
    nwarm = max(args.warmup, 2)
    for i in range(nwarm):
        pipe.step(timers=warm if i > 0 else None)
    torch.cuda.synchronize()
    conv_ms = {li: sum(a.elapsed_time(b) for a, b in warm[f"conv{li + 1}"])
               for li in range(len(work))}
    dom = max(conv_ms, key=conv_ms.get)
    dom_name = f"conv{dom + 1}"

    timers = {}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        pipe.step(timers=timers, only={dom_name})
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    dom_ms = sum(a.elapsed_time(b) for a, b in timers[dom_name]) / len(timers[dom_name])

    ms_per_step = elapsed * 1e3 / args.steps
    value = wl.batch * args.steps / elapsed

    # per-stage breakdown (separate, untimed pass) and per-layer events
    per_layer = []
    stage_ms = {}
    if not args.no_breakdown:
        br = {}
        kept = None
        for i in range(max(3, min(args.steps, 10))):
            o = pipe.step(timers=br, keep=(i == 0))
            kept = kept or o
        torch.cuda.synchronize()
        stage_ms = {k: sum(a.elapsed_time(b) for a, b in v) / len(v) for k, v in br.items()}
        for li, spec in enumerate(wl.convs):
            n = li + 1
            ev = fanout_events(kept.layer_in[li], spec, torch)
            names = [f"conv{n}", f"wta{n}", f"select{n}", f"stdp{n}"]
            lay_ms = sum(stage_ms.get(k, 0.0) for k in names)
            c_ms = stage_ms[f"conv{n}"]
            per_layer.append({
                "layer": f"conv{n}", "ms": round(lay_ms, 4), "conv_ms": round(c_ms, 4),
                "samples_per_s": wl.batch / (lay_ms * 1e-3),
                "events": ev, "events_per_s": ev / (c_ms * 1e-3),
                "work_flop": work[li][0], "work": work[li][1],
                "tflops": work[li][0] / (c_ms * 1e-3) / 1e12,
                "mfma_frac": work[li][0] / (c_ms * 1e-3) / 1e12 / PEAK_F16_MFMA_TFLOPS,
                "dense_interface_tflops": flops_dense[li] / (c_ms * 1e-3) / 1e12})

    hbm = hbm_stages(wl, pipe, kept, stage_ms) if per_layer else {}
    passes = None
    if per_layer and wl.coding == "rank" and (args.hbm_passes or wl.index == 5):
        passes = hbm_passes(pipe, kept, torch, spk)

    achieved = work[dom][0] / (dom_ms * 1e-3) / 1e12
    sparse_dom = args.sparse and dom == 0
    roofline = {"bound": "mfma", "achieved": achieved, "peak": PEAK_F16_MFMA_TFLOPS,
                "unit": "TFLOP/s", "frac": achieved / PEAK_F16_MFMA_TFLOPS,
                "traffic": None if sparse_dom else measured_traffic(wl, dom + 1),
                "kernel": f"spk_conv_fire{'_sparse' if sparse_dom else ''} ({dom_name})",
                "kernel_ms": dom_ms,
                "work": f"{work[dom][1]} = {work[dom][0]:.4g} flop per launch"}
    if sparse_dom:
        # the event conv does not compute the dense product: its frac is the
        # dense-equivalent rate, above 1 where the skipped work outweighs
        roofline["effective"] = True
        if per_layer:
            roofline["events_per_s"] = per_layer[0]["events_per_s"]
    line = {
        "metric": "samples/sec and synaptic events/sec per layer; % fp16 MFMA / HBM peak",
        "value": value, "unit": "samples/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f16", "data": "synthetic",
        "config": {"workload": wl.name, "description": wl.description, "batch": wl.batch,
                   "T": wl.T, "parallelism": "single GPU"},
        "per_layer": per_layer, "stage_ms": stage_ms, "hbm_stages": hbm, "roofline": roofline,
        "library": spk.version(),
    }
    if passes is not None:
        line["hbm_passes"] = passes
    if args.sparse:
        line["config"]["interface"] = "sparse (spike-list input)"
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds, sparse=args.sparse)
    print(json.dumps(line))


if __name__ == "__main__":
    main()
