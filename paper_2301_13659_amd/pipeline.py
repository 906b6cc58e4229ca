"""One step of a workload's spiking network, chained through libspk.

A step is one pass of the hot path over one batch (the layer-wise training
of Spyker's listings, §IV): DoG filtering and rank-order coding of the images
(or a given spike-time input), then per conv layer: conv + fire, and for a
learning layer lateral inhibition + k-WTA + STDP (R-STDP for a readout
layer trained with labels), with pooling between layers.  The forward pass
between layers is not inhibited; learning uses the outputs computed with the
weights from before the step.  Readout layers (infinite threshold) pick
their winners by potential.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch

from . import spk
from . import workloads as wls


@dataclass
class LayerState:
    spec: wls.ConvSpec
    w: torch.Tensor                       # float32 master
    w16: torch.Tensor | None = None       # half operand (f16 layers)
    packed: torch.Tensor | None = None    # readout layers: the operand as packed B fragments

    @property
    def w_op(self) -> torch.Tensor:
        return self.w16 if self.w16 is not None else self.w

    def repack(self):
        """Rebuild the packed fragments after the weights changed."""
        if self.packed is not None:
            spk.spk_conv_pack_weights(self.w_op, out=self.packed)


@dataclass
class StepOutputs:
    dog: torch.Tensor | None = None
    times0: torch.Tensor | None = None
    layer_in: list = field(default_factory=list)     # input time map of each conv layer
    layer_out: list = field(default_factory=list)    # (t_f, v_key) of each conv layer
    winners: dict = field(default_factory=dict)      # conv index -> (winners, n_winners)
    winner_cfg: dict = field(default_factory=dict)   # conv index -> winner_cfg (R-STDP)
    pooled: list = field(default_factory=list)
    features: torch.Tensor | None = None             # gather of the last stage's spikes


class Pipeline:
    def __init__(self, wl: wls.Workload, device="cuda", density_index: int = 0, sparse: bool = False):
        """sparse: a spike-input workload takes its input as a spike list (the
        sparse interface of §II-B): the first conv layer runs
        spk_conv_fire_sparse on it, and the step rebuilds the input time map
        for STDP with spk_spikes_to_times."""
        self.wl = wl
        self.device = torch.device(device)
        self.sparse = sparse
        self.spike_list = None
        if wl.image_hw is not None:
            if sparse:
                raise ValueError("the sparse interface takes a spike input; this workload codes images")
            self.images = torch.from_numpy(wls.make_images(wl)).to(self.device)
            self.spike_input = None
        else:
            self.images = None
            self.spike_input = torch.from_numpy(wls.make_spike_times(wl, density_index)).to(self.device)
            if sparse:
                self.spike_list = spk.spk_times_to_spikes(self.spike_input, wl.T)
        self.layers = []
        for li, spec in enumerate(wl.convs, start=1):
            w = torch.from_numpy(wls.make_weights(wl, li)).to(self.device)
            w16 = w.to(torch.float16) if spec.w_dtype == "f16" else None
            layer = LayerState(spec, w, w16)
            if spec.readout and wl.coding == "rank":
                layer.packed = spk.spk_conv_pack_weights(layer.w_op)
            self.layers.append(layer)
        self.labels = torch.from_numpy(wls.make_labels(wl)).to(self.device) if wl.rstdp_group else None
        self.base_cfgs = [(c.a_causal, c.a_anticausal, c.lower, c.upper, c.stabilize) for c in wl.stdp]
        self.cfgs = list(self.base_cfgs)
        self.filters = [(f.ksize, f.sigma1, f.sigma2) for f in wl.dog]
        self.samples_seen = 0   # samples learnt from, for the learning-rate schedule

    def rate_factor(self) -> float:
        """Multiplier of the STDP rates for the next batch under the workload's
        schedule (§IV's example): x factor after every `every` samples, until
        the first configuration's causal rate reaches the cap."""
        if self.wl.lr_schedule is None:
            return 1.0
        every, factor, cap = self.wl.lr_schedule
        a0 = abs(self.base_cfgs[0][0])
        f = 1.0
        for _ in range(self.samples_seen // every):
            if a0 * f >= cap:
                break
            f = min(f * factor, cap / a0)
        return f

    def quantize(self, lower: float = 0.0, mid: float = 0.5, upper: float = 1.0):
        """Binarize the weights of the learning layers (§IV's example, after a
        layer's training)."""
        for layer in self.layers:
            if layer.spec.stdp:
                spk.spk_quantize(layer.w, lower, mid, upper, w_f16=layer.w16)
                layer.repack()

    def snapshot_weights(self):
        return [(l.w.clone(), None if l.w16 is None else l.w16.clone()) for l in self.layers]

    def restore_weights(self, snap):
        for l, (w, w16) in zip(self.layers, snap):
            l.w.copy_(w)
            if w16 is not None:
                l.w16.copy_(w16)
            l.repack()

    def step(self, keep: bool = False, learn: bool = True, timers: dict | None = None,
             only: set | None = None, gate=None, reps: int = 1) -> StepOutputs | None:
        """One pass over the batch.  timers, only, gate, reps: see _stage_timer."""
        wl = self.wl
        out = StepOutputs() if keep else None

        timed = _stage_timer(timers, only, gate, reps)

        if self.wl.lr_schedule is not None and learn:
            f = self.rate_factor()
            self.cfgs = [(a * f, b * f, lo, up, st) for a, b, lo, up, st in self.base_cfgs]
        if self.images is not None and not wl.log_stds and wl.pre_threshold is None:
            # filter bank and coding in one call; the filter outputs are kept when asked for
            x = None
            if keep:
                B, C, H, W = self.images.shape
                x = torch.empty((B, C * len(self.filters), H, W), dtype=torch.float32,
                                device=self.images.device)
            t = timed("code", lambda: spk.spk_dog_latency_code(self.images, self.filters, wl.T,
                                                               wl.min_value, dog_out=x))
            if keep:
                out.dog, out.times0 = x, t
        elif self.images is not None:
            if wl.log_stds:
                x = timed("dog", lambda: spk.spk_log_filter(self.images, wl.log_stds, wl.log_ksize))
            else:
                x = timed("dog", lambda: spk.spk_dog_filter(self.images, self.filters))
            if wl.pre_threshold is not None:
                timed("threshold", lambda: spk.spk_threshold(x, wl.pre_threshold, 0.0))
            t = timed("code", lambda: spk.spk_latency_code(x, wl.T, wl.min_value))
            if keep:
                out.dog, out.times0 = x, t
        elif self.spike_list is not None:
            t = None  # rebuilt from the list where a stage needs the time map
        else:
            t = self.spike_input
        li = 0
        pi = 0
        pending = None  # a pool whose conv runs next pools inside that conv's call
        for si, (kind, s) in enumerate(wl.stages):
            if kind == "gather":
                feats = timed("gather", lambda: spk.spk_gather(t, wl.T))
                if keep:
                    out.features = feats
                continue
            if kind == "pool":
                pi += 1
                if si + 1 < len(wl.stages) and wl.stages[si + 1][0] == "conv":
                    pending = s
                    continue
                t = timed(f"pool{pi}", lambda: spk.spk_pool(t, s.k, s.stride, s.pad))
                if keep:
                    out.pooled.append(t)
                continue
            layer = self.layers[li]
            w_op = layer.w_op
            n = li + 1
            if t is None:
                sp, off = self.spike_list
                tf, vk = timed(f"conv{n}", lambda: spk.spk_conv_fire_sparse(
                    sp, off, wl.input_chw(), w_op, wl.T, s.stride, s.pad, s.theta))
                if (s.stdp and learn) or keep:
                    t = timed("unpack", lambda: spk.spk_spikes_to_times(sp, off, wl.input_chw(), wl.T))
            elif pending is not None:
                pl = pending
                pending = None
                keep_in = keep or (s.stdp and learn)
                res = timed(f"conv{n}", lambda: spk.spk_pool_conv_fire(
                    t, (pl.k, pl.stride, pl.pad), w_op, wl.T, s.stride, s.pad, s.theta,
                    packed_w=layer.packed, keep_pooled=keep_in))
                if keep_in:
                    t, tf, vk = res
                    if keep:
                        out.pooled.append(t)
                else:
                    tf, vk = res
                    t = None
            else:
                tf, vk = timed(f"conv{n}", lambda: spk.spk_conv_fire(t, w_op, wl.T, s.stride, s.pad,
                                                                     s.theta))
            if keep:
                out.layer_in.append(t)
                out.layer_out.append((tf, vk))
            if s.stdp or s.readout:
                win, nw = timed(f"wta{n}", lambda: spk.spk_inhibit_winners(
                    tf, vk, wl.T, s.k_win, s.radius, pointwise=not s.readout, readout=s.readout))
                if keep:
                    out.winners[li] = (win, nw)
                if s.stdp and learn:
                    wc = None
                    if wl.rstdp_group:
                        wc = timed(f"select{n}", lambda: spk.spk_rstdp_select(
                            win, nw, self.labels, wl.rstdp_group))
                        if keep:
                            out.winner_cfg[li] = wc
                    timed(f"stdp{n}", lambda: spk.spk_stdp_update(
                        layer.w, t, win, nw, self.cfgs, s.stride, s.pad, winner_cfg=wc,
                        w_f16=layer.w16))
                    if layer.packed is not None:
                        timed(f"pack{n}", layer.repack)
            t = tf
            li += 1
        if learn:
            self.samples_seen += wl.batch
        return out



def _stage_timer(timers: dict | None, only: set | None, gate, reps: int):
    """Wraps each stage of a step.  With timers given, a stage (or only those
    named in `only`) is bracketed by a pair of torch.cuda.Event records on the
    current stream, appended to timers[name] as (start, end, reps).  gate
    (optional) is called before the start event: a GPU delay that lets the
    host enqueue the whole stage before the GPU reaches it, so the pair
    measures the stage's kernels and not the host's launch overhead.  reps > 1
    runs the stage that many times between the events (same inputs; a
    learning stage then updates its weights reps times)."""
    def timed(name, fn):
        if timers is None or (only is not None and name not in only):
            return fn()
        if gate is not None:
            gate()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        r = fn()
        for _ in range(reps - 1):
            r = fn()
        b.record()
        timers.setdefault(name, []).append((a, b, reps))
        return r
    return timed


def stage_ms(timers: dict) -> dict:
    """Average milliseconds per call of each timed stage."""
    return {k: sum(a.elapsed_time(b) for a, b, _ in v) / sum(r for _, _, r in v) for k, v in timers.items()}

def conv_flops(wl: wls.Workload) -> list:
    """Dense-interface work per conv layer and batch: 2*B*T*Ho*Wo*Co*Ci*Kh*Kw."""
    return [f for f, _ in conv_work(wl, dense=True)]


def conv_work(wl: wls.Workload, dense: bool = False) -> list:
    """Algorithmic flop per conv layer and batch, with a label.

    A firing layer needs every step's potential to find the first crossing:
    T dense convolutions of the cumulative frames, 2*B*T*Ho*Wo*Co*Ci*Kh*Kw.
    A readout layer (infinite threshold) needs only the last step's potential,
    one dense convolution of the final frame, 2*B*Ho*Wo*Co*Ci*Kh*Kw, unless
    `dense` asks for the per-step figure of every layer."""
    C, H, W = wl.input_chw()
    res = []
    for kind, s in wl.stages:
        if kind == "gather":
            continue
        if kind == "pool":
            H = (H + 2 * s.pad - s.k) // s.stride + 1
            W = (W + 2 * s.pad - s.k) // s.stride + 1
            continue
        Ho = (H + 2 * s.pad - s.k) // s.stride + 1
        Wo = (W + 2 * s.pad - s.k) // s.stride + 1
        one = 2 * wl.batch * Ho * Wo * s.co * s.ci * s.k * s.k
        if s.readout and not dense:
            res.append((one, "2*B*Ho*Wo*Co*Ci*Kh*Kw (readout: last step only)"))
        else:
            res.append((one * wl.T, "2*B*T*Ho*Wo*Co*Ci*Kh*Kw"))
        C, H, W = s.co, Ho, Wo
    return res


class RatePipeline:
    """Rate-coded inference of a workload (§II-D.1, §III-D): filter bank and
    threshold, rate coding with the workload's uniform draws, then per conv
    layer integrate-and-fire over the frames (reset after a spike), rate
    pooling between layers, and the firing rates of the last stage as
    features.  No learning: the weights are a trained network's (binarized)."""

    def __init__(self, wl: wls.Workload, device="cuda"):
        if wl.coding != "rate":
            raise ValueError("RatePipeline runs rate-coded workloads")
        self.wl = wl
        self.device = torch.device(device)
        self.images = torch.from_numpy(wls.make_images(wl)).to(self.device)
        self.draws = torch.from_numpy(wls.make_rate_draws(wl)).to(self.device)
        self.layers = []
        for li, spec in enumerate(wl.convs, start=1):
            w = torch.from_numpy(wls.make_weights(wl, li)).to(self.device)
            w16 = w.to(torch.float16) if spec.w_dtype == "f16" else None
            layer = LayerState(spec, w, w16)
            if spec.readout and wl.coding == "rank":
                layer.packed = spk.spk_conv_pack_weights(layer.w_op)
            self.layers.append(layer)
        self.filters = [(f.ksize, f.sigma1, f.sigma2) for f in wl.dog]

    def step(self, keep: bool = False, timers: dict | None = None, only: set | None = None, gate=None,
             reps: int = 1):
        wl = self.wl
        out = StepOutputs() if keep else None

        timed = _stage_timer(timers, only, gate, reps)

        if wl.log_stds:
            x = timed("dog", lambda: spk.spk_log_filter(self.images, wl.log_stds, wl.log_ksize))
        else:
            x = timed("dog", lambda: spk.spk_dog_filter(self.images, self.filters))
        if wl.pre_threshold is not None:
            timed("threshold", lambda: spk.spk_threshold(x, wl.pre_threshold, 0.0))
        f = timed("code", lambda: spk.spk_rate_code(x, self.draws, wl.T, wl.min_value))
        if keep:
            out.dog, out.times0 = x, f
        counts = None
        li = pi = 0
        for kind, s in wl.stages:
            if kind == "gather":
                feats = timed("gather", lambda: spk.spk_rate_features(counts, wl.T))
                if keep:
                    out.features = feats
                continue
            if kind == "pool":
                pi += 1
                f, counts = timed(f"pool{pi}", lambda: spk.spk_rate_pool(f, counts, s.k, s.stride, s.pad))
                if keep:
                    out.pooled.append((f, counts))
                continue
            layer = self.layers[li]
            w_op = layer.w16 if layer.w16 is not None else layer.w
            if keep:
                out.layer_in.append(f)
            f, counts = timed(f"conv{li + 1}", lambda: spk.spk_conv_if_rate(f, w_op, s.stride, s.pad,
                                                                            s.theta))
            if keep:
                out.layer_out.append((f, counts))
            li += 1
        return out
