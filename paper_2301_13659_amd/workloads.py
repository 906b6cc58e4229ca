"""Seeded synthetic inputs and layer parameters for the seven spiking-conv workloads.

This module only lays out workload parameters and draws random numbers: images,
spike-time maps, initial weights and labels.  It holds none of the method's
arithmetic (no filtering, coding, convolution, firing, inhibition or learning);
the GPU library and the CPU oracle each implement that on their own and both are
fed the arrays made here.

The paper (Spyker, arXiv 2301.13659) trains its networks on MNIST (§III-A) and
on recorded stimuli (§III-B).  Neither dataset is used: the generators below
only mimic the shapes, value ranges and sparsity of such inputs.

Seeds: image = 13659 + 100*cfg, weights of layer l (1-based) = 13659 + 100*cfg
+ 10*l, labels = 13659 + 100*cfg + 50, spike-time maps = 13659 + 100*cfg + 60 +
density index, rate-coding draws = 13659 + 100*cfg + 70.  Every draw uses numpy's PCG64 generator.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass, field

import numpy as np

NEVER = 255  # "did not fire" in a uint8 first-spike-time map
SEED_BASE = 13659
INF = math.inf


@dataclass(frozen=True)
class DogFilter:
    ksize: int
    sigma1: float
    sigma2: float


@dataclass(frozen=True)
class StdpConfig:
    """Mirror of the paper's STDPConfig(positive, negative, stabilize, lower, upper), §II-F.1."""
    a_causal: float
    a_anticausal: float
    lower: float = 0.0
    upper: float = 1.0
    stabilize: int = 1


@dataclass(frozen=True)
class ConvSpec:
    co: int
    ci: int
    k: int
    stride: int
    pad: int
    theta: float          # +inf = readout (no neuron fires; rank by final potential)
    k_win: int            # winners per sample (k-WTA count)
    radius: int           # inhibition radius (Chebyshev)
    stdp: bool            # this layer learns in the workload's step
    w_dtype: str = "f32"  # "f32" master on the conv, or "f16" operand
    w_mean: float = 0.8   # initial weights: normal(w_mean, w_std) clipped to [0, 1]
    w_std: float = 0.05

    @property
    def readout(self) -> bool:
        return math.isinf(self.theta)


@dataclass(frozen=True)
class PoolSpec:
    k: int
    stride: int
    pad: int


@dataclass(frozen=True)
class Workload:
    index: int                       # 1..7
    name: str
    batch: int
    T: int
    image_hw: tuple | None           # (H, W) of uint8 images, or None for spike input
    image_kind: str | None           # "uniform" | "strokes" | "noise_edges"
    dog: tuple = ()                  # DogFilter bank, channel order c*F + f
    min_value: float = 0.01          # values <= min_value never spike
    spikes_chw: tuple | None = None  # (C, H, W) of a direct spike-time input
    densities: tuple = ()            # final spike densities of the direct input
    stages: tuple = ()               # ("conv", ConvSpec) / ("pool", PoolSpec)
    stdp: tuple = (StdpConfig(0.004, -0.003),)
    rstdp_group: int = 0             # >0: R-STDP with class(o) = o // group
    n_classes: int = 0
    log_stds: tuple = ()             # LoG bank (two DoGs per deviation) instead of `dog`
    log_ksize: int = 0
    pre_threshold: float | None = None  # filter outputs <= this are zeroed before coding
    lr_schedule: tuple | None = None    # (every samples, factor, cap of the causal rate)
    coding: str = "rank"             # "rank": rank-order (time maps); "rate": rate coding (frames)
    binarize: float | None = None    # weights w < this -> 0 else 1 (a trained, quantized net)
    description: str = ""

    def with_batch(self, batch: int) -> "Workload":
        return dataclasses.replace(self, batch=batch, name=f"{self.name}-b{batch}")

    @property
    def convs(self) -> list:
        return [s for kind, s in self.stages if kind == "conv"]

    def input_chw(self) -> tuple:
        if self.spikes_chw is not None:
            return self.spikes_chw
        nf = 2 * len(self.log_stds) if self.log_stds else len(self.dog)
        return (nf, self.image_hw[0], self.image_hw[1])


def _dog_pair(k: int, s1: float) -> tuple:
    # on-centre (s1, 2*s1) then off-centre (2*s1, s1)
    return (DogFilter(k, s1, 2.0 * s1), DogFilter(k, 2.0 * s1, s1))


def _cfg2_stages(readout_learns: bool, k3: int) -> tuple:
    return (
        ("conv", ConvSpec(30, 6, 5, 1, 2, 15.0, 5, 3, not readout_learns)),
        ("pool", PoolSpec(2, 2, 0)),
        ("conv", ConvSpec(250, 30, 3, 1, 1, 10.0, 8, 1, not readout_learns)),
        ("pool", PoolSpec(3, 3, 1)),
        ("conv", ConvSpec(200, 250, 5, 1, 2, INF, k3, 0, readout_learns)),
    )


WORKLOADS = {
    1: Workload(
        index=1, name="cfg1-1layer-b8", batch=8, T=15, image_hw=(28, 28), image_kind="uniform",
        dog=_dog_pair(7, 1.0),
        stages=(("conv", ConvSpec(32, 2, 5, 1, 2, 15.0, 5, 2, True)),),
        description="one spiking conv layer, batch 8, 28x28 uniform uint8, DoG 2ch 7x7, T=15, "
                    "32 filters 5x5 pad 2, theta 15, k=5 r=2, STDP"),
    2: Workload(
        index=2, name="cfg2-3layer-b64", batch=64, T=15, image_hw=(28, 28), image_kind="strokes",
        dog=_dog_pair(3, 3 / 7) + _dog_pair(7, 1.0) + _dog_pair(13, 13 / 7),
        stages=_cfg2_stages(False, 1),
        description="three-layer conv SNN, batch 64, T=15, 28x28 strokes, DoG 6ch 3/7/13, "
                    "conv1 30x5x5 -> pool 2/2 -> conv2 250x3x3 -> pool 3/3 -> conv3 200x5x5 readout; "
                    "STDP on conv1 and conv2"),
    3: Workload(
        index=3, name="cfg3-rstdp-b256", batch=256, T=15, image_hw=(28, 28), image_kind="strokes",
        dog=_dog_pair(3, 3 / 7) + _dog_pair(7, 1.0) + _dog_pair(13, 13 / 7),
        stages=_cfg2_stages(True, 1),
        stdp=(StdpConfig(0.004, -0.003), StdpConfig(-0.0005, 0.004)),
        rstdp_group=20, n_classes=10,
        description="R-STDP readout on the three-layer stack, batch 256, 10 classes x 20 filters"),
    4: Workload(
        index=4, name="cfg4-large-b32", batch=32, T=30, image_hw=(160, 250), image_kind="noise_edges",
        dog=_dog_pair(7, 0.5) + _dog_pair(7, 1.0) + _dog_pair(7, 1.5),
        stages=(
            ("conv", ConvSpec(4, 6, 5, 1, 2, 15.0, 1, 0, True)),
            ("pool", PoolSpec(7, 6, 0)),
            ("conv", ConvSpec(20, 4, 17, 1, 0, 42.0, 1, 0, True)),
        ),
        description="160x250 images, batch 32, T=30, DoG 6ch 7x7, conv1 4x5x5 -> pool 7/6 -> "
                    "conv2 20x17x17; STDP on both"),
    5: Workload(
        index=5, name="cfg5-sweep-b128", batch=128, T=30, image_hw=None, image_kind=None,
        spikes_chw=(64, 64, 64), densities=(0.02, 0.05, 0.10),
        stages=(("conv", ConvSpec(128, 64, 3, 1, 1, 20.0, 16, 2, True, "f16")),),
        description="fp16 spiking conv 128x64x3x3 pad 1 on 64ch 64x64 spike frames, batch 128, "
                    "T=30, theta 20, k=16 r=2, STDP"),
    6: Workload(
        index=6, name="cfg6-demo-b64", batch=64, T=15, image_hw=(28, 28), image_kind="strokes",
        log_stds=(0.471, 1.099, 2.042), log_ksize=7, pre_threshold=0.01, min_value=0.0,
        stages=(
            ("conv", ConvSpec(100, 6, 5, 1, 2, 16.0, 5, 3, True, w_mean=0.5, w_std=0.02)),
            ("pool", PoolSpec(2, 2, 0)),
            ("conv", ConvSpec(200, 100, 3, 1, 1, 5.0, 8, 1, True, w_mean=0.5, w_std=0.02)),
            ("pool", PoolSpec(3, 3, 0)),
            ("gather", None),
        ),
        stdp=(StdpConfig(0.0004, -0.0003),),
        lr_schedule=(2000, 1.5, 0.15),
        description="the paper's example network: LoG bank (3 deviations, 7x7) -> threshold 0.01 -> "
                    "T=15 -> conv1 100x5x5 theta 16 k5 r3 -> pool 2 -> conv2 200x3x3 theta 5 k8 r1 -> "
                    "pool 3 -> gather; STDP with the learning-rate schedule, batch 64"),
    7: Workload(
        index=7, name="cfg7-rate-b64", batch=64, T=300, image_hw=(28, 28), image_kind="strokes",
        log_stds=(0.471, 1.099, 2.042), log_ksize=7, pre_threshold=0.01, min_value=0.0,
        coding="rate", binarize=0.5,
        stages=(
            ("conv", ConvSpec(25, 6, 5, 1, 2, 16.0, 0, 0, False, "f16", w_mean=0.5, w_std=0.02)),
            ("pool", PoolSpec(2, 2, 0)),
            ("conv", ConvSpec(50, 25, 3, 1, 1, 5.0, 0, 0, False, "f16", w_mean=0.5, w_std=0.02)),
            ("pool", PoolSpec(3, 3, 0)),
            ("gather", None),
        ),
        description="rate-coded inference of the example network with 25 and 50 maps: LoG bank -> "
                    "threshold 0.01 -> rate code T=300 -> conv1 25x5x5 theta 16 -> rate pool 2 -> "
                    "conv2 50x3x3 theta 5 -> rate pool 3 -> firing rates; binarized weights, batch 64"),
}


def get(index: int) -> Workload:
    return WORKLOADS[index]


# --------------------------------------------------------------------------- images

def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _segment_distance(py, px, y0, x0, y1, x1):
    dy, dx = y1 - y0, x1 - x0
    L2 = dy * dy + dx * dx
    if L2 == 0.0:
        return np.hypot(py - y0, px - x0)
    u = np.clip(((py - y0) * dy + (px - x0) * dx) / L2, 0.0, 1.0)
    return np.hypot(py - (y0 + u * dy), px - (x0 + u * dx))


def _strokes(rng, H, W):
    img = np.zeros((H, W), np.float64)
    py, px = np.mgrid[0:H, 0:W].astype(np.float64) + 0.5
    for _ in range(int(rng.integers(3, 7))):
        npts = int(rng.integers(2, 5))
        pts = rng.uniform(4.0, 24.0, size=(npts, 2)) * np.array([H / 28.0, W / 28.0])
        width = float(rng.integers(1, 4))
        inten = float(rng.integers(160, 256))
        for a, b in zip(pts[:-1], pts[1:]):
            d = _segment_distance(py, px, a[0], a[1], b[0], b[1])
            img = np.where(d <= max(width / 2.0, 0.5), np.maximum(img, inten), img)
    return img.astype(np.uint8)


def _noise_edges(rng, H, W):
    from scipy.ndimage import gaussian_filter  # data synthesis only
    base = gaussian_filter(rng.standard_normal((H, W)), sigma=6.0, mode="reflect")
    base = (base - base.min()) / max(base.max() - base.min(), 1e-12) * 160.0
    py, px = np.mgrid[0:H, 0:W].astype(np.float64) + 0.5
    for _ in range(int(rng.integers(4, 11))):
        ang = rng.uniform(0.0, math.pi)
        length = rng.uniform(20.0, 80.0)
        cy, cx = rng.uniform(0, H), rng.uniform(0, W)
        dy, dx = math.sin(ang) * length / 2, math.cos(ang) * length / 2
        d = _segment_distance(py, px, cy - dy, cx - dx, cy + dy, cx + dx)
        base = base + np.where(d <= 1.0, rng.uniform(60.0, 95.0), 0.0)
    return np.clip(np.rint(base), 0, 255).astype(np.uint8)


def make_images(wl: Workload) -> np.ndarray:
    """uint8 B x 1 x H x W."""
    H, W = wl.image_hw
    rng = _rng(SEED_BASE + 100 * wl.index)
    if wl.image_kind == "uniform":
        return rng.integers(0, 256, size=(wl.batch, 1, H, W), dtype=np.uint8)
    make = {"strokes": _strokes, "noise_edges": _noise_edges}[wl.image_kind]
    return np.stack([make(rng, H, W)[None] for _ in range(wl.batch)])


def make_spike_times(wl: Workload, density_index: int) -> np.ndarray:
    """uint8 B x C x H x W first-spike times for a direct spike input.

    Each neuron fires with probability rho (the final-frame density) at a time
    drawn uniformly from 0..T-1, so the density of frame t grows as rho*(t+1)/T.
    """
    rho = wl.densities[density_index]
    rng = _rng(SEED_BASE + 100 * wl.index + 60 + density_index)
    shape = (wl.batch,) + tuple(wl.spikes_chw)
    fires = rng.random(shape, dtype=np.float32) < rho
    t = rng.integers(0, wl.T, size=shape, dtype=np.uint8)
    return np.where(fires, t, np.uint8(NEVER)).astype(np.uint8)


def make_weights(wl: Workload, layer: int) -> np.ndarray:
    """float32 Co x Ci x K x K initial weights of conv layer `layer` (1-based).

    f32 layers: normal(w_mean, w_std) clipped to [0, 1] (0.8, 0.05 unless the layer
    says otherwise).  A workload with `binarize` draws those and keeps 0 / 1 (the
    weights of a trained network after quantization).  f16 layers: uniform(0.7, 0.9)
    rounded to half precision and held as float32 (the exact half values).
    """
    spec = wl.convs[layer - 1]
    rng = _rng(SEED_BASE + 100 * wl.index + 10 * layer)
    shape = (spec.co, spec.ci, spec.k, spec.k)
    if wl.binarize is not None:
        w = np.clip(rng.normal(spec.w_mean, spec.w_std, size=shape), 0.0, 1.0)
        return (w >= wl.binarize).astype(np.float32)
    if spec.w_dtype == "f16":
        return rng.uniform(0.7, 0.9, size=shape).astype(np.float16).astype(np.float32)
    return np.clip(rng.normal(spec.w_mean, spec.w_std, size=shape), 0.0, 1.0).astype(np.float32)


def make_labels(wl: Workload) -> np.ndarray:
    rng = _rng(SEED_BASE + 100 * wl.index + 50)
    return rng.integers(0, max(wl.n_classes, 1), size=wl.batch, dtype=np.int32)


# ---------------------------------------------------------------- small random cases

def random_times(rng: np.random.Generator, shape, T: int, density: float) -> np.ndarray:
    """uint8 time map with the given final density, times uniform over 0..T-1."""
    fires = rng.random(shape) < density
    t = rng.integers(0, T, size=shape)
    return np.where(fires, t, NEVER).astype(np.uint8)



def uniform_draws(seed: int, shape) -> np.ndarray:
    """float32 draws, uniform on [0, 1), for stochastic coding (rate coding
    takes them as an input)."""
    return _rng(seed).random(shape, dtype=np.float32)


def make_rate_draws(wl: Workload) -> np.ndarray:
    """float32 B x T x C x H x W uniform draws of a rate-coded workload's input."""
    return uniform_draws(SEED_BASE + 100 * wl.index + 70, (wl.batch, wl.T) + tuple(wl.input_chw()))
