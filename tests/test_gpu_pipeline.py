"""End-to-end parity of one workload step (the step bench.py times), stage by stage.

Every stage of the GPU step is checked against the oracle run on the inputs
that stage received on the GPU (stage isolation), so a neuron that sits on its
threshold cannot cascade into later stages.  Every output is compared in full,
at reduced batches and at each workload's real batch; the outputs the binding
allocates start filled with sentinels (see conftest.py), so one a kernel leaves
unwritten fails.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from parity import (NEVER, V_ABS, V_REL, W_ABS, check_fire, check_potentials,
                    excused_from_potentials, gpu, np_, winners_list)
from paper_2301_13659_amd import spk, workloads
from paper_2301_13659_amd.pipeline import Pipeline

pytestmark = pytest.mark.gpu


def _oracle_conv_spikes(t_in, w, spec, T):
    """The oracle's event form of the layer (every arrival's weights scattered
    into the change of potential at its step, then the running sum over the
    steps and the first crossing), run over every sample.  Samples are
    independent: chunks of them run on threads (the C calls release the GIL)."""
    B = t_in.shape[0]
    nthreads = max(1, min(16, os.cpu_count() or 1, B))
    chunks = [c for c in np.array_split(np.arange(B), nthreads) if len(c)]

    def run(idx):
        x = np.ascontiguousarray(t_in[idx[0]:idx[-1] + 1])
        sp, off = oracle.times_to_spikes(x, T)
        return oracle.conv_fire_spikes(sp, off, x.shape[1:], w, T, spec.stride, spec.pad, spec.theta)

    with ThreadPoolExecutor(len(chunks)) as ex:
        res = list(ex.map(run, chunks))
    return np.concatenate([r[0] for r in res]), np.concatenate([r[1] for r in res])


def _check_conv_full(t_in, w, spec, T, g_tf, g_vk):
    """Every output neuron of the layer against the oracle.  A neuron whose
    time or V_key disagrees is looked at on its own: it is excused only if its
    oracle potential comes within 1e-4 |theta| of theta at some step.
    Half-weight layers (multiples of 2^-11 summing below 2^13: exact in any
    order) must match bit for bit.  Returns the number of excused neurons."""
    assert np.all((g_tf < T) | (g_tf == NEVER)), "spike times outside [0, T) that are not NEVER"
    assert np.all(np.isfinite(g_vk)), "non-finite V_key (an output left unwritten?)"
    o_tf, o_vk = _oracle_conv_spikes(t_in, w, spec, T)
    if spec.w_dtype == "f16":
        np.testing.assert_array_equal(g_tf, o_tf)
        np.testing.assert_array_equal(g_vk, o_vk)
        return 0
    if not np.isfinite(spec.theta):
        assert np.all(g_tf == NEVER)
        check_potentials(g_vk, o_vk, "readout v_key")
        return 0
    vbad = ~(np.abs(g_vk.astype(np.float64) - o_vk) <= V_REL * np.abs(o_vk.astype(np.float64)) + V_ABS)
    mism = np.argwhere((g_tf != o_tf) | vbad)
    assert len(mism) <= max(50, g_tf.size // 1000), f"{len(mism)} of {g_tf.size} neurons disagree"
    for (b, o, y, x) in mism:
        V = oracle.conv_neuron(t_in, w, T, spec.stride, spec.pad, int(b), int(o), int(y), int(x))
        excused = np.any(np.abs(V - spec.theta) <= 1e-4 * abs(spec.theta))
        assert excused, ((b, o, y, x), int(g_tf[b, o, y, x]), int(o_tf[b, o, y, x]),
                         float(g_vk[b, o, y, x]), float(o_vk[b, o, y, x]))
    return len(mism)


def _run_and_check(wl, dense_oracle: bool, density_index: int = 1, samples_seen: int = 0):
    """One step of the workload, every stage against the oracle on the inputs
    that stage received.  dense_oracle: the conv oracle also computes every
    potential of every step (small batches); otherwise its event form checks
    every output neuron."""
    dev = gpu()
    pipe = Pipeline(wl, dev, density_index=density_index)
    pipe.samples_seen = samples_seen
    w_before = [np_(l.w16.float() if l.w16 is not None else l.w).copy() for l in pipe.layers]
    master_before = [np_(l.w).copy() for l in pipe.layers]
    out = pipe.step(keep=True)
    torch.cuda.synchronize()
    filters = [(f.ksize, f.sigma1, f.sigma2) for f in wl.dog]
    if wl.log_stds:
        filters = oracle.log_filters(wl.log_stds, wl.log_ksize)
    if pipe.images is not None:
        img = np_(pipe.images)
        g_dog = np_(out.dog)
        o_dog = oracle.dog_filter(img, filters)
        if wl.pre_threshold is not None:
            o_dog = oracle.threshold(o_dog, wl.pre_threshold, 0.0)
        np.testing.assert_array_equal(g_dog.view(np.uint32), o_dog.view(np.uint32))
        np.testing.assert_array_equal(np_(out.times0), oracle.latency_code(g_dog, wl.T, wl.min_value))
    excused_total = 0
    pool_i = 0
    li = 0
    for kind, s in wl.stages:
        if kind == "gather":
            last = np_(out.pooled[pool_i - 1]) if wl.stages[-2][0] == "pool" else np_(out.layer_out[li - 1][0])
            np.testing.assert_array_equal(np_(out.features), oracle.gather(last, wl.T))
            continue
        if kind == "pool":
            src = np_(out.layer_out[li - 1][0])
            np.testing.assert_array_equal(np_(out.pooled[pool_i]), oracle.pool(src, s.k, s.stride, s.pad))
            pool_i += 1
            continue
        t_in = np_(out.layer_in[li])
        g_tf, g_vk = (np_(a) for a in out.layer_out[li])
        if dense_oracle:
            o_tf, o_vk, o_V = oracle.conv_fire(t_in, w_before[li], wl.T, s.stride, s.pad, s.theta,
                                               potentials=True)
            excused_total += check_fire(g_tf, g_vk, o_tf, o_vk, excused_from_potentials(o_V, s.theta))
        else:
            excused_total += _check_conv_full(t_in, w_before[li], s, wl.T, g_tf, g_vk)
        if li in out.winners:
            win, n = out.winners[li]
            g_win, g_n = spk.winners_numpy(win), np_(n)
            cand = g_tf if s.readout else oracle.inhibit(g_tf, g_vk)
            o_win, o_n = oracle.kwta(cand, g_vk, wl.T, s.k_win, s.radius, s.readout)
            np.testing.assert_array_equal(g_n, o_n)
            assert winners_list(g_win, g_n) == winners_list(o_win, o_n)
            if s.stdp:
                wc = None
                if wl.rstdp_group:
                    wc = np_(out.winner_cfg[li])
                    np.testing.assert_array_equal(
                        wc, oracle.rstdp_select(g_win, g_n, np_(pipe.labels), wl.rstdp_group))
                f = oracle.lr_factor(samples_seen, wl.stdp[0].a_causal, *wl.lr_schedule) if wl.lr_schedule else 1.0
                cfgs = [(c.a_causal * f, c.a_anticausal * f, c.lower, c.upper, c.stabilize) for c in wl.stdp]
                ref = oracle.stdp_update(master_before[li], t_in, g_win, g_n, cfgs, s.stride, s.pad,
                                         winner_cfg=wc)
                got = np_(pipe.layers[li].w)
                np.testing.assert_allclose(got, ref, rtol=0, atol=W_ABS)
                if pipe.layers[li].w16 is not None:
                    np.testing.assert_array_equal(np_(pipe.layers[li].w16), got.astype(np.float16))
        li += 1
    return excused_total


@pytest.mark.parametrize("cfg,batch", [(1, 8), (2, 2), (3, 3), (4, 1)])
def test_workload_step_reduced_batch(cfg, batch):
    wl = workloads.get(cfg).with_batch(batch)
    excused = _run_and_check(wl, dense_oracle=True)
    assert excused <= 5


@pytest.mark.parametrize("samples_seen", [0, 4000, 10 ** 6])
def test_demo_step_reduced_batch(samples_seen):
    """The paper's example network: LoG bank, threshold, two learning layers
    with the learning-rate schedule at three points of training, gather."""
    wl = workloads.get(6).with_batch(2)
    _run_and_check(wl, dense_oracle=True, samples_seen=samples_seen)


def test_demo_quantize_after_training():
    dev = gpu()
    pipe = Pipeline(workloads.get(6).with_batch(4), dev)
    pipe.step()
    before = [np_(l.w).copy() for l in pipe.layers]
    pipe.quantize()
    for b, l in zip(before, pipe.layers):
        np.testing.assert_array_equal(np_(l.w), oracle.quantize(b, 0.0, 0.5, 1.0))


@pytest.mark.parametrize("density_index", [0, 1, 2])
def test_cfg5_step_reduced_batch(density_index):
    wl = workloads.get(5).with_batch(1)
    assert _run_and_check(wl, dense_oracle=False, density_index=density_index) == 0


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 6])
def test_workload_step_full_size(cfg):
    """Every workload at its real batch, in the launch configuration bench.py
    times: every output neuron of every conv layer against the oracle."""
    wl = workloads.get(cfg)
    excused = _run_and_check(wl, dense_oracle=(cfg == 1), density_index=1)
    assert excused <= 200


@pytest.mark.parametrize("density_index", [0, 1, 2])
def test_cfg5_step_full_size(density_index):
    """The spike-input layer at B = 128 and each input density: its half
    weights are multiples of 2^-11 with sums below 2^13, exact in any order,
    so every neuron must agree with the oracle bit for bit."""
    wl = workloads.get(5)
    assert _run_and_check(wl, dense_oracle=False, density_index=density_index) == 0


def test_step_is_deterministic():
    dev = gpu()
    wl = workloads.get(2).with_batch(4)
    outs = []
    for _ in range(2):
        pipe = Pipeline(wl, dev)
        o = pipe.step(keep=True)
        torch.cuda.synchronize()
        outs.append((np_(o.times0), [np_(a[0]) for a in o.layer_out], [np_(a[1]) for a in o.layer_out],
                     [np_(l.w) for l in pipe.layers]))
    a, b = outs
    # the outputs were allocated filled with sentinels (NaN, 0xAB bytes): none may remain
    for tf in a[1]:
        assert np.all((tf < wl.T) | (tf == NEVER))
    for v in a[2] + a[3]:
        assert np.all(np.isfinite(v))
    np.testing.assert_array_equal(a[0], b[0])
    for x, y in zip(a[1] + a[2] + a[3], b[1] + b[2] + b[3]):
        np.testing.assert_array_equal(x, y)


def _rate_chain_check(wl, out, pipe, samples):
    """Every stage of the rate-coded inference against the oracle, on the
    given samples (each sample's chain is independent of the others)."""
    from paper_2301_13659_amd.pipeline import RatePipeline  # noqa: F401
    filters = oracle.log_filters(wl.log_stds, wl.log_ksize)
    imgs = np_(pipe.images)
    draws = np_(pipe.draws)
    ws = [np_(l.w) for l in pipe.layers]
    for b in samples:
        x = oracle.threshold(oracle.dog_filter(imgs[b:b + 1], filters), wl.pre_threshold, 0.0)
        np.testing.assert_array_equal(np_(out.dog[b:b + 1]).view(np.uint32), x.view(np.uint32))
        f = oracle.rate_code(x, draws[b:b + 1], wl.T, wl.min_value)
        np.testing.assert_array_equal(np_(out.times0[b:b + 1]), f)
        c = None
        li = pi = 0
        for kind, s in wl.stages:
            if kind == "gather":
                np.testing.assert_array_equal(np_(out.features[b:b + 1]), (c / np.float32(wl.T)).astype(np.float32))
                continue
            if kind == "pool":
                f, c = oracle.rate_pool(f, c, s.k, s.stride, s.pad)
                gf, gc = out.pooled[pi]
                np.testing.assert_array_equal(np_(gc[b:b + 1]), c)
                np.testing.assert_array_equal(np_(gf[b:b + 1]), f)
                pi += 1
                continue
            f, c = oracle.conv_if_rate(f, ws[li], s.stride, s.pad, s.theta)
            gf, gc = out.layer_out[li]
            np.testing.assert_array_equal(np_(gc[b:b + 1]), c)
            np.testing.assert_array_equal(np_(gf[b:b + 1]), f)
            li += 1


def test_rate_inference_reduced_batch():
    from paper_2301_13659_amd.pipeline import RatePipeline
    dev = gpu()
    wl = workloads.get(7).with_batch(2)
    pipe = RatePipeline(wl, dev)
    out = pipe.step(keep=True)
    torch.cuda.synchronize()
    assert 0 < int(np_(out.layer_out[0][1]).sum())  # the layer is in its firing regime
    _rate_chain_check(wl, out, pipe, [0, 1])


def test_rate_inference_full_size_sampled():
    from paper_2301_13659_amd.pipeline import RatePipeline
    dev = gpu()
    wl = workloads.get(7)
    pipe = RatePipeline(wl, dev)
    out = pipe.step(keep=True)
    torch.cuda.synchronize()
    _rate_chain_check(wl, out, pipe, [wl.batch - 1])
