"""Comparison rules between the GPU library and the CPU oracle.

 - spike times, winners, pooled times, DoG outputs and latency codes:
   bit-exact;
 - a spike time may differ only for an *excused* neuron, one whose oracle
   potential comes within 1e-4 * |theta| of theta at some step (float
   accumulation order can move it across the threshold);
 - potentials: |V_gpu - V_oracle| <= 1e-4 * |V_oracle| + 1e-6;
 - weights: |W_gpu - W_oracle| <= 1e-5.
"""
import numpy as np
import torch

NEVER = 255
V_REL, V_ABS = 1e-4, 1e-6
W_ABS = 1e-5


def gpu():
    import pytest
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def np_(t):
    return t.detach().cpu().numpy()


def excused_from_potentials(V, theta):
    """V: oracle potentials B x T x C x H x W -> bool B x C x H x W."""
    if not np.isfinite(theta):
        return np.zeros(V.shape[:1] + V.shape[2:], bool)
    return (np.abs(V.astype(np.float64) - theta) <= 1e-4 * abs(theta)).any(axis=1)


def check_potentials(got, ref, what="potentials"):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    bad = ~(np.abs(got - ref) <= V_REL * np.abs(ref) + V_ABS)  # NaN (an unwritten sentinel) is bad
    assert not bad.any(), (f"{what}: {bad.sum()} of {bad.size} outside tolerance, e.g. "
                           f"{got[bad][:5]} vs {ref[bad][:5]}")


def check_fire(g_tf, g_vk, o_tf, o_vk, excused):
    """Returns the number of excused neurons whose times differ."""
    diff = g_tf != o_tf
    bad = diff & ~excused
    assert not bad.any(), (f"spike times differ on {bad.sum()} non-excused neurons, e.g. at "
                           f"{np.argwhere(bad)[:5].tolist()}: gpu {g_tf[bad][:5]} oracle {o_tf[bad][:5]}")
    keep = ~excused
    check_potentials(g_vk[keep], o_vk[keep], "v_key")
    return int((diff & excused).sum())


def winners_list(win, n):
    """numpy structured winners + counts -> list of per-sample tuples."""
    return [[(int(w["c"]), int(w["y"]), int(w["x"]), int(w["t"]), float(w["v"]))
             for w in win[b, :n[b]]] for b in range(win.shape[0])]
