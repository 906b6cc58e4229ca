"""The C ABI without a GPU: the library loads, exports every symbol of
include/spk.h, and rejects bad arguments on the host before any launch."""
import ctypes
import math
import os
import re

import pytest

from paper_2301_13659_amd import spk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spk.h")
P1 = ctypes.c_void_p(256)   # never dereferenced: every call below fails validation first


def _header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(spk_[a-z0-9_]+)\s*\(", text)))


def test_header_symbols_are_exported_and_bound():
    L = spk.load()
    names = _header_functions()
    assert len(names) >= 16
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(spk.symbols())


def test_version_and_out_extent():
    assert spk.version().startswith("spk ")
    L = spk.load()
    # Eq. 2 / Eq. 3 of the paper for a few shapes
    for n, k, s, p in [(28, 5, 1, 2), (28, 2, 2, 0), (14, 3, 3, 1), (160, 7, 6, 0), (26, 17, 1, 0),
                       (9, 4, 2, 1), (1, 1, 1, 0)]:
        assert L.spk_out_extent(n, k, s, p) == (n + 2 * p - k) // s + 1
    assert L.spk_out_extent(3, 5, 1, 0) == -1
    assert L.spk_out_extent(3, 0, 1, 0) == -1
    assert L.spk_out_extent(3, 3, 0, 0) == -1


def _err(status, code, fragment):
    assert status == code, spk.load().spk_last_error()
    assert fragment in spk.load().spk_last_error().decode()


def test_dog_validation():
    L = spk.load()
    good = (spk.DogDesc * 1)(spk.DogDesc(7, 1.0, 2.0))
    _err(L.spk_dog_filter(None, 1, 1, 8, 8, good, 1, -1, P1, None), spk.SPK_E_ARG, "NULL")
    even = (spk.DogDesc * 1)(spk.DogDesc(6, 1.0, 2.0))
    _err(L.spk_dog_filter(P1, 1, 1, 8, 8, even, 1, -1, P1, None), spk.SPK_E_ARG, "odd")
    big = (spk.DogDesc * 1)(spk.DogDesc(23, 1.0, 2.0))
    _err(L.spk_dog_filter(P1, 1, 1, 64, 64, big, 1, -1, P1, None), spk.SPK_E_SHAPE, "ksize")
    mixed = (spk.DogDesc * 2)(spk.DogDesc(3, 1.0, 2.0), spk.DogDesc(5, 1.0, 2.0))
    _err(L.spk_dog_filter(P1, 1, 1, 8, 8, mixed, 2, 1, P1, None), spk.SPK_E_UNSUPPORTED, "pad")
    _err(L.spk_dog_filter(P1, 1, 1, 2, 2, good, 1, 0, P1, None), spk.SPK_E_SHAPE, "empty")
    neg = (spk.DogDesc * 1)(spk.DogDesc(7, -1.0, 2.0))
    _err(L.spk_dog_filter(P1, 1, 1, 8, 8, neg, 1, -1, P1, None), spk.SPK_E_ARG, "sigma")


def test_latency_code_validation_and_workspace():
    L = spk.load()
    _err(L.spk_latency_code(P1, 1, 1, 4, 4, 255, 0.01, 0, P1, None, None, 0, None), spk.SPK_E_SHAPE, "T=")
    _err(L.spk_latency_code(P1, 1, 1, 4, 4, 0, 0.01, 0, P1, None, None, 0, None), spk.SPK_E_SHAPE, "T=")
    _err(L.spk_latency_code(P1, 1, 1, 4, 4, 5, 0.01, 7, P1, None, None, 0, None), spk.SPK_E_ARG, "mode")
    assert L.spk_latency_code_workspace_size(64, 6, 28, 28) == 0           # whole sample in LDS
    need = L.spk_latency_code_workspace_size(32, 6, 160, 250)
    # the bucket lists (up to one key per value) and a 65536-bucket histogram per sample
    assert need >= 32 * 6 * 160 * 250 * 8 + 32 * 65536 * 4
    _err(L.spk_latency_code(P1, 32, 6, 160, 250, 30, 0.01, 0, P1, None, P1, need - 1, None),
         spk.SPK_E_WORKSPACE, "workspace")


def test_dog_latency_code_validation_and_workspace():
    L = spk.load()
    six = (spk.DogDesc * 6)(*[spk.DogDesc(k, s1, s2) for k, s1, s2 in
                              [(3, 0.43, 0.86), (3, 0.86, 0.43), (7, 1.0, 2.0), (7, 2.0, 1.0),
                               (13, 1.86, 3.71), (13, 3.71, 1.86)]])
    # the three-layer net's input stage runs fused: no workspace
    assert L.spk_dog_latency_code_workspace_size(64, 1, 28, 28, six, 6, -1) == 0
    # 6 x 160 x 250 values per sample: filter outputs plus the large-sample coder's workspace
    need = L.spk_dog_latency_code_workspace_size(32, 1, 160, 250, six, 6, -1)
    assert need >= 32 * 6 * 160 * 250 * 4 + L.spk_latency_code_workspace_size(32, 6, 160, 250)
    _err(L.spk_dog_latency_code(P1, 32, 1, 160, 250, six, 6, -1, 30, 0.01, P1, None, P1, need - 1, None),
         spk.SPK_E_WORKSPACE, "workspace")
    _err(L.spk_dog_latency_code(None, 1, 1, 28, 28, six, 6, -1, 15, 0.01, P1, None, None, 0, None),
         spk.SPK_E_ARG, "NULL")
    _err(L.spk_dog_latency_code(P1, 1, 1, 28, 28, six, 6, -1, 255, 0.01, P1, None, None, 0, None),
         spk.SPK_E_SHAPE, "T=")
    even = (spk.DogDesc * 1)(spk.DogDesc(6, 1.0, 2.0))
    _err(L.spk_dog_latency_code(P1, 1, 1, 8, 8, even, 1, -1, 15, 0.01, P1, None, None, 0, None),
         spk.SPK_E_ARG, "odd")
    assert L.spk_dog_latency_code_workspace_size(1, 1, 8, 8, even, 1, -1) == 0


def test_conv_fire_validation():
    L = spk.load()
    args = lambda **kw: dict(dict(B=1, T=5, Ci=2, Hi=8, Wi=8, dt=0, Co=3, Kh=3, Kw=3, s=1, p=1,
                                  theta=1.0), **kw)

    def call(a, w=P1):
        return L.spk_conv_fire(P1, a["B"], a["T"], a["Ci"], a["Hi"], a["Wi"], w, a["dt"], a["Co"],
                               a["Kh"], a["Kw"], a["s"], a["p"], a["theta"], P1, P1, None, None, 0,
                               None)
    _err(call(args(), w=None), spk.SPK_E_ARG, "NULL")
    _err(call(args(T=300)), spk.SPK_E_SHAPE, "T=")
    _err(call(args(dt=5)), spk.SPK_E_UNSUPPORTED, "dtype")
    _err(call(args(Kh=11, p=0)), spk.SPK_E_SHAPE, "no output")
    _err(call(args(s=0)), spk.SPK_E_ARG, "positive")
    _err(call(args(theta=math.nan)), spk.SPK_E_ARG, "NaN")


def test_pool_conv_fire_and_pack_weights_validation():
    L = spk.load()
    F32, F16 = spk.SPK_F32, spk.SPK_F16

    def call(B=2, T=15, Ci=30, H0=28, W0=28, pk=2, pw=2, ps=2, pp=0, packed=None, Co=250, K=3,
             s=1, p=1, theta=10.0, ws=P1, nbytes=1 << 30, w=P1, src=P1):
        return L.spk_pool_conv_fire(src, B, T, Ci, H0, W0, pk, pw, ps, pp, None, w, F32, packed, Co,
                                    K, K, s, p, theta, P1, P1, ws, nbytes, None)
    _err(call(src=None), spk.SPK_E_ARG, "NULL")
    _err(call(w=None), spk.SPK_E_ARG, "NULL")
    _err(call(ps=0), spk.SPK_E_ARG, "positive")
    _err(call(pk=30), spk.SPK_E_SHAPE, "no pooled output")
    _err(call(packed=ctypes.c_void_p(256 + 8)), spk.SPK_E_ARG, "aligned")
    _err(call(T=300), spk.SPK_E_SHAPE, "T=")
    _err(call(K=20, p=0), spk.SPK_E_SHAPE, "no output")
    _err(call(theta=math.nan), spk.SPK_E_ARG, "NaN")
    _err(call(ws=ctypes.c_void_p(256 + 16)), spk.SPK_E_ARG, "aligned")
    need = L.spk_pool_conv_fire_workspace_size(2, 15, 30, 28, 28, 2, 2, 2, 0, 250, 3, 3, 1, 1, 10.0)
    conv = L.spk_conv_fire_workspace_size(2, 15, 30, 14, 14, 250, 3, 3, 1, 1, 10.0, 0)
    # the conv's own workspace, then room for a pooled map
    assert need == (conv + 255) // 256 * 256 + (2 * 30 * 14 * 14 + 255) // 256 * 256
    _err(call(nbytes=need - 1), spk.SPK_E_WORKSPACE, "workspace")
    assert L.spk_pool_conv_fire_workspace_size(2, 15, 30, 28, 28, 40, 40, 1, 0, 250, 3, 3, 1, 1,
                                               10.0) == 0

    # B fragments of the three-layer net's readout: 7 tiles of 32 maps, 5 kernel
    # rows of 5 x 264 taps (250 channels padded to 33 x 8) = 413 slices of 16
    assert L.spk_conv_packed_weights_size(200, 250, 5, 5, F32) == 7 * 413 * 2 * 64 * 16
    assert L.spk_conv_packed_weights_size(200, 250, 5, 5, F16) == 7 * 413 * 1 * 64 * 16
    # 16 channels -> 24: 3 rows of 72 taps = 14 slices
    assert L.spk_conv_packed_weights_size(40, 16, 3, 3, F32) == 2 * 14 * 2 * 64 * 16
    assert L.spk_conv_packed_weights_size(1, 3, 1, 1, F16) == 1 * 1 * 1 * 64 * 16
    assert L.spk_conv_packed_weights_size(200, 250, 5, 5, 7) == 0
    assert L.spk_conv_packed_weights_size(0, 250, 5, 5, F32) == 0
    n = L.spk_conv_packed_weights_size(200, 250, 5, 5, F32)
    _err(L.spk_conv_pack_weights(None, F32, 200, 250, 5, 5, P1, n, None), spk.SPK_E_ARG, "NULL")
    _err(L.spk_conv_pack_weights(P1, 9, 200, 250, 5, 5, P1, n, None), spk.SPK_E_UNSUPPORTED, "dtype")
    _err(L.spk_conv_pack_weights(P1, F32, 200, 250, 5, 5, P1, n - 1, None), spk.SPK_E_WORKSPACE,
         "needed")
    _err(L.spk_conv_pack_weights(P1, F32, 200, 250, 5, 5, ctypes.c_void_p(264), n, None),
         spk.SPK_E_ARG, "aligned")
    _err(L.spk_conv_pack_weights(P1, F32, 2, 2000, 3, 3, P1, 1 << 30, None), spk.SPK_E_SHAPE, "taps")
    _err(L.spk_conv_pack_weights(P1, F32, 0, 250, 5, 5, P1, n, None), spk.SPK_E_ARG, "positive")


def test_pool_inhibit_stdp_validation():
    L = spk.load()
    _err(L.spk_pool(P1, 1, 1, 2, 2, 3, 3, 1, 0, P1, None), spk.SPK_E_SHAPE, "no output")
    _err(L.spk_inhibit_winners(P1, P1, 1, 4, 5, 5, 15, 1, 2, 1, 1, None, P1, P1, P1, 1 << 20, None),
         spk.SPK_E_UNSUPPORTED, "readout")
    _err(L.spk_inhibit_winners(P1, P1, 2, 4, 5, 5, 15, 1, 2, 1, 0, None, P1, P1, None, 0, None),
         spk.SPK_E_WORKSPACE, "workspace")
    _err(L.spk_inhibit_winners(P1, P1, 2, 4, 5, 5, 15, 1, -1, 1, 0, None, P1, P1, P1, 1 << 20, None),
         spk.SPK_E_ARG, "k=")
    cfg = (spk.StdpConfig * 2)(spk.StdpConfig(0.004, -0.003, 0.0, 1.0, 1),
                               spk.StdpConfig(0.004, -0.003, 0.1, 1.0, 1))
    _err(L.spk_stdp_update(P1, None, 3, 2, 3, 3, 1, 1, P1, 2, 8, 8, P1, P1, 1, cfg, 2, None, None, 0,
                           None), spk.SPK_E_UNSUPPORTED, "bounds")
    _err(L.spk_stdp_update(P1, None, 3, 2000, 3, 3, 1, 1, P1, 2, 8, 8, P1, P1, 1, cfg, 1, None, None,
                           0, None), spk.SPK_E_SHAPE, "Ci*Kh*Kw")
    _err(L.spk_rstdp_select(P1, P1, 2, 1, P1, 0, P1, None), spk.SPK_E_ARG, "group")
    _err(L.spk_times_to_frames(P1, 1, 0, 10, P1, None), spk.SPK_E_SHAPE, "T=")


def test_binding_rejects_host_tensors():
    import torch
    with pytest.raises(ValueError):
        spk.spk_pool(torch.zeros((1, 1, 4, 4), dtype=torch.uint8), 2)


@pytest.mark.skipif(__import__("torch").cuda.is_available(),
                    reason="launches with placeholder pointers: only meaningful without a GPU")
def test_conv_fire_planning_survives_every_layer_shape():
    # Valid arguments reach the launch (which fails without a device): the
    # host-side tile planning must not trap on any workload shape.
    L = spk.load()
    shapes = [(8, 15, 2, 28, 28, 32, 5, 2, 15.0), (64, 15, 6, 28, 28, 30, 5, 2, 15.0),
              (64, 15, 30, 14, 14, 250, 3, 1, 10.0), (64, 15, 250, 5, 5, 200, 5, 2, math.inf),
              (32, 30, 6, 160, 250, 4, 5, 2, 15.0), (32, 30, 4, 26, 41, 20, 17, 0, 42.0),
              (128, 30, 64, 64, 64, 128, 3, 1, 20.0), (1, 1, 1, 1, 1, 1, 1, 0, 0.5)]
    for B, T, Ci, H, W, Co, K, pad, theta in shapes:
        ws = L.spk_conv_fire_workspace_size(B, T, Ci, H, W, Co, K, K, 1, pad, theta, 0)
        st = L.spk_conv_fire(P1, B, T, Ci, H, W, P1, 0, Co, K, K, 1, pad, theta, P1, P1, None,
                             P1 if ws else None, ws, None)
        assert st == spk.SPK_E_HIP, spk.load().spk_last_error()
    # and with the pooling in front: (B, T, Ci, H0, W0, pool k, stride, pad, Co, K, pad, theta, packed)
    pooled = [(64, 15, 30, 28, 28, 2, 2, 0, 250, 3, 1, 10.0, None),
              (64, 15, 250, 14, 14, 3, 3, 1, 200, 5, 2, math.inf, P1),
              (32, 30, 4, 160, 250, 7, 6, 0, 20, 17, 0, 42.0, None),
              (2, 40, 8, 12, 12, 2, 2, 1, 20, 3, 1, 5.0, None)]
    for B, T, Ci, H0, W0, pk, ps, pp, Co, K, pad, theta, packed in pooled:
        ws = L.spk_pool_conv_fire_workspace_size(B, T, Ci, H0, W0, pk, pk, ps, pp, Co, K, K, 1, pad,
                                                 theta)
        st = L.spk_pool_conv_fire(P1, B, T, Ci, H0, W0, pk, pk, ps, pp, P1, P1, 0, packed, Co, K, K,
                                  1, pad, theta, P1, P1, P1, ws, None)
        assert st == spk.SPK_E_HIP, spk.load().spk_last_error()
    n = L.spk_conv_packed_weights_size(200, 250, 5, 5, 0)
    assert L.spk_conv_pack_weights(P1, 0, 200, 250, 5, 5, P1, n, None) == spk.SPK_E_HIP


def test_fc_validation():
    L = spk.load()
    _err(L.spk_fc_winners(None, P1, 1, 8, 4, 1, 0, 0, P1, P1, None), spk.SPK_E_ARG, "NULL")
    _err(L.spk_fc_winners(P1, P1, 1, 8, 4, 1, -1, 0, P1, P1, None), spk.SPK_E_ARG, "radius")
    _err(L.spk_fc_winners(P1, P1, 1, 1 << 17, 4, 1, 0, 0, P1, P1, None), spk.SPK_E_SHAPE, "O=")
    _err(L.spk_fc_winners(P1, P1, 1, 8, 0, 1, 0, 0, P1, P1, None), spk.SPK_E_SHAPE, "T=")
    _err(L.spk_fc_winners(P1, P1, 1, 8, 4, 5000, 0, 0, P1, P1, None), spk.SPK_E_SHAPE, "k=")
    _err(L.spk_fc_fire(P1, 0, 4, 8, P1, spk.SPK_F32, 3, 1.0, P1, P1, None, None, 0, None),
         spk.SPK_E_ARG, "positive")
    _err(L.spk_fc_fire(None, 1, 4, 8, P1, spk.SPK_F32, 3, 1.0, P1, P1, None, None, 0, None),
         spk.SPK_E_ARG, "NULL")


def test_sparse_validation():
    L = spk.load()
    F32, F16 = spk.SPK_F32, spk.SPK_F16
    _err(L.spk_times_to_spikes(None, 1, 2, 3, 4, 5, 10, P1, P1, P1, 1 << 20, None), spk.SPK_E_ARG,
         "NULL")
    _err(L.spk_times_to_spikes(P1, 1, 2, 3, 4, 255, 10, P1, P1, P1, 1 << 20, None), spk.SPK_E_SHAPE,
         "T=")
    _err(L.spk_times_to_spikes(P1, 1, 2, 3, 4, 5, 10, P1, P1, P1, 0, None), spk.SPK_E_WORKSPACE,
         "workspace")
    assert L.spk_times_to_spikes_workspace_size(2, 64, 64, 64, 30) > 0
    _err(L.spk_spikes_to_times(P1, P1, -1, 1, 2, 3, 4, 5, P1, None), spk.SPK_E_ARG, "cap")
    _err(L.spk_spikes_to_times(P1, None, 4, 1, 2, 3, 4, 5, P1, None), spk.SPK_E_ARG, "NULL")
    args = [P1, P1, 100, 2, 15, 6, 28, 28, P1, F32, 30, 5, 5, 1, 2, 10.0, P1, P1, P1, 1 << 30, None]
    ok = list(args)
    bad = list(ok); bad[4] = 0
    _err(L.spk_conv_fire_sparse(*bad), spk.SPK_E_SHAPE, "T=")
    bad = list(ok); bad[9] = 7
    _err(L.spk_conv_fire_sparse(*bad), spk.SPK_E_UNSUPPORTED, "dtype")
    bad = list(ok); bad[11] = 40
    _err(L.spk_conv_fire_sparse(*bad), spk.SPK_E_SHAPE, "empty")
    bad = list(ok); bad[15] = float("nan")
    _err(L.spk_conv_fire_sparse(*bad), spk.SPK_E_ARG, "NaN")
    bad = list(ok); bad[19] = 16
    _err(L.spk_conv_fire_sparse(*bad), spk.SPK_E_WORKSPACE, "workspace")
    bad = list(ok); bad[5] = 4096; bad[9] = F16
    _err(L.spk_conv_fire_sparse(*bad), spk.SPK_E_UNSUPPORTED, "LDS")
    assert L.spk_conv_fire_sparse_workspace_size(2, 15, 6, 28, 28, 30, 5, 5, 1, 2, F32) > 0
    assert L.spk_conv_fire_sparse_workspace_size(2, 15, 4096, 28, 28, 30, 5, 5, 1, 2, F16) == 0


def test_demo_ops_validation():
    import ctypes
    L = spk.load()
    stds = (ctypes.c_float * 5)(0.5, 1.0, 1.5, 2.0, 2.5)
    _err(L.spk_log_filter(P1, 1, 1, 8, 8, stds, 5, 7, -1, P1, None), spk.SPK_E_SHAPE, "8 filters")
    bad = (ctypes.c_float * 1)(-1.0)
    _err(L.spk_log_filter(P1, 1, 1, 8, 8, bad, 1, 7, -1, P1, None), spk.SPK_E_ARG, "positive")
    _err(L.spk_log_filter(P1, 1, 1, 8, 8, stds, 1, 6, -1, P1, None), spk.SPK_E_ARG, "odd")
    _err(L.spk_threshold(P1, 10, float("nan"), 0.0, None), spk.SPK_E_ARG, "NaN")
    _err(L.spk_threshold(None, 10, 0.1, 0.0, None), spk.SPK_E_ARG, "NULL")
    _err(L.spk_quantize(P1, None, -1, 0.0, 0.5, 1.0, None), spk.SPK_E_ARG, "n=")
    _err(L.spk_gather(P1, 10, 0, P1, None), spk.SPK_E_SHAPE, "T=")
    assert L.spk_threshold(None, 0, 0.1, 0.0, None) == spk.SPK_OK


def test_rate_and_batch_limits_validation():
    L = spk.load()
    F16 = spk.SPK_F16
    _err(L.spk_spikes_to_times(P1, P1, 4, 70000, 2, 3, 4, 5, P1, None), spk.SPK_E_SHAPE, "B=")
    _err(L.spk_rate_code(P1, P1, 2, 10, 5, -0.1, P1, P1, 8, None), spk.SPK_E_ARG, "min_value")
    _err(L.spk_rate_code(P1, P1, 2, 10, 5, 0.0, P1, P1, 4, None), spk.SPK_E_WORKSPACE, "workspace")
    _err(L.spk_conv_if_rate(P1, 1, 10, 6, 8, 8, P1, F16, 4, 3, 3, 1, 1, float("inf"), P1, P1, P1,
                            1 << 30, None), spk.SPK_E_ARG, "finite")
    _err(L.spk_conv_if_rate(P1, 1, 10, 6, 8, 8, P1, F16, 4, 13, 3, 1, 1, 1.0, P1, P1, P1, 1 << 30, None),
         spk.SPK_E_SHAPE, "empty")
    _err(L.spk_conv_if_rate(P1, 1, 10, 6, 8, 8, P1, F16, 4, 3, 3, 1, 1, 1.0, P1, P1, P1, 8, None),
         spk.SPK_E_WORKSPACE, "workspace")
    _err(L.spk_rate_pool(P1, P1, 1, 10, 3, 4, 4, 5, 5, 1, 0, P1, P1, None), spk.SPK_E_SHAPE, "empty")
    assert L.spk_conv_if_rate_workspace_size(2, 300, 6, 28, 28, 25, 5, 5, 1, 2, F16) > 0


def test_misaligned_workspace_is_rejected():
    """Workspaces must be 256-byte aligned: every call that takes one says so
    before launching anything."""
    L = spk.load()
    bad = ctypes.c_void_p(256 + 16)
    _err(L.spk_latency_code(P1, 32, 6, 160, 250, 30, 0.01, 0, P1, None, bad, 1 << 30, None),
         spk.SPK_E_ARG, "aligned")
    _err(L.spk_conv_fire(P1, 1, 5, 2, 8, 8, P1, 0, 3, 3, 3, 1, 1, 1.0, P1, P1, None, bad, 1 << 30,
                         None), spk.SPK_E_ARG, "aligned")
    _err(L.spk_inhibit_winners(P1, P1, 2, 4, 5, 5, 15, 1, 2, 1, 0, None, P1, P1, bad, 1 << 20, None),
         spk.SPK_E_ARG, "aligned")
    _err(L.spk_rate_code(P1, P1, 2, 10, 5, 0.0, P1, bad, 1 << 20, None), spk.SPK_E_ARG, "aligned")



def test_conv_fire_noalloc_rejects_layers_beyond_its_scratch():
    """The no-allocation conv checks the layer's scratch need against its
    static maximum before it touches the device."""
    L = spk.load()
    # the spike-input layer at batch 1024 needs about 275 MiB of scratch
    st = L.spk_conv_fire_noalloc(P1, 1024, 30, 64, 64, 64, P1, spk.SPK_F16, 128, 3, 3, 1, 1, 20.0,
                                 P1, P1, None, None)
    _err(st, spk.SPK_E_WORKSPACE, "static")
