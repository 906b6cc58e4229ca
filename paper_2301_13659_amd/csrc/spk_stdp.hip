// spk_stdp_update: STDP and R-STDP on the winners' receptive fields
// (Spyker §II-F.1 Eq. 4-6, §II-F.2 Eq. 7).
//
// Scatter-free: one workgroup owns kernel o.  It gathers, in (sample, slot)
// order, the winners of map o (a block-wide ordered compaction into LDS), and
// every thread accumulates the changes of its synapses over that list in a
// fixed order, so the float sums are reproducible.  The clamp and the
// optional half refresh happen once at the end.  At most one winner per
// sample can own map o (k-WTA retires a winner's map), so the lists are short.
#include <hip/hip_fp16.h>

#include "spk_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kMaxTaps = 16384;
constexpr int kMaxCfg = 16;

struct StdpCfgs {
    int n;
    spk_stdp_config c[kMaxCfg];
};

struct StdpGeom {
    int Co, Ci, Kh, Kw, stride, pad, B, Hi, Wi, k;
};

struct Entry {
    int b, y, x, t, q;
};

__global__ __launch_bounds__(kThreads) void k_stdp(float *__restrict__ w, uint16_t *__restrict__ w16,
                                                   const uint8_t *__restrict__ in_times,
                                                   const spk_winner *__restrict__ winners,
                                                   const int32_t *__restrict__ n_winners,
                                                   const int32_t *__restrict__ winner_cfg,
                                                   StdpGeom g, StdpCfgs cfg)
{
#pragma clang fp contract(off)
    extern __shared__ float D[];                   // [taps]
    __shared__ Entry list[kThreads];
    __shared__ int s_scan[kThreads];
    const int o = blockIdx.x;
    const int taps = g.Ci * g.Kh * g.Kw;
    const float L = cfg.c[0].lower, U = cfg.c[0].upper;
    for (int j = threadIdx.x; j < taps; j += blockDim.x) D[j] = 0.0f;
    const int total = g.B * g.k;
    int n_total = 0;
    for (int base = 0; base < total; base += blockDim.x) {
        // ordered compaction of this chunk's winners of map o
        const int i = base + threadIdx.x;
        Entry e{0, 0, 0, 0, 0};
        int keep = 0;
        if (i < total) {
            const int b = i / g.k, s = i - b * g.k;
            const spk_winner wn = winners[i];
            const int q = winner_cfg ? winner_cfg[i] : 0;
            if (s < n_winners[b] && wn.c == o && q >= 0 && q < cfg.n) {
                keep = 1;
                e = Entry{b, wn.y, wn.x, wn.t, q};
            }
        }
        s_scan[threadIdx.x] = keep;
        __syncthreads();
        for (int off = 1; off < (int)blockDim.x; off <<= 1) {
            int v = threadIdx.x >= off ? s_scan[threadIdx.x - off] : 0;
            __syncthreads();
            s_scan[threadIdx.x] += v;
            __syncthreads();
        }
        const int n_chunk = s_scan[blockDim.x - 1];
        if (keep) list[s_scan[threadIdx.x] - 1] = e;
        __syncthreads();
        for (int j = threadIdx.x; j < taps; j += blockDim.x) {
            const int c = j / (g.Kh * g.Kw), r = j - c * g.Kh * g.Kw;
            const int ky = r / g.Kw, kx = r - ky * g.Kw;
            const float w0 = w[(size_t)o * taps + j];
            float acc = D[j];
            for (int m = 0; m < n_chunk; m++) {
                const Entry en = list[m];
                const int iy = en.y * g.stride + ky - g.pad, ix = en.x * g.stride + kx - g.pad;
                int t_pre = spk::kNever;
                if (iy >= 0 && iy < g.Hi && ix >= 0 && ix < g.Wi)
                    t_pre = in_times[(((size_t)en.b * g.Ci + c) * g.Hi + iy) * g.Wi + ix];
                const spk_stdp_config &q = cfg.c[en.q];
                const float a = (t_pre <= en.t) ? q.a_causal : q.a_anticausal;
                float d;
                if (q.stabilize) {
                    float lo = a * (w0 - L);
                    d = lo * (U - w0);
                } else {
                    d = a;
                }
                acc = acc + d;
            }
            D[j] = acc;
        }
        n_total += n_chunk;
        __syncthreads();
    }
    if (n_total == 0) return;
    for (int j = threadIdx.x; j < taps; j += blockDim.x) {
        const size_t at = (size_t)o * taps + j;
        float v = w[at] + D[j];
        v = fminf(U, fmaxf(L, v));
        w[at] = v;
        if (w16) {
            __half h = __float2half_rn(v);
            w16[at] = *reinterpret_cast<uint16_t *>(&h);
        }
    }
}

}  // namespace

extern "C" size_t spk_stdp_update_workspace_size(int Co, int Ci, int Kh, int Kw, int B, int k)
{
    (void)Co; (void)Ci; (void)Kh; (void)Kw; (void)B; (void)k;
    return 0;
}

extern "C" spk_status spk_stdp_update(float *w, uint16_t *w_f16, int Co, int Ci, int Kh, int Kw,
                                      int stride, int pad, const uint8_t *in_times, int B, int Hi,
                                      int Wi, const spk_winner *winners, const int32_t *n_winners,
                                      int k, const spk_stdp_config *cfg, int n_cfg,
                                      const int32_t *winner_cfg, void *ws, size_t ws_bytes,
                                      spk_stream stream)
{
    (void)ws; (void)ws_bytes;
    spk::clear_error();
    SPK_REQUIRE(w && in_times && n_winners && cfg && (winners || k == 0), SPK_E_ARG,
                "spk_stdp_update: NULL pointer");
    SPK_REQUIRE(Co > 0 && Ci > 0 && Kh > 0 && Kw > 0 && stride > 0 && pad >= 0 && B > 0 && Hi > 0 &&
                    Wi > 0 && k >= 0 && n_cfg > 0,
                SPK_E_ARG, "spk_stdp_update: sizes must be positive (pad, k >= 0)");
    SPK_REQUIRE((long long)Ci * Kh * Kw <= kMaxTaps && n_cfg <= kMaxCfg, SPK_E_SHAPE,
                "spk_stdp_update: Ci*Kh*Kw <= %d and n_cfg <= %d required", kMaxTaps, kMaxCfg);
    SPK_REQUIRE((long long)B * k < (1LL << 31), SPK_E_SHAPE, "spk_stdp_update: B*k too large");
    for (int q = 0; q < n_cfg; q++) {
        SPK_REQUIRE(cfg[q].lower == cfg[0].lower && cfg[q].upper == cfg[0].upper, SPK_E_UNSUPPORTED,
                    "spk_stdp_update: configurations %d and 0 have different bounds", q);
        SPK_REQUIRE(cfg[q].lower <= cfg[q].upper, SPK_E_ARG,
                    "spk_stdp_update: configuration %d has lower > upper", q);
    }
    SPK_REQUIRE(Co <= 65535 * 64, SPK_E_SHAPE, "spk_stdp_update: Co too large");
    if (k == 0) return SPK_OK;
    StdpGeom g{Co, Ci, Kh, Kw, stride, pad, B, Hi, Wi, k};
    StdpCfgs c{};
    c.n = n_cfg;
    for (int q = 0; q < n_cfg; q++) c.c[q] = cfg[q];
    const size_t lds = (size_t)Ci * Kh * Kw * sizeof(float);
    hipLaunchKernelGGL(k_stdp, dim3(Co), dim3(kThreads), lds, spk::stream_of(stream), w, w_f16,
                       in_times, winners, n_winners, winner_cfg, g, c);
    SPK_LAUNCHED("spk_stdp_update");
    return SPK_OK;
}
