// spk_stdp_update: STDP and R-STDP on the winners' receptive fields
// (Spyker §II-F.1 Eq. 4-6, §II-F.2 Eq. 7).
//
// Scatter-free: one workgroup owns kernel o.  It gathers, in (sample, slot)
// order, the winners of map o (an ordered ballot compaction into LDS), and
// every thread accumulates the changes of its synapses over that list in a
// fixed order, so the float sums are reproducible.  The clamp and the
// optional half refresh happen once at the end.  At most one winner per
// sample can own map o (k-WTA retires a winner's map), so the lists are short.
#include <hip/hip_fp16.h>

#include "spk_internal.h"

namespace {

constexpr int kThreads = 1024;
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

// Sum, from `init`, of the changes of synapse j of map o over the winners
// first, first + step, ... of the list.  The pre-spike loads do not depend on
// each other: they are unconditional (clamped index) so several overlap.
__device__ __forceinline__ float patch_sum(const float *__restrict__ w,
                                           const uint8_t *__restrict__ in_times, const Entry *list,
                                           const StdpGeom &g, int o, int taps, int KK, int j,
                                           int first, int step, int n, float L, float U,
                                           const float (*rate)[2], const int *stab, float init)
{
#pragma clang fp contract(off)
    const int c = j / KK, r = j - c * KK;
    const int ky = r / g.Kw, kx = r - ky * g.Kw;
    const float w0 = w[(size_t)o * taps + j];
    const float wl = w0 - L, wu = U - w0;
    float acc = init;
    auto pre_time = [&](const Entry &en) {
        const int iy = en.y * g.stride + ky - g.pad, ix = en.x * g.stride + kx - g.pad;
        const bool inside = (unsigned)iy < (unsigned)g.Hi && (unsigned)ix < (unsigned)g.Wi;
        const size_t at = inside ? (((size_t)en.b * g.Ci + c) * g.Hi + iy) * g.Wi + ix : 0;
        const int t = in_times[at];
        return inside ? t : spk::kNever;
    };
    auto add = [&](const Entry &en, int t_pre) {
        const float a = rate[en.q][t_pre <= en.t ? 0 : 1];
        float d = a * wl;
        d = d * wu;
        acc = acc + (stab[en.q] ? d : a);
    };
    // winners in batches of 8: the pre-spike loads of a batch are issued
    // before any is used; the sum keeps the winners' order
    int m = first;
    for (; m + 7 * step < n; m += 8 * step) {
        Entry en[8];
        int tp[8];
#pragma unroll
        for (int u = 0; u < 8; u++) en[u] = list[m + u * step];
#pragma unroll
        for (int u = 0; u < 8; u++) tp[u] = pre_time(en[u]);
#pragma unroll
        for (int u = 0; u < 8; u++) add(en[u], tp[u]);
    }
    for (; m < n; m += step) {
        const Entry en = list[m];
        add(en, pre_time(en));
    }
    return acc;
}

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
    __shared__ float part[kThreads];
    __shared__ int wave_cnt[kThreads / 64];
    __shared__ float s_rate[kMaxCfg][2];           // a_causal, a_anticausal
    __shared__ int s_stab[kMaxCfg];
    const int o = blockIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int taps = g.Ci * g.Kh * g.Kw, KK = g.Kh * g.Kw;
    const float L = cfg.c[0].lower, U = cfg.c[0].upper;
    if (threadIdx.x < cfg.n) {
        s_rate[threadIdx.x][0] = cfg.c[threadIdx.x].a_causal;
        s_rate[threadIdx.x][1] = cfg.c[threadIdx.x].a_anticausal;
        s_stab[threadIdx.x] = cfg.c[threadIdx.x].stabilize;
    }
    for (int j = threadIdx.x; j < taps; j += blockDim.x) D[j] = 0.0f;
    const int total = g.B * g.k;
    int n_total = 0;
    for (int base = 0; base < total; base += blockDim.x) {
        // ordered compaction of this chunk's winners of map o: ballot rank
        // within the wave, wave counts through LDS
        const int i = base + threadIdx.x;
        Entry e{0, 0, 0, 0, 0};
        bool keep = false;
        if (i < total) {
            const int b = i / g.k, slot = i - b * g.k;
            const spk_winner wn = winners[i];
            const int q = winner_cfg ? winner_cfg[i] : 0;
            keep = slot < n_winners[b] && wn.c == o && q >= 0 && q < cfg.n;
            e = Entry{b, wn.y, wn.x, wn.t, q};
        }
        const uint64_t m = __ballot(keep);
        const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        if (lane == 0) wave_cnt[wave] = __popcll(m);
        __syncthreads();
        int before = 0, n_chunk = 0;
#pragma unroll
        for (int v = 0; v < kThreads / 64; v++) {
            const int c = wave_cnt[v];
            before += v < wave ? c : 0;
            n_chunk += c;
        }
        if (keep) list[before + rank] = e;
        __syncthreads();
        if (n_chunk > 0) {
            // G groups of `taps` threads share the winners (group g takes
            // winners g, g + G, ...); the G partial sums are added to D in
            // group order, so the result is the same on every run.
            const int G = taps <= kThreads / 2 ? min(n_chunk, kThreads / taps) : 1;
            if (G > 1) {
                if (threadIdx.x < G * taps) {
                    const int grp = threadIdx.x / taps, j = threadIdx.x - grp * taps;
                    part[threadIdx.x] = patch_sum(w, in_times, list, g, o, taps, KK, j, grp, G,
                                                  n_chunk, L, U, s_rate, s_stab, 0.0f);
                }
                __syncthreads();
                for (int j = threadIdx.x; j < taps; j += blockDim.x) {
                    float acc = D[j];
                    for (int q = 0; q < G; q++) acc = acc + part[q * taps + j];
                    D[j] = acc;
                }
            } else {
                for (int j = threadIdx.x; j < taps; j += blockDim.x)
                    D[j] = patch_sum(w, in_times, list, g, o, taps, KK, j, 0, 1, n_chunk, L, U, s_rate,
                                     s_stab, D[j]);
            }
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
