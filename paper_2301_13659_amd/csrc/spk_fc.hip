// Fully connected spiking layer (Spyker §II-E.2) and its winner selection
// (fcwta, §II-F.3).
//
// The FC layer has an I x O kernel over B x T x I input spikes and IF
// neurons; under rank-order coding each output neuron fires once.  Its
// potential V_t[b, o] = sum_i W[o, i] * [in_times[b, i] <= t] is the spiking
// convolution of a 1 x 1 kernel over I input channels on a 1 x 1 image, so
// spk_fc_fire and spk_fc_stdp_update run the convolution and STDP kernels on
// that geometry (the B x I and O x I arrays are B x I x 1 x 1 and
// O x I x 1 x 1 as they are laid out).  The winner selection of an FC layer
// differs from convwta: its radius runs along the neuron index, the only
// dimension an FC layer has, so it has its own kernel here.
#include <cstdint>

#include "spk_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kMaxFcO = 1 << 16;  // neurons per sample: alive flags in LDS

// Order key of a candidate, smaller is better: spike time (0 in readout
// mode), then higher potential, then lower index.
__device__ __forceinline__ uint64_t fc_key(uint32_t t, float v, uint32_t o)
{
    uint32_t u = __float_as_uint(v);
    u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);  // ascending with v
    return ((uint64_t)t << 56) | ((uint64_t)(~u) << 24) | (uint64_t)o;
}

__device__ __forceinline__ uint64_t wave_min64(uint64_t x)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)x, m);
        const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(x >> 32), m);
        const uint64_t y = ((uint64_t)hi << 32) | lo;
        x = y < x ? y : x;
    }
    return x;
}

// One block per sample: up to k rounds of a block-wide arg-min over the
// remaining candidates, each followed by removing the winner's index window.
__global__ __launch_bounds__(kThreads) void k_fc_wta(const uint8_t *__restrict__ times,
                                                     const float *__restrict__ vkey, int O, int T,
                                                     int k, int radius, int readout,
                                                     spk_winner *__restrict__ winners,
                                                     int32_t *__restrict__ n_winners)
{
    extern __shared__ uint8_t alive[];
    __shared__ uint64_t s_min[kThreads / 64];
    const int b = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint8_t *tb = times + (size_t)b * O;
    const float *vb = vkey + (size_t)b * O;
    for (int o = threadIdx.x; o < O; o += kThreads) alive[o] = readout ? 1 : (tb[o] != spk::kNever);
    __syncthreads();
    const uint64_t none = ~0ull;
    int count = 0;
    for (int round = 0; round < k; round++) {
        uint64_t best = none;
        for (int o = threadIdx.x; o < O; o += kThreads)
            if (alive[o]) {
                const uint64_t key = fc_key(readout ? 0u : (uint32_t)tb[o], vb[o], (uint32_t)o);
                best = key < best ? key : best;
            }
        best = wave_min64(best);
        if (lane == 0) s_min[wave] = best;
        __syncthreads();
        best = s_min[0];
#pragma unroll
        for (int w = 1; w < kThreads / 64; w++) best = s_min[w] < best ? s_min[w] : best;
        __syncthreads();  // s_min is reused next round
        if (best == none) break;
        const int o = (int)(best & 0xFFFFFFu);
        if (threadIdx.x == 0) {
            spk_winner wn;
            wn.c = o;
            wn.y = 0;
            wn.x = 0;
            wn.t = readout ? T - 1 : (int)tb[o];
            wn.v = vb[o];
            winners[(size_t)b * k + count] = wn;
        }
        count++;
        const int lo = max(0, o - radius), hi = min(O - 1, o + radius);
        for (int j = lo + (int)threadIdx.x; j <= hi; j += kThreads) alive[j] = 0;
        __syncthreads();
    }
    if (threadIdx.x == 0) n_winners[b] = count;
    for (int s = count + (int)threadIdx.x; s < k; s += kThreads) {
        spk_winner wn;
        wn.c = -1;
        wn.y = wn.x = wn.t = -1;
        wn.v = 0.0f;
        winners[(size_t)b * k + s] = wn;
    }
}

}  // namespace

extern "C" size_t spk_fc_fire_workspace_size(int B, int T, int I, int O, float theta, int potentials)
{
    return spk_conv_fire_workspace_size(B, T, I, 1, 1, O, 1, 1, 1, 0, theta, potentials);
}

extern "C" spk_status spk_fc_fire(const uint8_t *in_times, int B, int T, int I, const void *w,
                                  spk_dtype w_dtype, int O, float theta, uint8_t *out_times,
                                  float *out_vkey, float *potentials, void *ws, size_t ws_bytes,
                                  spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(B > 0 && I > 0 && O > 0, SPK_E_ARG, "spk_fc_fire: sizes must be positive");
    return spk_conv_fire(in_times, B, T, I, 1, 1, w, w_dtype, O, 1, 1, 1, 0, theta, out_times,
                         out_vkey, potentials, ws, ws_bytes, stream);
}

extern "C" spk_status spk_fc_winners(const uint8_t *times, const float *vkey, int B, int O, int T,
                                     int k, int radius, int readout, spk_winner *winners,
                                     int32_t *n_winners, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(times && vkey && winners && n_winners, SPK_E_ARG, "spk_fc_winners: NULL pointer");
    SPK_REQUIRE(B > 0 && O > 0 && k > 0 && radius >= 0, SPK_E_ARG,
                "spk_fc_winners: sizes must be positive (radius >= 0)");
    SPK_REQUIRE(T >= 1 && T <= SPK_MAX_T, SPK_E_SHAPE, "spk_fc_winners: T=%d not in [1, %d]", T,
                SPK_MAX_T);
    SPK_REQUIRE(O <= kMaxFcO, SPK_E_SHAPE, "spk_fc_winners: O=%d > %d", O, kMaxFcO);
    SPK_REQUIRE(k <= 4096, SPK_E_SHAPE, "spk_fc_winners: k=%d > 4096", k);
    hipLaunchKernelGGL(k_fc_wta, dim3(B), dim3(kThreads), (size_t)O, spk::stream_of(stream), times,
                       vkey, O, T, k, radius, readout ? 1 : 0, winners, n_winners);
    SPK_LAUNCHED("spk_fc_winners");
    return SPK_OK;
}

extern "C" size_t spk_fc_stdp_update_workspace_size(int O, int I, int B, int k)
{
    return spk_stdp_update_workspace_size(O, I, 1, 1, B, k);
}

extern "C" spk_status spk_fc_stdp_update(float *w, uint16_t *w_f16, int O, int I,
                                         const uint8_t *in_times, int B,
                                         const spk_winner *winners, const int32_t *n_winners,
                                         int k, const spk_stdp_config *cfg, int n_cfg,
                                         const int32_t *winner_cfg, void *ws, size_t ws_bytes,
                                         spk_stream stream)
{
    spk::clear_error();
    return spk_stdp_update(w, w_f16, O, I, 1, 1, 1, 0, in_times, B, 1, 1, winners, n_winners, k,
                           cfg, n_cfg, winner_cfg, ws, ws_bytes, stream);
}
