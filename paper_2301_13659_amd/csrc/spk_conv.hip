// spk_conv_fire: spiking convolution + integrate-and-fire (Spyker §II-E.1, Eq. 2).
//
// Dispatch: firing layers whose weights fit the registers of a wave (see
// spk_conv_fast.hip), with T <= 32 and no dense potentials requested, run the
// register-resident kernels there; other shapes the matrix-core kernels of
// spk_conv_mfma.hip cover (readout layers and the dense-potential mode among
// them) go there; the rest take the direct form below:
// one thread per output neuron (b, o, y, x) walks the time steps, sums the
// weights of the inputs of its window that have fired by step t (the
// cumulative frame S_t = [time <= t]) and records the first step whose
// potential exceeds theta.  Kernel o's weights are staged in LDS as float.
#include <hip/hip_fp16.h>

#include <algorithm>

#include "spk_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kMaxTaps = 16384;  // Ci*Kh*Kw staged in LDS (64 KB of float)

struct ConvGeom {
    int B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo;
};

template <bool kHalf>
__global__ __launch_bounds__(kThreads) void k_conv_fire_direct(
    const uint8_t *__restrict__ in_times, const void *__restrict__ wv, ConvGeom g, float theta,
    uint8_t *__restrict__ out_times, float *__restrict__ out_vkey, float *__restrict__ potentials)
{
    extern __shared__ float wl[];
    const int o = blockIdx.y, b = blockIdx.z;
    const int taps = g.Ci * g.Kh * g.Kw;
    for (int i = threadIdx.x; i < taps; i += blockDim.x) {
        size_t at = (size_t)o * taps + i;
        if (kHalf) {
            __half h = reinterpret_cast<const __half *>(wv)[at];
            wl[i] = __half2float(h);
        } else {
            wl[i] = reinterpret_cast<const float *>(wv)[at];
        }
    }
    __syncthreads();
    const int pos = blockIdx.x * blockDim.x + threadIdx.x;
    if (pos >= g.Ho * g.Wo) return;
    const int y = pos / g.Wo, x = pos - y * g.Wo;
    const uint8_t *src = in_times + (size_t)b * g.Ci * g.Hi * g.Wi;
    uint8_t tf = spk::kNever;
    float vkey = 0.0f;
    for (int t = 0; t < g.T; t++) {
        float acc = 0.0f;
        for (int c = 0; c < g.Ci; c++)
            for (int ky = 0; ky < g.Kh; ky++) {
                int iy = y * g.stride + ky - g.pad;
                if (iy < 0 || iy >= g.Hi) continue;
                const uint8_t *row = src + ((size_t)c * g.Hi + iy) * g.Wi;
                const float *wr = wl + (c * g.Kh + ky) * g.Kw;
                for (int kx = 0; kx < g.Kw; kx++) {
                    int ix = x * g.stride + kx - g.pad;
                    if (ix >= 0 && ix < g.Wi && row[ix] <= t) acc += wr[kx];
                }
            }
        if (potentials)
            potentials[(((size_t)b * g.T + t) * g.Co + o) * g.Ho * g.Wo + pos] = acc;
        if (tf == spk::kNever && acc > theta) {
            tf = (uint8_t)t;
            vkey = acc;
        }
        if (t == g.T - 1 && tf == spk::kNever) vkey = acc;
    }
    const size_t n = ((size_t)b * g.Co + o) * g.Ho * g.Wo + pos;
    out_times[n] = tf;
    out_vkey[n] = vkey;
}

}  // namespace

static bool is_readout(float theta, bool potentials) { return !(theta <= 3.4e38f) && !potentials; }

extern "C" size_t spk_conv_fire_workspace_size(int B, int T, int Ci, int Hi, int Wi, int Co,
                                               int Kh, int Kw, int stride, int pad, float theta,
                                               int potentials)
{
    const int Ho = spk_out_extent(Hi, Kh, stride, pad), Wo = spk_out_extent(Wi, Kw, stride, pad);
    if (B <= 0 || Ci <= 0 || Co <= 0 || Ho <= 0 || Wo <= 0) return 0;
    const bool readout = is_readout(theta, potentials != 0);
    size_t need = spk::conv_mfma_workspace(B, Ho, Wo, Co, Ci * Kh * Kw, readout);
    // the channels-last path is open to half weights on more shapes than to
    // float ones, and its workspace does not depend on the weight type
    if (spk::conv_fast_supported(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo, true, readout,
                                 potentials != 0))
        need = std::max(need, spk::conv_fast_workspace(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo));
    if (readout && spk::readout_fast_supported(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo))
        need = std::max(need,
                        spk::readout_fast_workspace(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo));
    for (int hw = 0; hw < 2; hw++)
        if (spk::conv_pt_supported(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo, hw != 0, readout,
                                   potentials != 0))
            need = std::max(need, spk::conv_pt_workspace(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo));
    return need;
}

extern "C" spk_status spk_conv_fire(const uint8_t *in_times, int B, int T, int Ci, int Hi, int Wi,
                                    const void *w, spk_dtype w_dtype, int Co, int Kh, int Kw,
                                    int stride, int pad, float theta, uint8_t *out_times,
                                    float *out_vkey, float *potentials, void *ws, size_t ws_bytes,
                                    spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(in_times && w && out_times && out_vkey, SPK_E_ARG, "spk_conv_fire: NULL pointer");
    SPK_REQUIRE(B > 0 && Ci > 0 && Hi > 0 && Wi > 0 && Co > 0 && Kh > 0 && Kw > 0 && stride > 0 &&
                    pad >= 0,
                SPK_E_ARG, "spk_conv_fire: sizes must be positive (pad >= 0)");
    SPK_REQUIRE(w_dtype == SPK_F32 || w_dtype == SPK_F16, SPK_E_UNSUPPORTED,
                "spk_conv_fire: unsupported weight dtype %d", (int)w_dtype);
    SPK_REQUIRE(T >= 1 && T <= SPK_MAX_T, SPK_E_SHAPE, "spk_conv_fire: T=%d not in [1, %d]", T,
                SPK_MAX_T);
    SPK_REQUIRE(theta == theta, SPK_E_ARG, "spk_conv_fire: theta is NaN");
    const int Ho = spk_out_extent(Hi, Kh, stride, pad), Wo = spk_out_extent(Wi, Kw, stride, pad);
    SPK_REQUIRE(Ho > 0 && Wo > 0, SPK_E_SHAPE, "spk_conv_fire: no output for %dx%d, kernel %dx%d",
                Hi, Wi, Kh, Kw);
    const long long taps = (long long)Ci * Kh * Kw;
    SPK_REQUIRE(taps <= kMaxTaps, SPK_E_SHAPE, "spk_conv_fire: Ci*Kh*Kw=%lld > %d", taps, kMaxTaps);
    SPK_REQUIRE(Co <= 65535 && B <= 65535, SPK_E_SHAPE, "spk_conv_fire: Co or B > 65535");
    const bool half_w = w_dtype == SPK_F16;
    const bool readout = is_readout(theta, potentials != nullptr);
    const size_t need = spk_conv_fire_workspace_size(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, theta,
                                                     potentials != nullptr);
    SPK_REQUIRE(ws_bytes >= need && (need == 0 || ws), SPK_E_WORKSPACE,
                "spk_conv_fire: workspace of %zu bytes needed, %zu given", need, ws_bytes);
    SPK_REQUIRE_WS_ALIGNED(ws, "spk_conv_fire");
    SPK_REQUIRE((long long)B * Ho * Wo < (1LL << 31) && (long long)Ci * Hi * Wi < (1LL << 31),
                SPK_E_SHAPE, "spk_conv_fire: layer too large");
    if (spk::conv_pt_supported(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo, half_w, readout,
                               potentials != nullptr))
        return spk::conv_fire_pt(in_times, B, T, Ci, Hi, Wi, w, half_w, Co, Kh, Kw, stride, pad, Ho, Wo,
                                 theta, out_times, out_vkey, ws, spk::stream_of(stream));
    if (spk::conv_fast_supported(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo, half_w, readout,
                                 potentials != nullptr))
        return spk::conv_fire_fast(in_times, B, T, Ci, Hi, Wi, w, half_w, Co, Kh, Kw, stride, pad, Ho,
                                   Wo, theta, out_times, out_vkey, ws, spk::stream_of(stream));
    if (readout && spk::readout_fast_supported(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo))
        return spk::readout_fast(in_times, B, T, Ci, Hi, Wi, w, half_w, Co, Kh, Kw, stride, pad, Ho,
                                 Wo, out_times, out_vkey, ws, spk::stream_of(stream));
    if (spk::conv_mfma_supported(Ci, Kh, Kw, Co, half_w, readout))
        return spk::conv_fire_mfma(in_times, B, T, Ci, Hi, Wi, w, half_w, Co, Kh, Kw, stride, pad, Ho,
                                   Wo, theta, out_times, out_vkey, potentials, ws,
                                   spk::stream_of(stream));
    ConvGeom g{B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo};
    dim3 grid(spk::ceil_div((long long)Ho * Wo, kThreads), Co, B);
    size_t lds = (size_t)taps * sizeof(float);
    hipStream_t s = spk::stream_of(stream);
    if (w_dtype == SPK_F16)
        hipLaunchKernelGGL(k_conv_fire_direct<true>, grid, dim3(kThreads), lds, s, in_times, w, g,
                           theta, out_times, out_vkey, potentials);
    else
        hipLaunchKernelGGL(k_conv_fire_direct<false>, grid, dim3(kThreads), lds, s, in_times, w, g,
                           theta, out_times, out_vkey, potentials);
    SPK_LAUNCHED("spk_conv_fire");
    return SPK_OK;
}
