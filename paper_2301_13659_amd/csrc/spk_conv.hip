// spk_conv_fire: spiking convolution + integrate-and-fire (Spyker §II-E.1, Eq. 2).
//
// Dispatch, first match: firing layers with T <= 32 whose weights fit the
// registers of a wave take the time-batched matrix-core kernel of
// spk_conv_pt.hip; readout layers (theta = +inf) the split-K kernel of
// spk_conv_fast.hip; other firing layers without dense potentials the
// register-resident kernels of spk_conv_fast.hip; shapes the matrix-core
// kernels of spk_conv_mfma.hip cover (the dense-potential mode among them) go
// there; the rest take the direct form below: one thread per output neuron
// (b, o, y, x) walks the time steps, sums the weights of the inputs of its
// window that have fired by step t (the cumulative frame S_t = [time <= t])
// and records the first step whose potential exceeds theta.  Kernel o's
// weights are staged in LDS as float.
//
// spk_pool_conv_fire pools (§II-E.3) inside the packing pass of the first two
// paths, and with the spk_pool kernel in front of the others.
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

// Checks of a convolution call and the choice of its kernels.  pool: the
// input is pooled from pool->src (in is then not read); the packing passes of
// the channels-last paths pool as they pack, the other paths read a pooled map
// written first to pool->pooled or, when that is NULL, to pool_scratch.
static spk_status conv_run(const char *what, const uint8_t *in_times, int B, int T, int Ci, int Hi,
                           int Wi, const void *w, spk_dtype w_dtype, int Co, int Kh, int Kw,
                           int stride, int pad, float theta, uint8_t *out_times, float *out_vkey,
                           float *potentials, void *ws, size_t ws_bytes, spk_stream stream,
                           const void *packed_w, const spk::PoolIn *pool, uint8_t *pool_scratch)
{
    SPK_REQUIRE(in_times && w && out_times && out_vkey, SPK_E_ARG, "%s: NULL pointer", what);
    SPK_REQUIRE(B > 0 && Ci > 0 && Hi > 0 && Wi > 0 && Co > 0 && Kh > 0 && Kw > 0 && stride > 0 &&
                    pad >= 0,
                SPK_E_ARG, "%s: sizes must be positive (pad >= 0)", what);
    SPK_REQUIRE(w_dtype == SPK_F32 || w_dtype == SPK_F16, SPK_E_UNSUPPORTED,
                "%s: unsupported weight dtype %d", what, (int)w_dtype);
    SPK_REQUIRE(T >= 1 && T <= SPK_MAX_T, SPK_E_SHAPE, "%s: T=%d not in [1, %d]", what, T, SPK_MAX_T);
    SPK_REQUIRE(theta == theta, SPK_E_ARG, "%s: theta is NaN", what);
    const int Ho = spk_out_extent(Hi, Kh, stride, pad), Wo = spk_out_extent(Wi, Kw, stride, pad);
    SPK_REQUIRE(Ho > 0 && Wo > 0, SPK_E_SHAPE, "%s: no output for %dx%d, kernel %dx%d", what, Hi, Wi,
                Kh, Kw);
    const long long taps = (long long)Ci * Kh * Kw;
    SPK_REQUIRE(taps <= kMaxTaps, SPK_E_SHAPE, "%s: Ci*Kh*Kw=%lld > %d", what, taps, kMaxTaps);
    SPK_REQUIRE(Co <= 65535 && B <= 65535, SPK_E_SHAPE, "%s: Co or B > 65535", what);
    const bool half_w = w_dtype == SPK_F16;
    const bool readout = is_readout(theta, potentials != nullptr);
    const size_t need = spk_conv_fire_workspace_size(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, theta,
                                                     potentials != nullptr);
    SPK_REQUIRE(ws_bytes >= need && (need == 0 || ws), SPK_E_WORKSPACE,
                "%s: workspace of %zu bytes needed, %zu given", what, need, ws_bytes);
    SPK_REQUIRE_WS_ALIGNED(ws, what);
    SPK_REQUIRE((long long)B * Ho * Wo < (1LL << 31) && (long long)Ci * Hi * Wi < (1LL << 31),
                SPK_E_SHAPE, "%s: layer too large", what);
    hipStream_t s = spk::stream_of(stream);
    if (spk::conv_pt_supported(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo, half_w, readout,
                               potentials != nullptr))
        return spk::conv_fire_pt(in_times, B, T, Ci, Hi, Wi, w, half_w, Co, Kh, Kw, stride, pad, Ho, Wo,
                                 theta, out_times, out_vkey, ws, s, pool);
    if (readout && spk::readout_fast_supported(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo))
        return spk::readout_fast(in_times, B, T, Ci, Hi, Wi, w, half_w, Co, Kh, Kw, stride, pad, Ho,
                                 Wo, out_times, out_vkey, ws, s, packed_w, pool);
    if (pool) {
        uint8_t *pooled = pool->pooled ? pool->pooled : pool_scratch;
        const spk_status st = spk_pool(pool->src, B, Ci, pool->H0, pool->W0, pool->kh, pool->kw,
                                       pool->stride, pool->pad, pooled, stream);
        if (st != SPK_OK) return st;
        in_times = pooled;
    }
    if (spk::conv_fast_supported(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo, half_w, readout,
                                 potentials != nullptr))
        return spk::conv_fire_fast(in_times, B, T, Ci, Hi, Wi, w, half_w, Co, Kh, Kw, stride, pad, Ho,
                                   Wo, theta, out_times, out_vkey, ws, s);
    if (spk::conv_mfma_supported(Ci, Kh, Kw, Co, half_w, readout))
        return spk::conv_fire_mfma(in_times, B, T, Ci, Hi, Wi, w, half_w, Co, Kh, Kw, stride, pad, Ho,
                                   Wo, theta, out_times, out_vkey, potentials, ws, s);
    ConvGeom g{B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo};
    dim3 grid(spk::ceil_div((long long)Ho * Wo, kThreads), Co, B);
    size_t lds = (size_t)taps * sizeof(float);
    if (w_dtype == SPK_F16)
        hipLaunchKernelGGL(k_conv_fire_direct<true>, grid, dim3(kThreads), lds, s, in_times, w, g,
                           theta, out_times, out_vkey, potentials);
    else
        hipLaunchKernelGGL(k_conv_fire_direct<false>, grid, dim3(kThreads), lds, s, in_times, w, g,
                           theta, out_times, out_vkey, potentials);
    SPK_LAUNCHED(what);
    return SPK_OK;
}

extern "C" spk_status spk_conv_fire(const uint8_t *in_times, int B, int T, int Ci, int Hi, int Wi,
                                    const void *w, spk_dtype w_dtype, int Co, int Kh, int Kw,
                                    int stride, int pad, float theta, uint8_t *out_times,
                                    float *out_vkey, float *potentials, void *ws, size_t ws_bytes,
                                    spk_stream stream)
{
    spk::clear_error();
    return conv_run("spk_conv_fire", in_times, B, T, Ci, Hi, Wi, w, w_dtype, Co, Kh, Kw, stride, pad,
                    theta, out_times, out_vkey, potentials, ws, ws_bytes, stream, nullptr, nullptr,
                    nullptr);
}

extern "C" size_t spk_pool_conv_fire_workspace_size(int B, int T, int Ci, int H0, int W0, int pool_kh,
                                                    int pool_kw, int pool_stride, int pool_pad, int Co,
                                                    int Kh, int Kw, int stride, int pad, float theta)
{
    const int Hi = spk_out_extent(H0, pool_kh, pool_stride, pool_pad);
    const int Wi = spk_out_extent(W0, pool_kw, pool_stride, pool_pad);
    if (B <= 0 || Ci <= 0 || Hi <= 0 || Wi <= 0) return 0;
    const size_t conv = spk_conv_fire_workspace_size(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, theta, 0);
    // and room for the pooled map of the paths that do not pool as they pack
    return spk::align_up(conv, 256) + spk::align_up((size_t)B * Ci * Hi * Wi, 256);
}

extern "C" spk_status spk_pool_conv_fire(const uint8_t *in_times, int B, int T, int Ci, int H0, int W0,
                                         int pool_kh, int pool_kw, int pool_stride, int pool_pad,
                                         uint8_t *pooled_times, const void *w, spk_dtype w_dtype,
                                         const void *packed_w, int Co, int Kh, int Kw, int stride,
                                         int pad, float theta, uint8_t *out_times, float *out_vkey,
                                         void *ws, size_t ws_bytes, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(in_times, SPK_E_ARG, "spk_pool_conv_fire: NULL pointer");
    SPK_REQUIRE(B > 0 && Ci > 0 && H0 > 0 && W0 > 0 && pool_kh > 0 && pool_kw > 0 &&
                    pool_stride > 0 && pool_pad >= 0,
                SPK_E_ARG, "spk_pool_conv_fire: sizes must be positive (pad >= 0)");
    SPK_REQUIRE((long long)B * Ci * H0 * W0 < (1LL << 31), SPK_E_SHAPE,
                "spk_pool_conv_fire: input too large");
    const int Hi = spk_out_extent(H0, pool_kh, pool_stride, pool_pad);
    const int Wi = spk_out_extent(W0, pool_kw, pool_stride, pool_pad);
    SPK_REQUIRE(Hi > 0 && Wi > 0, SPK_E_SHAPE,
                "spk_pool_conv_fire: no pooled output for %dx%d, window %dx%d", H0, W0, pool_kh,
                pool_kw);
    SPK_REQUIRE(((uintptr_t)packed_w & 15u) == 0u, SPK_E_ARG,
                "spk_pool_conv_fire: packed_w not 16-byte aligned");
    const size_t need = spk_pool_conv_fire_workspace_size(B, T, Ci, H0, W0, pool_kh, pool_kw,
                                                          pool_stride, pool_pad, Co, Kh, Kw, stride,
                                                          pad, theta);
    SPK_REQUIRE(ws_bytes >= need && ws, SPK_E_WORKSPACE,
                "spk_pool_conv_fire: workspace of %zu bytes needed, %zu given", need, ws_bytes);
    const size_t conv_ws = need - spk::align_up((size_t)B * Ci * Hi * Wi, 256);
    const spk::PoolIn pool{in_times, pooled_times, H0,      W0,
                           pool_kh,  pool_kw,      pool_stride, pool_pad,
                           (long long)B * Ci * H0 * W0, -1};
    return conv_run("spk_pool_conv_fire", in_times, B, T, Ci, Hi, Wi, w, w_dtype, Co, Kh, Kw, stride,
                    pad, theta, out_times, out_vkey, nullptr, ws, conv_ws, stream, packed_w, &pool,
                    reinterpret_cast<uint8_t *>(ws) + conv_ws);
}

extern "C" size_t spk_conv_packed_weights_size(int Co, int Ci, int Kh, int Kw, spk_dtype w_dtype)
{
    if (Co <= 0 || Ci <= 0 || Kh <= 0 || Kw <= 0 || (w_dtype != SPK_F32 && w_dtype != SPK_F16))
        return 0;
    return spk::readout_packed_bytes(Co, Ci, Kh, Kw, w_dtype == SPK_F16);
}

extern "C" spk_status spk_conv_pack_weights(const void *w, spk_dtype w_dtype, int Co, int Ci, int Kh,
                                            int Kw, void *packed, size_t packed_bytes,
                                            spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(w && packed, SPK_E_ARG, "spk_conv_pack_weights: NULL pointer");
    SPK_REQUIRE(Co > 0 && Ci > 0 && Kh > 0 && Kw > 0, SPK_E_ARG,
                "spk_conv_pack_weights: sizes must be positive");
    SPK_REQUIRE(w_dtype == SPK_F32 || w_dtype == SPK_F16, SPK_E_UNSUPPORTED,
                "spk_conv_pack_weights: unsupported weight dtype %d", (int)w_dtype);
    SPK_REQUIRE((long long)Ci * Kh * Kw * 4 <= 64 * 1024 && Co <= 65535, SPK_E_SHAPE,
                "spk_conv_pack_weights: Ci*Kh*Kw=%lld taps or Co=%d too large",
                (long long)Ci * Kh * Kw, Co);
    SPK_REQUIRE(((uintptr_t)packed & 15u) == 0u, SPK_E_ARG,
                "spk_conv_pack_weights: packed not 16-byte aligned");
    const size_t need = spk_conv_packed_weights_size(Co, Ci, Kh, Kw, w_dtype);
    SPK_REQUIRE(packed_bytes >= need, SPK_E_WORKSPACE,
                "spk_conv_pack_weights: %zu bytes needed, %zu given", need, packed_bytes);
    return spk::readout_pack_weights(w, w_dtype == SPK_F16, Co, Ci, Kh, Kw, packed,
                                     spk::stream_of(stream));
}
