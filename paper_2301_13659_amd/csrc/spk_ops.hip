// The steps around the hot path in Spyker's example network (§II-C.3 and the
// usage listings of §IV): the LoG filter bank, thresholding, weight
// quantization and gathering spike outputs into feature values.
#include <cmath>

#include "spk_internal.h"

namespace {

constexpr int kThreads = 256;

__global__ void k_threshold(float *__restrict__ x, int64_t n, float threshold, float value)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const float v = x[i];
        x[i] = v > threshold ? v : value;
    }
}

// Weights below mid become lower, the rest upper; the half copy follows.
__global__ void k_quantize(float *__restrict__ w, uint16_t *__restrict__ w16, int64_t n, float lower,
                           float mid, float upper)
{
    const _Float16 hl = (_Float16)lower, hu = (_Float16)upper;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const bool lo = w[i] < mid;
        w[i] = lo ? lower : upper;
        if (w16) w16[i] = __builtin_bit_cast(uint16_t, lo ? hl : hu);
    }
}

// Number of steps at which a neuron's cumulative frame is on: T - t for a
// neuron that fired at t < T, else 0.
__global__ void k_gather(const uint8_t *__restrict__ times, int64_t n, int T, float *__restrict__ out)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int t = times[i];
        out[i] = t < T ? (float)(T - t) : 0.0f;
    }
}

unsigned grid_for(int64_t n) { return (unsigned)std::min<int64_t>(4096, (n + kThreads - 1) / kThreads); }

}  // namespace

extern "C" spk_status spk_log_filter(const uint8_t *img, int B, int C, int H, int W, const float *stds,
                                     int n_std, int ksize, int pad, float *out, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(img && stds && out, SPK_E_ARG, "spk_log_filter: NULL pointer");
    SPK_REQUIRE(n_std > 0, SPK_E_ARG, "spk_log_filter: n_std=%d must be positive", n_std);
    SPK_REQUIRE(2 * n_std <= 8, SPK_E_SHAPE, "spk_log_filter: %d deviations give more than 8 filters",
                n_std);
    spk_dog_desc d[8];
    for (int i = 0; i < n_std; i++) {
        SPK_REQUIRE(stds[i] > 0.0f && std::isfinite(stds[i]), SPK_E_ARG,
                    "spk_log_filter: deviation %d must be positive", i);
        const double s = stds[i], a = s / std::sqrt(2.0), b = s * std::sqrt(2.0);
        d[2 * i] = spk_dog_desc{ksize, (float)a, (float)b};      // on-centre
        d[2 * i + 1] = spk_dog_desc{ksize, (float)b, (float)a};  // off-centre
    }
    const spk_status st = spk_dog_filter(img, B, C, H, W, d, 2 * n_std, pad, out, stream);
    if (st != SPK_OK) return st;
    return SPK_OK;
}

extern "C" spk_status spk_threshold(float *x, int64_t n, float threshold, float value, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(x || n == 0, SPK_E_ARG, "spk_threshold: NULL pointer");
    SPK_REQUIRE(n >= 0, SPK_E_ARG, "spk_threshold: n=%lld", (long long)n);
    SPK_REQUIRE(!std::isnan(threshold), SPK_E_ARG, "spk_threshold: threshold is NaN");
    if (n == 0) return SPK_OK;
    hipLaunchKernelGGL(k_threshold, dim3(grid_for(n)), dim3(kThreads), 0, spk::stream_of(stream), x, n,
                       threshold, value);
    SPK_LAUNCHED("spk_threshold");
    return SPK_OK;
}

extern "C" spk_status spk_quantize(float *w, uint16_t *w_f16, int64_t n, float lower, float mid,
                                   float upper, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(w || n == 0, SPK_E_ARG, "spk_quantize: NULL pointer");
    SPK_REQUIRE(n >= 0, SPK_E_ARG, "spk_quantize: n=%lld", (long long)n);
    SPK_REQUIRE(!std::isnan(mid), SPK_E_ARG, "spk_quantize: mid is NaN");
    if (n == 0) return SPK_OK;
    hipLaunchKernelGGL(k_quantize, dim3(grid_for(n)), dim3(kThreads), 0, spk::stream_of(stream), w,
                       w_f16, n, lower, mid, upper);
    SPK_LAUNCHED("spk_quantize");
    return SPK_OK;
}

extern "C" spk_status spk_gather(const uint8_t *times, int64_t n, int T, float *out, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE((times && out) || n == 0, SPK_E_ARG, "spk_gather: NULL pointer");
    SPK_REQUIRE(n >= 0, SPK_E_ARG, "spk_gather: n=%lld", (long long)n);
    SPK_REQUIRE(T >= 1 && T <= SPK_MAX_T, SPK_E_SHAPE, "spk_gather: T=%d not in [1, %d]", T, SPK_MAX_T);
    if (n == 0) return SPK_OK;
    hipLaunchKernelGGL(k_gather, dim3(grid_for(n)), dim3(kThreads), 0, spk::stream_of(stream), times, n,
                       T, out);
    SPK_LAUNCHED("spk_gather");
    return SPK_OK;
}
