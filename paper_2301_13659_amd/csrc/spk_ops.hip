// The steps around the hot path in Spyker's example network (§II-C.3 and the
// usage listings of §IV): the LoG filter bank, thresholding, weight
// quantization and gathering spike outputs into feature values; and the fire
// step on its own, over dense potentials (§II-E with the firing rule of
// §II-D.3).
#include <cmath>

#include "spk_internal.h"

namespace {

constexpr int kThreads = 256;
typedef float nf4 __attribute__((ext_vector_type(4)));

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

// Fire over dense potentials B x T x n: four neurons per thread, one 16-byte
// load per step; the first step with V > theta and the potential there, or
// NEVER and V[T-1].  Every step is read (a streaming pass over HBM).
__global__ void k_fire4(const float *__restrict__ V, int B, int T, int64_t n, float theta,
                        uint8_t *__restrict__ out_t, float *__restrict__ out_v)
{
    const int64_t n4 = n / 4;
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // over B * n4
    if (q >= (int64_t)B * n4) return;
    const int64_t b = q / n4, i = (q - b * n4) * 4;
    const float *src = V + (size_t)b * T * n + i;
    uint32_t tf[4] = {spk::kNever, spk::kNever, spk::kNever, spk::kNever};
    float vk[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    float4 last = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (int t0 = 0; t0 < T; t0 += 6) {
        float4 v[6];
#pragma unroll
        for (int u = 0; u < 6; u++)
            if (t0 + u < T)  // read once: streaming (non-temporal) loads
                v[u] = __builtin_bit_cast(float4, __builtin_nontemporal_load(
                                                      reinterpret_cast<const nf4 *>(src + (size_t)(t0 + u) * n)));
#pragma unroll
        for (int u = 0; u < 6; u++) {
            if (t0 + u < T) {
                const float e[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
                for (int k = 0; k < 4; k++) {
                    const bool f = tf[k] == (uint32_t)spk::kNever && e[k] > theta;
                    tf[k] = f ? (uint32_t)(t0 + u) : tf[k];
                    vk[k] = f ? e[k] : vk[k];
                }
                last = v[u];
            }
        }
    }
    const float l[4] = {last.x, last.y, last.z, last.w};
    uint32_t packed = 0;
#pragma unroll
    for (int k = 0; k < 4; k++) {
        vk[k] = tf[k] == (uint32_t)spk::kNever ? l[k] : vk[k];
        packed |= tf[k] << (8 * k);
    }
    *reinterpret_cast<uint32_t *>(out_t + (size_t)b * n + i) = packed;
    *reinterpret_cast<float4 *>(out_v + (size_t)b * n + i) = make_float4(vk[0], vk[1], vk[2], vk[3]);
}

// One neuron per thread (n not a multiple of 4, or unaligned arrays).
__global__ void k_fire1(const float *__restrict__ V, int B, int T, int64_t n, float theta,
                        uint8_t *__restrict__ out_t, float *__restrict__ out_v)
{
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= (int64_t)B * n) return;
    const int64_t b = q / n, i = q - b * n;
    const float *src = V + (size_t)b * T * n + i;
    uint32_t tf = spk::kNever;
    float vk = 0.0f, last = 0.0f;
    for (int t = 0; t < T; t++) {
        const float e = src[(size_t)t * n];
        const bool f = tf == (uint32_t)spk::kNever && e > theta;
        tf = f ? (uint32_t)t : tf;
        vk = f ? e : vk;
        last = e;
    }
    out_t[q] = (uint8_t)tf;
    out_v[q] = tf == (uint32_t)spk::kNever ? last : vk;
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

extern "C" spk_status spk_fire(const float *potentials, int B, int T, int64_t n, float theta,
                               uint8_t *out_times, float *out_vkey, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(potentials && out_times && out_vkey, SPK_E_ARG, "spk_fire: NULL pointer");
    SPK_REQUIRE(B > 0 && n > 0, SPK_E_ARG, "spk_fire: sizes must be positive");
    SPK_REQUIRE(T >= 1 && T <= SPK_MAX_T, SPK_E_SHAPE, "spk_fire: T=%d not in [1, %d]", T, SPK_MAX_T);
    SPK_REQUIRE(!std::isnan(theta), SPK_E_ARG, "spk_fire: theta is NaN");
    hipStream_t s = spk::stream_of(stream);
    const bool vec = n % 4 == 0 && (uintptr_t)potentials % 16 == 0 && (uintptr_t)out_vkey % 16 == 0 &&
                     (uintptr_t)out_times % 4 == 0;
    const int64_t work = vec ? (int64_t)B * (n / 4) : (int64_t)B * n;
    const unsigned blocks = (unsigned)((work + kThreads - 1) / kThreads);
    if (vec)
        hipLaunchKernelGGL(k_fire4, dim3(blocks), dim3(kThreads), 0, s, potentials, B, T, n, theta, out_times,
                           out_vkey);
    else
        hipLaunchKernelGGL(k_fire1, dim3(blocks), dim3(kThreads), 0, s, potentials, B, T, n, theta, out_times,
                           out_vkey);
    SPK_LAUNCHED("spk_fire");
    return SPK_OK;
}
