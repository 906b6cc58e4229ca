// libspk core: error reporting, shape rule, and the small element-wise calls
// (frames <-> first-spike times, the half cast, the R-STDP selector).
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include <hip/hip_fp16.h>

#include "spk_internal.h"

namespace spk {

static thread_local char g_error[512];

void clear_error() { g_error[0] = '\0'; }

void set_error(const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_error, sizeof(g_error), fmt, ap);
    va_end(ap);
}

spk_status check_launch(const char *what)
{
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        set_error("%s: kernel launch failed: %s", what, hipGetErrorString(e));
        return SPK_E_HIP;
    }
    return SPK_OK;
}

}  // namespace spk

// ---------------------------------------------------------------- kernels

// One thread per (sample, neuron); a neuron's time is its first on frame.
__global__ void k_frames_to_times(const uint8_t *__restrict__ frames, int B, int T, int64_t n,
                                  uint8_t *__restrict__ times)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)B * n) return;
    int64_t b = i / n, j = i - b * n;
    const uint8_t *f = frames + b * T * n + j;
    uint8_t t_first = spk::kNever;
    for (int t = 0; t < T; t++)
        if (f[(int64_t)t * n]) { t_first = (uint8_t)t; break; }
    times[i] = t_first;
}

// One thread per (sample, frame, neuron).
__global__ void k_times_to_frames(const uint8_t *__restrict__ times, int B, int T, int64_t n,
                                  uint8_t *__restrict__ frames)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // over B * T * n
    if (i >= (int64_t)B * T * n) return;
    int64_t per = (int64_t)T * n;
    int64_t b = i / per, r = i - b * per;
    int64_t t = r / n, j = r - t * n;
    frames[i] = (uint8_t)(times[b * n + j] <= t);
}

__global__ void k_cast_f16(const float *__restrict__ x, uint16_t *__restrict__ y, int64_t n)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    __half h = __float2half_rn(x[i]);
    y[i] = *reinterpret_cast<uint16_t *>(&h);
}

__global__ void k_rstdp_select(const spk_winner *__restrict__ win, const int32_t *__restrict__ nw,
                               int B, int k, const int32_t *__restrict__ labels, int group,
                               int32_t *__restrict__ cfg)
{
    int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= B * k) return;
    int b = i / k, s = i - b * k;
    int q = 1;
    if (s < nw[b] && win[i].c >= 0 && win[i].c / group == labels[b]) q = 0;
    cfg[i] = q;
}

// ---------------------------------------------------------------- ABI

extern "C" const char *spk_version(void) { return "spk 0.1 gfx950"; }

extern "C" const char *spk_last_error(void) { return spk::g_error; }

extern "C" int spk_out_extent(int in, int k, int stride, int pad)
{
    if (in < 1 || k < 1 || stride < 1 || pad < 0) return -1;
    long long span = (long long)in + 2LL * pad - k;
    if (span < 0) return -1;
    return (int)(span / stride + 1);
}

extern "C" spk_status spk_frames_to_times(const uint8_t *frames, int B, int T, int64_t n,
                                          uint8_t *times, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(frames && times, SPK_E_ARG, "spk_frames_to_times: NULL pointer");
    SPK_REQUIRE(B > 0 && n > 0, SPK_E_ARG, "spk_frames_to_times: B=%d n=%lld", B, (long long)n);
    SPK_REQUIRE(T >= 1 && T <= SPK_MAX_T, SPK_E_SHAPE, "spk_frames_to_times: T=%d not in [1, %d]",
                T, SPK_MAX_T);
    int64_t total = (int64_t)B * n;
    hipLaunchKernelGGL(k_frames_to_times, dim3(spk::ceil_div(total, 256)), dim3(256), 0,
                       spk::stream_of(stream), frames, B, T, n, times);
    SPK_LAUNCHED("spk_frames_to_times");
    return SPK_OK;
}

extern "C" spk_status spk_times_to_frames(const uint8_t *times, int B, int T, int64_t n,
                                          uint8_t *frames, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(frames && times, SPK_E_ARG, "spk_times_to_frames: NULL pointer");
    SPK_REQUIRE(B > 0 && n > 0, SPK_E_ARG, "spk_times_to_frames: B=%d n=%lld", B, (long long)n);
    SPK_REQUIRE(T >= 1 && T <= SPK_MAX_T, SPK_E_SHAPE, "spk_times_to_frames: T=%d not in [1, %d]",
                T, SPK_MAX_T);
    int64_t total = (int64_t)B * T * n;
    hipLaunchKernelGGL(k_times_to_frames, dim3(spk::ceil_div(total, 256)), dim3(256), 0,
                       spk::stream_of(stream), times, B, T, n, frames);
    SPK_LAUNCHED("spk_times_to_frames");
    return SPK_OK;
}

extern "C" spk_status spk_cast_f16(const float *x, uint16_t *y, int64_t n, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(x && y, SPK_E_ARG, "spk_cast_f16: NULL pointer");
    SPK_REQUIRE(n > 0, SPK_E_ARG, "spk_cast_f16: n=%lld", (long long)n);
    hipLaunchKernelGGL(k_cast_f16, dim3(spk::ceil_div(n, 256)), dim3(256), 0,
                       spk::stream_of(stream), x, y, n);
    SPK_LAUNCHED("spk_cast_f16");
    return SPK_OK;
}

extern "C" spk_status spk_rstdp_select(const spk_winner *winners, const int32_t *n_winners, int B,
                                       int k, const int32_t *labels, int group,
                                       int32_t *winner_cfg, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(winners && n_winners && labels && winner_cfg, SPK_E_ARG,
                "spk_rstdp_select: NULL pointer");
    SPK_REQUIRE(B > 0 && k > 0 && group > 0, SPK_E_ARG, "spk_rstdp_select: B=%d k=%d group=%d",
                B, k, group);
    hipLaunchKernelGGL(k_rstdp_select, dim3(spk::ceil_div((long long)B * k, 256)), dim3(256), 0,
                       spk::stream_of(stream), winners, n_winners, B, k, labels, group, winner_cfg);
    SPK_LAUNCHED("spk_rstdp_select");
    return SPK_OK;
}
