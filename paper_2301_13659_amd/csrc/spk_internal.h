// Internal helpers of libspk (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "spk.h"

namespace spk {

constexpr int kNever = SPK_NEVER;

void clear_error();
void set_error(const char *fmt, ...) __attribute__((format(printf, 1, 2)));

// Report the first launch failure of a call as SPK_E_HIP.
spk_status check_launch(const char *what);

inline hipStream_t stream_of(spk_stream s) { return reinterpret_cast<hipStream_t>(s); }

inline size_t align_up(size_t n, size_t a) { return (n + a - 1) / a * a; }

inline int ceil_div(long long a, long long b) { return (int)((a + b - 1) / b); }

// Matrix-core spiking convolution (spk_conv_mfma.hip).  A readout call is a
// call with theta = +inf and no dense potentials.
bool conv_mfma_supported(int Ci, int Kh, int Kw, int Co, bool half_w, bool readout);
size_t conv_mfma_workspace(int B, int Ho, int Wo, int Co, int K, bool readout);
spk_status conv_fire_mfma(const uint8_t *in, int B, int T, int Ci, int Hi, int Wi, const void *w,
                          bool half_w, int Co, int Kh, int Kw, int stride, int pad, int Ho, int Wo,
                          float theta, uint8_t *out_t, float *out_v, float *pot, void *ws,
                          hipStream_t s);

// Register-resident firing kernels on a channels-last copy of the input
// (spk_conv_fast.hip): firing layers without the dense potentials.
bool conv_fast_supported(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride,
                         int pad, int Ho, int Wo, bool half_w, bool readout, bool potentials);
size_t conv_fast_workspace(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride,
                           int pad, int Ho, int Wo);
spk_status conv_fire_fast(const uint8_t *in, int B, int T, int Ci, int Hi, int Wi, const void *w,
                          bool half_w, int Co, int Kh, int Kw, int stride, int pad, int Ho, int Wo,
                          float theta, uint8_t *out_t, float *out_v, void *ws, hipStream_t s);
// Firing layers with T <= 32 whose weights fit a wave's registers: every
// step of a tile in one matrix-core product (spk_conv_pt.hip).
bool conv_pt_supported(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride,
                       int pad, int Ho, int Wo, bool half_w, bool readout, bool potentials);
size_t conv_pt_workspace(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride,
                         int pad, int Ho, int Wo);
spk_status conv_fire_pt(const uint8_t *in, int B, int T, int Ci, int Hi, int Wi, const void *w,
                        bool half_w, int Co, int Kh, int Kw, int stride, int pad, int Ho, int Wo,
                        float theta, uint8_t *out_t, float *out_v, void *ws, hipStream_t s);
// Readout layers (theta = +inf, no dense potentials): the split-K GEMM of the
// last frame on the same channels-last copy (spk_conv_fast.hip).
bool readout_fast_supported(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw,
                            int stride, int pad, int Ho, int Wo);
size_t readout_fast_workspace(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw,
                              int stride, int pad, int Ho, int Wo);
spk_status readout_fast(const uint8_t *in, int B, int T, int Ci, int Hi, int Wi, const void *w,
                        bool half_w, int Co, int Kh, int Kw, int stride, int pad, int Ho, int Wo,
                        uint8_t *out_t, float *out_v, void *ws, hipStream_t s);

}  // namespace spk

#define SPK_REQUIRE(cond, code, ...)        \
    do {                                    \
        if (!(cond)) {                      \
            spk::set_error(__VA_ARGS__);    \
            return (code);                  \
        }                                   \
    } while (0)

// Workspaces hold 16-byte vectors and the sources of direct-to-LDS loads:
// they must be 256-byte aligned (hipMalloc and torch allocations are).
#define SPK_REQUIRE_WS_ALIGNED(ws, what)                                                     \
    SPK_REQUIRE(((uintptr_t)(ws) & 255u) == 0u, SPK_E_ARG, "%s: workspace not 256-byte aligned", \
                what)

#define SPK_LAUNCHED(what)                                  \
    do {                                                    \
        spk_status st_ = spk::check_launch(what);           \
        if (st_ != SPK_OK) return st_;                      \
    } while (0)
