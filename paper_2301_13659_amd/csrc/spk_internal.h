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

// Max-pooling read by a convolution's packing pass (spk_pool_conv_fire): the
// layer input cell (iy, ix) of a channel plane is the earliest time of its
// kh x kw window of src (§II-E.3); window cells in the padding never fire.
struct PoolIn {
    const uint8_t *src;  // B x C x H0 x W0 time map
    uint8_t *pooled;     // nullable: the pooled map B x C x Hi x Wi is also written here
    int H0, W0, kh, kw, stride, pad;
    long long bytes;     // B * C * H0 * W0: the extent of src
    int stage;           // set by the packing pass: LDS byte offset of pool_row's staging, or
                         // -1 when the rows do not fit and cells are pooled one by one
};

// Dwords pool_row stages per channel (the window rows of one input row, kh
// rows of W0 bytes, from a dword boundary), and its LDS bytes for C channels.
__host__ __device__ inline int pool_stage_words(const PoolIn &p) { return (p.kh * p.W0 + 3) / 4 + 1; }
inline size_t pool_stage_bytes(const PoolIn &p, int C) { return (size_t)C * pool_stage_words(p) * 4; }

// Input row iy (Wi cells) of the C channel planes plane0.. pooled, by the
// whole block: the window rows of every channel are copied to LDS at `st`
// (dword loads, all of a thread's in flight; bytes near the end of src are
// read one by one so nothing past it is touched), then each cell takes the
// minimum of its window there.  put(c, x, time) receives each cell once, and
// the cell also goes to p.pooled when that is set.
template <typename Put>
__device__ __forceinline__ void pool_row(const PoolIn &p, long long plane0, int C, int Hi, int Wi,
                                         int iy, uint32_t *st, Put put)
{
    const int SW = pool_stage_words(p);
    const int y0 = iy * p.stride - p.pad;
    const int ylo = max(y0, 0), nr = max(0, min(y0 + p.kh, p.H0) - ylo);  // window rows in the map
    const long long plane_b = (long long)p.H0 * p.W0;
    const long long last_full = p.bytes / 4;  // dwords [0, last_full) lie wholly inside src
    const int n = C * SW;
    constexpr int kIn = 16;
    for (int f0 = threadIdx.x; f0 < n; f0 += kIn * (int)blockDim.x) {
        uint32_t v[kIn];
#pragma unroll
        for (int u = 0; u < kIn; u++) {
            const int f = f0 + u * (int)blockDim.x;
            const int c = f / SW, i = f - c * SW;
            const long long d = (((plane0 + c) * plane_b + (long long)ylo * p.W0) >> 2) + i;
            v[u] = 0u;
            if (f < n) {
                if (d < last_full) {
                    v[u] = reinterpret_cast<const uint32_t *>(p.src)[d];
                } else {
                    for (int k = 0; k < 4; k++)
                        if (4 * d + k < p.bytes) v[u] |= (uint32_t)p.src[4 * d + k] << (8 * k);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kIn; u++)
            if (f0 + u * (int)blockDim.x < n) st[f0 + u * (int)blockDim.x] = v[u];
    }
    __syncthreads();
    const uint8_t *sb = reinterpret_cast<const uint8_t *>(st);
    for (int e = threadIdx.x; e < C * Wi; e += blockDim.x) {
        const int c = e / Wi, x = e - c * Wi;
        const int lead = (int)(((plane0 + c) * plane_b + (long long)ylo * p.W0) & 3);
        const uint8_t *rows = sb + (size_t)c * SW * 4 + lead;
        const int x0 = x * p.stride - p.pad;
        const int xlo = max(x0, 0), xhi = min(x0 + p.kw, p.W0);
        uint32_t m = (uint32_t)kNever;
        for (int r = 0; r < nr; r++)
            for (int xx = xlo; xx < xhi; xx++) m = min(m, (uint32_t)rows[r * p.W0 + xx]);
        if (p.pooled) p.pooled[((plane0 + c) * Hi + iy) * Wi + x] = (uint8_t)m;
        put(c, x, (uint8_t)m);
    }
}

// Pooled time of input cell (iy, ix) of channel plane `plane` (b*C + c),
// read from global memory (for rows too wide to stage).
__device__ __forceinline__ uint32_t pool_cell(const PoolIn &p, long long plane, int iy, int ix)
{
    const uint8_t *s = p.src + plane * p.H0 * p.W0;
    const int y0 = iy * p.stride - p.pad, x0 = ix * p.stride - p.pad;
    const int ylo = max(y0, 0), yhi = min(y0 + p.kh, p.H0);
    const int xlo = max(x0, 0), xhi = min(x0 + p.kw, p.W0);
    uint32_t m = (uint32_t)kNever;
    for (int y = ylo; y < yhi; y++) {
        const uint8_t *row = s + (long long)y * p.W0;
        for (int x = xlo; x < xhi; x++) m = min(m, (uint32_t)row[x]);
    }
    return m;
}

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
// pool: nullable; when given, `in` is ignored and the input is pooled from
// pool->src in the packing pass.
spk_status conv_fire_pt(const uint8_t *in, int B, int T, int Ci, int Hi, int Wi, const void *w,
                        bool half_w, int Co, int Kh, int Kw, int stride, int pad, int Ho, int Wo,
                        float theta, uint8_t *out_t, float *out_v, void *ws, hipStream_t s,
                        const PoolIn *pool = nullptr);
// Readout layers (theta = +inf, no dense potentials): the split-K GEMM of the
// last frame on the same channels-last copy (spk_conv_fast.hip).  packed_w:
// nullable B fragments from spk_conv_pack_weights, used instead of packing w;
// pool as for conv_fire_pt.
bool readout_fast_supported(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw,
                            int stride, int pad, int Ho, int Wo);
size_t readout_fast_workspace(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw,
                              int stride, int pad, int Ho, int Wo);
spk_status readout_fast(const uint8_t *in, int B, int T, int Ci, int Hi, int Wi, const void *w,
                        bool half_w, int Co, int Kh, int Kw, int stride, int pad, int Ho, int Wo,
                        uint8_t *out_t, float *out_v, void *ws, hipStream_t s,
                        const void *packed_w = nullptr, const PoolIn *pool = nullptr);
// Bytes of the readout B fragments of a Co x Ci x Kh x Kw weight tensor, and
// the packing pass that writes them (spk_conv_fast.hip).
size_t readout_packed_bytes(int Co, int Ci, int Kh, int Kw, bool half_w);
spk_status readout_pack_weights(const void *w, bool half_w, int Co, int Ci, int Kh, int Kw,
                                void *packed, hipStream_t s);

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
