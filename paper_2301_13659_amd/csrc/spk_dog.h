// DoG filter bank pieces shared by spk_dog_filter and the fused DoG + rank
// coding call (Spyker §II-C.1, shape rule Eq. 1).  Internal to libspk.
#pragma once

#include <algorithm>
#include <cmath>

#include "spk_internal.h"

namespace spk {
namespace dog {

constexpr int kMaxF = 8;
constexpr int kMaxK = 21;
constexpr int kMaxCoef = 480;  // coefficients carried by one launch

// One launch's filters.  The coefficients travel by value in the kernel
// arguments; the kernels copy them to LDS.
struct DogParams {
    int nf;
    int lo, hi;            // input offsets spanned by the launch: [lo, hi] around an output
    int ks[kMaxF];         // kernel size
    int off[kMaxF];        // input offset of the first kernel tap (-padding)
    int cbase[kMaxF];      // first coefficient of each kernel in coef[]
    int fidx[kMaxF];       // output filter index f
    float coef[kMaxCoef];
};

// Unit-sum discrete Gaussian difference, double, rounded once to float.
inline void coefficients(int K, double s1, double s2, float *k)
{
    const int R = (K - 1) / 2;
    double g1[kMaxK * kMaxK], g2[kMaxK * kMaxK];
    double n1 = 0.0, n2 = 0.0;
    for (int i = -R; i <= R; i++)
        for (int j = -R; j <= R; j++) {
            const double r2 = (double)(i * i + j * j);
            const int at = (i + R) * K + (j + R);
            g1[at] = std::exp(-r2 / (2.0 * s1 * s1));
            g2[at] = std::exp(-r2 / (2.0 * s2 * s2));
            n1 += g1[at];
            n2 += g2[at];
        }
    for (int at = 0; at < K * K; at++) k[at] = (float)(g1[at] / n1 - g2[at] / n2);
}

// Checks the descriptors and gives the output extent (what names the
// calling entry point in the messages).
inline spk_status plan(const char *what, int B, int C, int H, int W, const spk_dog_desc *filters,
                       int F, int pad, int &Ho, int &Wo)
{
    SPK_REQUIRE(B > 0 && C > 0 && H > 0 && W > 0 && F > 0, SPK_E_ARG,
                "%s: B=%d C=%d H=%d W=%d F=%d must be positive", what, B, C, H, W, F);
    SPK_REQUIRE(F <= kMaxF, SPK_E_SHAPE, "%s: F=%d > %d", what, F, kMaxF);
    SPK_REQUIRE(pad >= -1, SPK_E_ARG, "%s: pad=%d (use -1 for same padding)", what, pad);
    for (int f = 0; f < F; f++) {
        const spk_dog_desc &d = filters[f];
        SPK_REQUIRE(d.ksize >= 1 && (d.ksize & 1), SPK_E_ARG,
                    "%s: filter %d ksize=%d must be odd and >= 1", what, f, d.ksize);
        SPK_REQUIRE(d.ksize <= kMaxK, SPK_E_SHAPE, "%s: filter %d ksize=%d > %d", what, f,
                    d.ksize, kMaxK);
        SPK_REQUIRE(d.sigma1 > 0.0 && d.sigma2 > 0.0, SPK_E_ARG,
                    "%s: filter %d sigmas must be positive", what, f);
        SPK_REQUIRE(pad < 0 || d.ksize == filters[0].ksize, SPK_E_UNSUPPORTED,
                    "%s: an explicit pad needs one kernel size for all filters", what);
    }
    Ho = pad < 0 ? H : H + 2 * pad - filters[0].ksize + 1;
    Wo = pad < 0 ? W : W + 2 * pad - filters[0].ksize + 1;
    SPK_REQUIRE(Ho > 0 && Wo > 0, SPK_E_SHAPE, "%s: output %dx%d is empty", what, Ho, Wo);
    return SPK_OK;
}

// Filters f0.. that fit one launch's coefficient block go into p; returns
// the first filter left over.
inline int group(const spk_dog_desc *filters, int F, int pad, int f0, DogParams &p)
{
    p = DogParams{};
    int used = 0, f = f0;
    p.lo = 1 << 30;
    p.hi = -(1 << 30);
    while (f < F && p.nf < kMaxF) {
        const int K = filters[f].ksize;
        if (used + K * K > kMaxCoef) break;
        const int P = pad < 0 ? (K - 1) / 2 : pad;
        p.ks[p.nf] = K;
        p.off[p.nf] = -P;
        p.cbase[p.nf] = used;
        p.fidx[p.nf] = f;
        coefficients(K, filters[f].sigma1, filters[f].sigma2, p.coef + used);
        p.lo = std::min(p.lo, -P);
        p.hi = std::max(p.hi, K - 1 - P);
        used += K * K;
        p.nf++;
        f++;
    }
    return f;
}

// One K x K window, fully unrolled: coefficients cf (LDS, broadcast reads)
// times the staged pixels from `tile` (row stride tw), summed in float in
// row-major order without contraction, so every caller gets the same bits.
template <int K>
__device__ __forceinline__ float window(const float *__restrict__ cf, const float *tile, int tw)
{
#pragma clang fp contract(off)
    float acc = 0.0f;
#pragma unroll
    for (int i = 0; i < K; i++)
#pragma unroll
        for (int j = 0; j < K; j++) {
            const float prod = cf[i * K + j] * tile[i * tw + j];
            acc = acc + prod;
        }
    return acc;
}

__device__ __forceinline__ float window_k(int K, const float *cf, const float *t0, int tw)
{
    switch (K) {
    case 1: return window<1>(cf, t0, tw);
    case 3: return window<3>(cf, t0, tw);
    case 5: return window<5>(cf, t0, tw);
    case 7: return window<7>(cf, t0, tw);
    case 9: return window<9>(cf, t0, tw);
    case 11: return window<11>(cf, t0, tw);
    case 13: return window<13>(cf, t0, tw);
    case 15: return window<15>(cf, t0, tw);
    case 17: return window<17>(cf, t0, tw);
    case 19: return window<19>(cf, t0, tw);
    default: return window<21>(cf, t0, tw);
    }
}

// R outputs of one row at once (output r's window starts at t0 + r), each
// summed exactly as window<K> sums it (same products, same row-major order,
// no contraction): a kernel row's K + R - 1 pixels and K coefficients are read
// once for the R outputs.
template <int K, int R>
__device__ __forceinline__ void window_run(const float *__restrict__ cf, const float *t0, int tw,
                                           float (&acc)[R])
{
#pragma clang fp contract(off)
#pragma unroll
    for (int r = 0; r < R; r++) acc[r] = 0.0f;
#pragma unroll
    for (int i = 0; i < K; i++) {
        float px[K + R - 1], c[K];
#pragma unroll
        for (int q = 0; q < K + R - 1; q++) px[q] = t0[i * tw + q];
#pragma unroll
        for (int j = 0; j < K; j++) c[j] = cf[i * K + j];
#pragma unroll
        for (int j = 0; j < K; j++)
#pragma unroll
            for (int r = 0; r < R; r++) {
                const float prod = c[j] * px[r + j];
                acc[r] = acc[r] + prod;
            }
    }
}

template <int R>
__device__ __forceinline__ void window_run_k(int K, const float *cf, const float *t0, int tw, float (&acc)[R])
{
    switch (K) {
    case 1: window_run<1, R>(cf, t0, tw, acc); break;
    case 3: window_run<3, R>(cf, t0, tw, acc); break;
    case 5: window_run<5, R>(cf, t0, tw, acc); break;
    case 7: window_run<7, R>(cf, t0, tw, acc); break;
    case 9: window_run<9, R>(cf, t0, tw, acc); break;
    case 11: window_run<11, R>(cf, t0, tw, acc); break;
    case 13: window_run<13, R>(cf, t0, tw, acc); break;
    case 15: window_run<15, R>(cf, t0, tw, acc); break;
    case 17: window_run<17, R>(cf, t0, tw, acc); break;
    case 19: window_run<19, R>(cf, t0, tw, acc); break;
    default: window_run<21, R>(cf, t0, tw, acc); break;
    }
}

// A staged pixel: u / 255 inside the image, 0 in the padding.
__device__ __forceinline__ float pixel(const uint8_t *src, int H, int W, int iy, int ix)
{
    const bool inside = (unsigned)iy < (unsigned)H && (unsigned)ix < (unsigned)W;
    const float u = (float)src[inside ? (size_t)iy * W + ix : 0];
    return inside ? u / 255.0f : 0.0f;
}

}  // namespace dog
}  // namespace spk
