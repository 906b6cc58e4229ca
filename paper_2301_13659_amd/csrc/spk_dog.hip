// spk_dog_filter: DoG feature enhancement (Spyker §II-C.1, shape rule Eq. 1).
//
// The filter bank is tiny (at most 8 kernels, K <= 21), so its coefficients
// are computed on the host and travel by value in the kernel arguments, where
// every lane reads them as uniform scalar loads.  A block evaluates one filter
// on a 32 x 8 output tile: it stages the scaled input pixels (u / 255) of the
// tile and its halo in LDS, then runs the fully unrolled window of that
// kernel size.  Accumulation is float, window row-major,
// no contraction, so every output is reproducible bit for bit (the rank-order
// coder downstream turns last-bit differences into different spike times).
#include <cmath>

#include "spk_internal.h"

namespace {

constexpr int kMaxF = 8;
constexpr int kMaxK = 21;
constexpr int kMaxCoef = 480;  // coefficients carried by one launch
constexpr int kTX = 32, kTY = 8;
constexpr int kMaxSpan = kMaxK - 1;

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
void dog_coefficients(int K, double s1, double s2, float *k)
{
    int R = (K - 1) / 2;
    double g1[kMaxK * kMaxK], g2[kMaxK * kMaxK];
    double n1 = 0.0, n2 = 0.0;
    for (int i = -R; i <= R; i++)
        for (int j = -R; j <= R; j++) {
            double r2 = (double)(i * i + j * j);
            int at = (i + R) * K + (j + R);
            g1[at] = std::exp(-r2 / (2.0 * s1 * s1));
            g2[at] = std::exp(-r2 / (2.0 * s2 * s2));
            n1 += g1[at];
            n2 += g2[at];
        }
    for (int at = 0; at < K * K; at++) k[at] = (float)(g1[at] / n1 - g2[at] / n2);
}

// One K x K window, fully unrolled, coefficients and pixels from LDS (the
// coefficient reads are broadcasts); the sum keeps the row-major order.
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

// Block = one filter on one 32 x 8 output tile of one (sample, channel).
__global__ __launch_bounds__(kTX *kTY) void k_dog(const uint8_t *__restrict__ img, int C, int H,
                                                  int W, int F, int Ho, int Wo, DogParams p,
                                                  float *__restrict__ out)
{
#pragma clang fp contract(off)
    __shared__ float tile[(kTY + kMaxSpan) * (kTX + kMaxSpan)];
    __shared__ float coef[kMaxK * kMaxK];
    const int bc = blockIdx.z;  // b * C + c
    const int fi = blockIdx.y % p.nf, ty = blockIdx.y / p.nf;
    const int K = p.ks[fi], off = p.off[fi], cbase = p.cbase[fi];
    const int x0 = blockIdx.x * kTX, y0 = ty * kTY;
    const int tw = kTX + K - 1, th = kTY + K - 1;
    const uint8_t *src = img + (size_t)bc * H * W;
    const int tid = threadIdx.y * kTX + threadIdx.x;
    for (int i = tid; i < K * K; i += kTX * kTY) coef[i] = p.coef[cbase + i];
    for (int i = tid; i < tw * th; i += kTX * kTY) {
        const int r = i / tw, q = i - r * tw;
        const int iy = y0 + off + r, ix = x0 + off + q;
        const bool inside = (unsigned)iy < (unsigned)H && (unsigned)ix < (unsigned)W;
        const float u = (float)src[inside ? (size_t)iy * W + ix : 0];
        tile[i] = inside ? u / 255.0f : 0.0f;
    }
    __syncthreads();
    const int x = x0 + threadIdx.x, y = y0 + threadIdx.y;
    if (x >= Wo || y >= Ho) return;
    const int b = bc / C, c = bc - b * C;
    const float *cf = coef;
    const float *t0 = tile + threadIdx.y * tw + threadIdx.x;
    float acc;
    switch (K) {
    case 1: acc = window<1>(cf, t0, tw); break;
    case 3: acc = window<3>(cf, t0, tw); break;
    case 5: acc = window<5>(cf, t0, tw); break;
    case 7: acc = window<7>(cf, t0, tw); break;
    case 9: acc = window<9>(cf, t0, tw); break;
    case 11: acc = window<11>(cf, t0, tw); break;
    case 13: acc = window<13>(cf, t0, tw); break;
    case 15: acc = window<15>(cf, t0, tw); break;
    case 17: acc = window<17>(cf, t0, tw); break;
    case 19: acc = window<19>(cf, t0, tw); break;
    default: acc = window<21>(cf, t0, tw); break;
    }
    out[(((size_t)b * C + c) * F + p.fidx[fi]) * Ho * Wo + (size_t)y * Wo + x] = acc;
}

}  // namespace

extern "C" spk_status spk_dog_filter(const uint8_t *img, int B, int C, int H, int W,
                                     const spk_dog_desc *filters, int F, int pad, float *out,
                                     spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(img && filters && out, SPK_E_ARG, "spk_dog_filter: NULL pointer");
    SPK_REQUIRE(B > 0 && C > 0 && H > 0 && W > 0 && F > 0, SPK_E_ARG,
                "spk_dog_filter: B=%d C=%d H=%d W=%d F=%d must be positive", B, C, H, W, F);
    SPK_REQUIRE(F <= kMaxF, SPK_E_SHAPE, "spk_dog_filter: F=%d > %d", F, kMaxF);
    SPK_REQUIRE(pad >= -1, SPK_E_ARG, "spk_dog_filter: pad=%d (use -1 for same padding)", pad);
    for (int f = 0; f < F; f++) {
        const spk_dog_desc &d = filters[f];
        SPK_REQUIRE(d.ksize >= 1 && (d.ksize & 1), SPK_E_ARG,
                    "spk_dog_filter: filter %d ksize=%d must be odd and >= 1", f, d.ksize);
        SPK_REQUIRE(d.ksize <= kMaxK, SPK_E_SHAPE, "spk_dog_filter: filter %d ksize=%d > %d", f,
                    d.ksize, kMaxK);
        SPK_REQUIRE(d.sigma1 > 0.0 && d.sigma2 > 0.0, SPK_E_ARG,
                    "spk_dog_filter: filter %d sigmas must be positive", f);
        SPK_REQUIRE(pad < 0 || d.ksize == filters[0].ksize, SPK_E_UNSUPPORTED,
                    "spk_dog_filter: an explicit pad needs one kernel size for all filters");
    }
    const int Ho = pad < 0 ? H : H + 2 * pad - filters[0].ksize + 1;
    const int Wo = pad < 0 ? W : W + 2 * pad - filters[0].ksize + 1;
    SPK_REQUIRE(Ho > 0 && Wo > 0, SPK_E_SHAPE, "spk_dog_filter: output %dx%d is empty", Ho, Wo);
    SPK_REQUIRE((long long)spk::ceil_div(Ho, kTY) * kMaxF <= 65535, SPK_E_SHAPE,
                "spk_dog_filter: output height %d too large", Ho);
    SPK_REQUIRE((long long)B * C <= 65535, SPK_E_SHAPE, "spk_dog_filter: B*C=%lld > 65535",
                (long long)B * C);

    // Group the filters into launches that fit the by-value coefficient block.
    int f = 0;
    while (f < F) {
        DogParams p{};
        int used = 0;
        p.lo = 1 << 30;
        p.hi = -(1 << 30);
        while (f < F && p.nf < kMaxF) {
            int K = filters[f].ksize;
            if (used + K * K > kMaxCoef) break;
            int P = pad < 0 ? (K - 1) / 2 : pad;
            p.ks[p.nf] = K;
            p.off[p.nf] = -P;
            p.cbase[p.nf] = used;
            p.fidx[p.nf] = f;
            dog_coefficients(K, filters[f].sigma1, filters[f].sigma2, p.coef + used);
            p.lo = std::min(p.lo, -P);
            p.hi = std::max(p.hi, K - 1 - P);
            used += K * K;
            p.nf++;
            f++;
        }
        dim3 grid(spk::ceil_div(Wo, kTX), spk::ceil_div(Ho, kTY) * p.nf, B * C);
        hipLaunchKernelGGL(k_dog, grid, dim3(kTX, kTY), 0, spk::stream_of(stream), img, C, H, W, F,
                           Ho, Wo, p, out);
        SPK_LAUNCHED("spk_dog_filter");
    }
    return SPK_OK;
}
