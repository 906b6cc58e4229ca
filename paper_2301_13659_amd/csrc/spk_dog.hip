// spk_dog_filter: DoG feature enhancement (Spyker §II-C.1, shape rule Eq. 1).
//
// The filter bank is tiny (at most 8 kernels, K <= 21), so its coefficients
// are computed on the host and travel by value in the kernel arguments.  A
// block evaluates one filter on a 128 x 8 output tile: it stages the scaled
// input pixels (u / 255) of the tile and its halo in LDS, then each thread
// runs the fully unrolled window of that kernel size over 4 consecutive
// outputs of a row, reading each kernel row's pixels once for the four.
// Every output is accumulated in float, window row-major, without
// contraction, so it is reproducible bit for bit (the rank-order coder
// downstream turns last-bit differences into different spike times).
#include "spk_dog.h"

namespace {

using spk::dog::DogParams;
constexpr int kTX = 32, kTY = 8;  // threads of a block
constexpr int kRun = 4;           // outputs along x per thread
constexpr int kOX = kTX * kRun;   // output columns of a block
constexpr int kMaxSpan = spk::dog::kMaxK - 1;

// Block = one filter on one 128 x 8 output tile of one (sample, channel);
// each thread computes 4 consecutive outputs of a row with window_run, which
// sums every output exactly as the single-output window does.
__global__ __launch_bounds__(kTX *kTY) void k_dog(const uint8_t *__restrict__ img, int C, int H,
                                                  int W, int F, int Ho, int Wo, DogParams p,
                                                  float *__restrict__ out)
{
    __shared__ float tile[(kTY + kMaxSpan) * (kOX + kMaxSpan)];
    __shared__ float coef[spk::dog::kMaxK * spk::dog::kMaxK];
    const int bc = blockIdx.z;  // b * C + c
    const int fi = blockIdx.y % p.nf, ty = blockIdx.y / p.nf;
    const int K = p.ks[fi], off = p.off[fi], cbase = p.cbase[fi];
    const int x0 = blockIdx.x * kOX, y0 = ty * kTY;
    const int tw = kOX + K - 1, th = kTY + K - 1;
    const uint8_t *src = img + (size_t)bc * H * W;
    const int tid = threadIdx.y * kTX + threadIdx.x;
    for (int i = tid; i < K * K; i += kTX * kTY) coef[i] = p.coef[cbase + i];
    for (int i = tid; i < tw * th; i += kTX * kTY) {
        const int r = i / tw, q = i - r * tw;
        tile[i] = spk::dog::pixel(src, H, W, y0 + off + r, x0 + off + q);
    }
    __syncthreads();
    const int xs = x0 + threadIdx.x * kRun, y = y0 + threadIdx.y;
    if (xs >= Wo || y >= Ho) return;
    const int b = bc / C, c = bc - b * C;
    float acc[kRun];
    spk::dog::window_run_k<kRun>(K, coef, tile + threadIdx.y * tw + threadIdx.x * kRun, tw, acc);
    float *o = out + (((size_t)b * C + c) * F + p.fidx[fi]) * Ho * Wo + (size_t)y * Wo;
#pragma unroll
    for (int r = 0; r < kRun; r++)
        if (xs + r < Wo) o[xs + r] = acc[r];
}

}  // namespace

extern "C" spk_status spk_dog_filter(const uint8_t *img, int B, int C, int H, int W,
                                     const spk_dog_desc *filters, int F, int pad, float *out,
                                     spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(img && filters && out, SPK_E_ARG, "spk_dog_filter: NULL pointer");
    int Ho = 0, Wo = 0;
    const spk_status st = spk::dog::plan("spk_dog_filter", B, C, H, W, filters, F, pad, Ho, Wo);
    if (st != SPK_OK) return st;
    SPK_REQUIRE((long long)spk::ceil_div(Ho, kTY) * spk::dog::kMaxF <= 65535, SPK_E_SHAPE,
                "spk_dog_filter: output height %d too large", Ho);
    SPK_REQUIRE((long long)B * C <= 65535, SPK_E_SHAPE, "spk_dog_filter: B*C=%lld > 65535",
                (long long)B * C);

    // Group the filters into launches that fit the by-value coefficient block.
    for (int f = 0; f < F;) {
        DogParams p;
        f = spk::dog::group(filters, F, pad, f, p);
        dim3 grid(spk::ceil_div(Wo, kOX), spk::ceil_div(Ho, kTY) * p.nf, B * C);
        hipLaunchKernelGGL(k_dog, grid, dim3(kTX, kTY), 0, spk::stream_of(stream), img, C, H, W, F,
                           Ho, Wo, p, out);
        SPK_LAUNCHED("spk_dog_filter");
    }
    return SPK_OK;
}
