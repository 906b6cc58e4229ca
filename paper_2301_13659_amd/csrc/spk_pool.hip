// spk_pool: max-pooling of spikes under rank-order coding (Spyker §II-E.3, Eq. 3).
// The earliest spike of the window wins: a minimum over uint8 first-spike
// times, one thread per output neuron.  Padding cells never fire.
#include "spk_internal.h"

namespace {

__global__ void k_pool(const uint8_t *__restrict__ in, int Hi, int Wi, int Kh, int Kw, int stride,
                       int pad, int Ho, int Wo, long long total, uint8_t *__restrict__ out)
{
    long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total) return;
    const int x = (int)(i % Wo);
    const int y = (int)((i / Wo) % Ho);
    const long long bc = i / ((long long)Ho * Wo);
    const uint8_t *src = in + bc * Hi * Wi;
    int m = spk::kNever;
    const int y0 = y * stride - pad, x0 = x * stride - pad;
    for (int ky = 0; ky < Kh; ky++) {
        int iy = y0 + ky;
        if (iy < 0 || iy >= Hi) continue;
        for (int kx = 0; kx < Kw; kx++) {
            int ix = x0 + kx;
            if (ix >= 0 && ix < Wi) m = min(m, (int)src[(long long)iy * Wi + ix]);
        }
    }
    out[i] = (uint8_t)m;
}

}  // namespace

extern "C" spk_status spk_pool(const uint8_t *in_times, int B, int C, int Hi, int Wi, int Kh,
                               int Kw, int stride, int pad, uint8_t *out_times, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(in_times && out_times, SPK_E_ARG, "spk_pool: NULL pointer");
    SPK_REQUIRE(B > 0 && C > 0 && Hi > 0 && Wi > 0 && Kh > 0 && Kw > 0 && stride > 0 && pad >= 0,
                SPK_E_ARG, "spk_pool: sizes must be positive (pad >= 0)");
    const int Ho = spk_out_extent(Hi, Kh, stride, pad), Wo = spk_out_extent(Wi, Kw, stride, pad);
    SPK_REQUIRE(Ho > 0 && Wo > 0, SPK_E_SHAPE, "spk_pool: no output for %dx%d, window %dx%d", Hi,
                Wi, Kh, Kw);
    const long long total = (long long)B * C * Ho * Wo;
    hipLaunchKernelGGL(k_pool, dim3(spk::ceil_div(total, 256)), dim3(256), 0,
                       spk::stream_of(stream), in_times, Hi, Wi, Kh, Kw, stride, pad, Ho, Wo, total,
                       out_times);
    SPK_LAUNCHED("spk_pool");
    return SPK_OK;
}
