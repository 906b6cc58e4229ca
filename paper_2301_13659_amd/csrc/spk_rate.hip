// Rate coding (Spyker §II-D.1) and the rate-coded network: integrate-and-
// fire over per-step frames (§II-E with the potential reset after a spike)
// and rate-based max pooling (§II-E.3).
//
// Under rate coding a neuron fires at many steps, so layers exchange frames
// B x T x C x H x W (one byte per neuron and step, the dense interface of
// §II-A) plus spike counts.  The convolution is an implicit GEMM per step on
// the matrix cores: a tile is 32 output positions x 32 maps, its 16-tap
// slices read one step's frame from a padded channels-last copy held as
// halves, and the
// accumulator is the potential itself: each step's products add the step's
// current to it, and after the step the neurons above theta spike and are
// set back to zero.  The wave walks all T steps of its tile, so the
// potential never leaves the registers.
#include <hip/hip_fp16.h>

#include <algorithm>
#include <cmath>

#include "spk_internal.h"

namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kSlack = 16;  // readable halves past the end of the packed frames
constexpr int kBatch = 16;  // slices loaded together

// ------------------------------------------------------------ rate code

// Per sample, the largest value above min_value (>= 0, so the float bits
// order like the values); 0 when there is none.
__global__ void k_rate_zero(uint32_t *m, int B)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < B) m[i] = 0u;
}

__global__ void k_rate_max(const float *__restrict__ x, int64_t n, float min_value, uint32_t *m)
{
    const int b = blockIdx.y;
    const float *xb = x + (size_t)b * n;
    uint32_t best = 0u;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const float v = xb[i];
        if (v > min_value) best = max(best, __float_as_uint(v));
    }
    for (int k = 32; k >= 1; k >>= 1) best = max(best, (uint32_t)__shfl_xor((int)best, k));
    if ((threadIdx.x & 63) == 0 && best) atomicMax(m + b, best);
}

// frames[b][t][i] = u[b][t][i] < x[b][i] / max_b (0 for x <= min_value).
__global__ void k_rate_frames(const float *__restrict__ x, const float *__restrict__ u, int64_t n,
                              int T, float min_value, const uint32_t *__restrict__ m,
                              uint8_t *__restrict__ frames)
{
    const int b = blockIdx.z;
    const int t = blockIdx.y;
    const float xm = __uint_as_float(m[b]);
    const size_t row = ((size_t)b * T + t) * n;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const float v = x[(size_t)b * n + i];
        const float p = (xm > 0.0f && v > min_value) ? v / xm : 0.0f;
        frames[row + i] = u[row + i] < p ? 1 : 0;
    }
}

// ------------------------------------------------------------ IF conv

struct RGeom {
    int B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo;
    int Cp;   // Ci rounded up to 8
    int Hp, Wp;
    int rowb;  // Wp * Cp
    int run;   // Kw * Cp
    int Q16;   // 16-tap slices per kernel row
    int SK;    // Kh * Q16
    int P, HoWo, NT;
    int ntb;   // column tiles per block (1, 2 or 4)
    int vec;   // 4-position vector stores possible
};

RGeom make_rgeom(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride, int pad)
{
    RGeom g{};
    g.B = B; g.T = T; g.Ci = Ci; g.Hi = Hi; g.Wi = Wi; g.Co = Co; g.Kh = Kh; g.Kw = Kw;
    g.stride = stride; g.pad = pad;
    g.Ho = (Hi + 2 * pad - Kh) / stride + 1;
    g.Wo = (Wi + 2 * pad - Kw) / stride + 1;
    g.Cp = (Ci + 7) / 8 * 8;
    g.Hp = Hi + 2 * pad;
    g.Wp = Wi + 2 * pad;
    g.rowb = g.Wp * g.Cp;
    g.run = Kw * g.Cp;
    g.Q16 = (g.run + 15) / 16;
    g.SK = Kh * g.Q16;
    g.HoWo = g.Ho * g.Wo;
    g.P = B * g.HoWo;
    g.NT = (Co + 31) / 32;
    return g;
}

size_t rate_xp_bytes(const RGeom &g)
{
    return spk::align_up(((size_t)g.B * g.T * g.Hp * g.rowb + kSlack) * sizeof(uint16_t), 256);
}

// One thread per padded pixel (b, t, yp, xp): its Cp channels as halves (1.0
// where the neuron spikes at that step, 0 in the padding and past Ci), so an
// A fragment is one 16-byte load.
__global__ void k_rate_pack(const uint8_t *__restrict__ frames, RGeom g, uint16_t *__restrict__ fp)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t npix = (int64_t)g.B * g.T * g.Hp * g.Wp;
    if (i >= npix) {
        if (i - npix < kSlack) fp[npix * g.Cp + (i - npix)] = 0;
        return;
    }
    const int xp = (int)(i % g.Wp);
    const int64_t r = i / g.Wp;
    const int yp = (int)(r % g.Hp);
    const int64_t bt = r / g.Hp;
    const int iy = yp - g.pad, ix = xp - g.pad;
    const bool in = (unsigned)iy < (unsigned)g.Hi && (unsigned)ix < (unsigned)g.Wi;
    const uint8_t *src = frames + (size_t)bt * g.Ci * g.Hi * g.Wi + (size_t)iy * g.Wi + ix;
    uint16_t *dst = fp + (size_t)i * g.Cp;
    for (int c0 = 0; c0 < g.Cp; c0 += 8) {
        u4 v;
#pragma unroll
        for (int q = 0; q < 4; q++) {
            uint32_t w = 0;
#pragma unroll
            for (int e = 0; e < 2; e++) {
                const int c = c0 + 2 * q + e;
                const bool on = in && c < g.Ci && src[(size_t)c * g.Hi * g.Wi] != 0;
                w |= (on ? 0x3C00u : 0u) << (16 * e);
            }
            v[q] = w;
        }
        *reinterpret_cast<u4 *>(dst + c0) = v;
    }
}

// B fragments [nt][s][k][lane]: lane l holds map 32*nt + l % 32 and taps
// 8*(l/32)..+7 of slice s (taps j = kx*Cp + c of kernel row ky); k = 0, 1:
// hi and lo halves of a float master, or k = 0 only: the half weights.
template <int NP, bool kHalfW>
__global__ void k_rate_pack_w(const void *__restrict__ wv, RGeom g, h8 *__restrict__ bp)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)g.NT * g.SK * NP * 64) return;
    const int lane = (int)(i % 64);
    const int64_t r = i / 64;
    const int k = (int)(r % NP);
    const int s = (int)((r / NP) % g.SK);
    const int nt = (int)(r / NP / g.SK);
    const int o = 32 * nt + lane % 32;
    const int ky = s / g.Q16, jq = s - ky * g.Q16;
    h8 f;
#pragma unroll
    for (int e = 0; e < 8; e++) {
        const int j = jq * 16 + 8 * (lane / 32) + e;
        const int kx = j / g.Cp, c = j - kx * g.Cp;
        float w = 0.0f;
        if (o < g.Co && j < g.run && c < g.Ci) {
            const size_t at = (((size_t)o * g.Ci + c) * g.Kh + ky) * g.Kw + kx;
            w = kHalfW ? (float)reinterpret_cast<const _Float16 *>(wv)[at]
                       : reinterpret_cast<const float *>(wv)[at];
        }
        const _Float16 hi = (_Float16)w;
        f[e] = k == 0 ? hi : (_Float16)(w - (float)hi);
    }
    bp[i] = f;
}

// Block: 4 waves = (4 / ntb) position tiles x ntb column tiles, whose B
// fragments sit in LDS.  A wave walks the T steps of its 32 x 32 tile; two
// accumulator chains (even and odd slices) keep the matrix cores busy, and
// are summed into the potential after each step.
template <int NP>
__global__ __launch_bounds__(kThreads) void k_rate_conv(const uint16_t *__restrict__ fp,
                                                        const h8 *__restrict__ bp, RGeom g,
                                                        float theta, uint8_t *__restrict__ out,
                                                        int32_t *__restrict__ counts)
{
    extern __shared__ __align__(16) uint8_t lds[];
    h8 *sb = reinterpret_cast<h8 *>(lds);
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int ntb = g.ntb;
    const int nt0 = blockIdx.y * ntb;
    const int per = g.SK * NP * 64;  // fragments of one column tile
    for (int i = threadIdx.x; i < ntb * per; i += blockDim.x) {
        const int tt = i / per;
        h8 z = {};
        sb[i] = nt0 + tt < g.NT ? bp[(size_t)(nt0 + tt) * per + (i - tt * per)] : z;
    }
    __syncthreads();
    const int ntl = wave % ntb;
    const int nt = nt0 + ntl;
    const int ptile = blockIdx.x * (4 / ntb) + wave / ntb;
    if (nt >= g.NT || ptile * 32 >= g.P) return;

    const int h = lane >> 5;
    const int p = ptile * 32 + (lane & 31);
    const int pc = min(p, g.P - 1);
    const int b = pc / g.HoWo, rem = pc - b * g.HoWo;
    const int y = rem / g.Wo, x = rem - y * g.Wo;
    const size_t stepb = (size_t)g.Hp * g.rowb;
    const uint16_t *src0 = fp + (size_t)b * g.T * stepb + (size_t)(y * g.stride) * g.rowb +
                           (size_t)(x * g.stride) * g.Cp + 8 * h;
    const h8 *bw = sb + (size_t)ntl * per + lane;
    const int o = 32 * nt + (lane & 31);
    const bool real_o = o < g.Co;

    f16v V = {}, V2 = {};
    int cnt[16];
#pragma unroll
    for (int e = 0; e < 16; e++) cnt[e] = 0;

    // a step's slices are loaded together, so the wave waits once per batch
    for (int t = 0; t < g.T; t++) {
        const uint16_t *src = src0 + (size_t)t * stepb;
        for (int q0 = 0; q0 < g.SK; q0 += kBatch) {
            h8 A[kBatch];
#pragma unroll
            for (int q = 0; q < kBatch; q++) {
                const int qq = q0 + q;
                const int ky = qq / g.Q16, jq = qq - ky * g.Q16;
                A[q] = qq < g.SK ? *reinterpret_cast<const h8 *>(src + ky * g.rowb + jq * 16) : h8{};
            }
#pragma unroll
            for (int q = 0; q < kBatch; q++) {
                const int qq = q0 + q;
                if (qq < g.SK) {
#pragma unroll
                    for (int k = 0; k < NP; k++) {
                        if (q & 1) V2 = __builtin_amdgcn_mfma_f32_32x32x16_f16(A[q], bw[(qq * NP + k) * 64], V2, 0, 0, 0);
                        else V = __builtin_amdgcn_mfma_f32_32x32x16_f16(A[q], bw[(qq * NP + k) * 64], V, 0, 0, 0);
                    }
                }
            }
        }
        uint32_t sp[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const float v = V[e] + V2[e];
            const bool f = v > theta;
            V[e] = f ? 0.0f : v;
            V2[e] = 0.0f;
            cnt[e] += f ? 1 : 0;
            sp[e >> 2] |= (f ? 1u : 0u) << (8 * (e & 3));
        }
        if (real_o) {
#pragma unroll
            for (int j = 0; j < 4; j++) {
                const int q0 = ptile * 32 + 8 * j + 4 * h;  // first of this lane's 4 positions
                if (q0 >= g.P) continue;
                const int bq = q0 / g.HoWo, rq = q0 - bq * g.HoWo;
                const size_t at = (((size_t)bq * g.T + t) * g.Co + o) * g.HoWo + rq;
                if (g.vec && q0 + 3 < g.P) {
                    *reinterpret_cast<uint32_t *>(out + at) = sp[j];
                } else {
                    for (int i = 0; i < 4 && q0 + i < g.P; i++) {
                        const int qi = q0 + i, bi = qi / g.HoWo, ri = qi - bi * g.HoWo;
                        out[(((size_t)bi * g.T + t) * g.Co + o) * g.HoWo + ri] = (uint8_t)(sp[j] >> (8 * i));
                    }
                }
            }
        }
    }
    if (real_o) {
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const int q = ptile * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
            if (q >= g.P) continue;
            const int bq = q / g.HoWo, rq = q - bq * g.HoWo;
            counts[((size_t)bq * g.Co + o) * g.HoWo + rq] = cnt[e];
        }
    }
}

// ------------------------------------------------------------ rate pool

// One thread per output neuron: the window's neuron with the most spikes
// (first in row-major order among equals) passes its train on.
__global__ void k_rate_pool(const uint8_t *__restrict__ in, const int32_t *__restrict__ cin, int B,
                            int T, int C, int Hi, int Wi, int Kh, int Kw, int stride, int pad, int Ho,
                            int Wo, uint8_t *__restrict__ out, int32_t *__restrict__ cout)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)B * C * Ho * Wo) return;
    const int xo = (int)(i % Wo);
    const int yo = (int)((i / Wo) % Ho);
    const int64_t bc = i / ((int64_t)Ho * Wo);
    const int32_t *cb = cin + (size_t)bc * Hi * Wi;
    int by = -1, bx = -1;
    int32_t best = -1;
    for (int ky = 0; ky < Kh; ky++) {
        const int iy = yo * stride + ky - pad;
        if ((unsigned)iy >= (unsigned)Hi) continue;
        for (int kx = 0; kx < Kw; kx++) {
            const int ix = xo * stride + kx - pad;
            if ((unsigned)ix >= (unsigned)Wi) continue;
            const int32_t v = cb[(size_t)iy * Wi + ix];
            if (v > best) {
                best = v;
                by = iy;
                bx = ix;
            }
        }
    }
    cout[i] = best < 0 ? 0 : best;
    const int b = (int)(bc / C), c = (int)(bc - (int64_t)b * C);
    for (int t = 0; t < T; t++) {
        const size_t ob = (((size_t)b * T + t) * C + c) * Ho * Wo + (size_t)yo * Wo + xo;
        out[ob] = by < 0 ? 0 : in[(((size_t)b * T + t) * C + c) * Hi * Wi + (size_t)by * Wi + bx];
    }
}

__global__ void k_rate_features(const int32_t *__restrict__ counts, int64_t n, int T, float *__restrict__ out)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        out[i] = (float)counts[i] / (float)T;
}

int lds_per_block()
{
    static int n = 0;
    if (n == 0) {
        int dev = 0, v = 0;
        n = (hipGetDevice(&dev) == hipSuccess &&
             hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess && v > 0)
                ? v
                : 65536;
    }
    return n;
}

// Column tiles per block whose B fragments fit LDS (0: none fits).
int rate_ntb(const RGeom &g, int np)
{
    for (int ntb : {4, 2, 1}) {
        if (ntb > 1 && g.NT <= ntb / 2) continue;
        if ((size_t)ntb * g.SK * np * 64 * sizeof(h8) <= (size_t)lds_per_block()) return ntb;
    }
    return 0;
}

}  // namespace

// ------------------------------------------------------------------ ABI

extern "C" spk_status spk_rate_code(const float *x, const float *u, int B, int64_t n, int T,
                                    float min_value, uint8_t *frames, void *ws, size_t ws_bytes,
                                    spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(x && u && frames && ws, SPK_E_ARG, "spk_rate_code: NULL pointer");
    SPK_REQUIRE(B > 0 && n > 0, SPK_E_ARG, "spk_rate_code: sizes must be positive");
    SPK_REQUIRE(T >= 1 && B <= 65535 && T <= 65535, SPK_E_SHAPE, "spk_rate_code: T=%d or B=%d out of range", T, B);
    SPK_REQUIRE(min_value >= 0.0f, SPK_E_ARG, "spk_rate_code: min_value must be >= 0");
    SPK_REQUIRE(ws_bytes >= (size_t)B * 4, SPK_E_WORKSPACE, "spk_rate_code: workspace %zu < %zu bytes",
                ws_bytes, (size_t)B * 4);
    SPK_REQUIRE_WS_ALIGNED(ws, "spk_rate_code");
    hipStream_t s = spk::stream_of(stream);
    uint32_t *m = static_cast<uint32_t *>(ws);
    hipLaunchKernelGGL(k_rate_zero, dim3((B + 255) / 256), dim3(256), 0, s, m, B);
    const unsigned bx = (unsigned)std::min<int64_t>(64, (n + 255) / 256);
    hipLaunchKernelGGL(k_rate_max, dim3(bx, B), dim3(256), 0, s, x, n, min_value, m);
    hipLaunchKernelGGL(k_rate_frames, dim3(bx, T, B), dim3(256), 0, s, x, u, n, T, min_value, m, frames);
    SPK_LAUNCHED("spk_rate_code");
    return SPK_OK;
}

extern "C" size_t spk_conv_if_rate_workspace_size(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh,
                                                  int Kw, int stride, int pad, spk_dtype w_dtype)
{
    if (B < 1 || T < 1 || Ci < 1 || Hi < 1 || Wi < 1 || Co < 1 || Kh < 1 || Kw < 1 || stride < 1 ||
        pad < 0 || Hi + 2 * pad < Kh || Wi + 2 * pad < Kw)
        return 0;
    const RGeom g = make_rgeom(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad);
    const int np = w_dtype == SPK_F16 ? 1 : 2;
    return rate_xp_bytes(g) + spk::align_up((size_t)g.NT * g.SK * np * 64 * sizeof(h8), 256);
}

extern "C" spk_status spk_conv_if_rate(const uint8_t *frames, int B, int T, int Ci, int Hi, int Wi,
                                       const void *w, spk_dtype w_dtype, int Co, int Kh, int Kw,
                                       int stride, int pad, float theta, uint8_t *out_frames,
                                       int32_t *counts, void *ws, size_t ws_bytes, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(frames && w && out_frames && counts && ws, SPK_E_ARG, "spk_conv_if_rate: NULL pointer");
    SPK_REQUIRE(B > 0 && T > 0 && Ci > 0 && Hi > 0 && Wi > 0 && Co > 0 && Kh > 0 && Kw > 0 &&
                    stride > 0 && pad >= 0,
                SPK_E_ARG, "spk_conv_if_rate: sizes must be positive (pad >= 0)");
    SPK_REQUIRE(w_dtype == SPK_F32 || w_dtype == SPK_F16, SPK_E_UNSUPPORTED,
                "spk_conv_if_rate: unknown weight dtype %d", (int)w_dtype);
    SPK_REQUIRE(std::isfinite(theta), SPK_E_ARG, "spk_conv_if_rate: theta must be finite");
    const int Ho = spk_out_extent(Hi, Kh, stride, pad), Wo = spk_out_extent(Wi, Kw, stride, pad);
    SPK_REQUIRE(Ho > 0 && Wo > 0, SPK_E_SHAPE, "spk_conv_if_rate: empty output (%d x %d)", Ho, Wo);
    SPK_REQUIRE((long long)B * T * Co * Ho * Wo < (1ll << 40) && (long long)B * Ho * Wo < (1ll << 31),
                SPK_E_SHAPE, "spk_conv_if_rate: tensor too large");
    RGeom g = make_rgeom(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad);
    const bool half_w = w_dtype == SPK_F16;
    const int np = half_w ? 1 : 2;
    g.ntb = rate_ntb(g, np);
    SPK_REQUIRE(g.ntb > 0, SPK_E_UNSUPPORTED, "spk_conv_if_rate: %d weight slices do not fit LDS", g.SK);
    SPK_REQUIRE(g.NT <= 65535 * g.ntb, SPK_E_SHAPE, "spk_conv_if_rate: Co=%d too large", Co);
    const size_t xb = rate_xp_bytes(g);
    const size_t need = xb + spk::align_up((size_t)g.NT * g.SK * np * 64 * sizeof(h8), 256);
    SPK_REQUIRE(ws_bytes >= need, SPK_E_WORKSPACE, "spk_conv_if_rate: workspace %zu < %zu bytes",
                ws_bytes, need);
    SPK_REQUIRE_WS_ALIGNED(ws, "spk_conv_if_rate");
    g.vec = (g.HoWo % 4 == 0) && ((uintptr_t)out_frames % 4 == 0);
    uint16_t *fp = static_cast<uint16_t *>(ws);
    h8 *bp = reinterpret_cast<h8 *>(static_cast<uint8_t *>(ws) + xb);
    hipStream_t s = spk::stream_of(stream);
    const int64_t npix = (int64_t)B * T * g.Hp * g.Wp + kSlack;
    hipLaunchKernelGGL(k_rate_pack, dim3((unsigned)((npix + 255) / 256)), dim3(256), 0, s, frames, g, fp);
    const int64_t nf = (int64_t)g.NT * g.SK * np * 64;
    if (half_w)
        hipLaunchKernelGGL((k_rate_pack_w<1, true>), dim3((unsigned)((nf + 255) / 256)), dim3(256), 0, s, w, g, bp);
    else
        hipLaunchKernelGGL((k_rate_pack_w<2, false>), dim3((unsigned)((nf + 255) / 256)), dim3(256), 0, s, w, g, bp);
    const int ptiles = (g.P + 31) / 32;
    const int per_block = 4 / g.ntb;
    const dim3 grid((unsigned)((ptiles + per_block - 1) / per_block), (unsigned)((g.NT + g.ntb - 1) / g.ntb));
    const size_t lds = (size_t)g.ntb * g.SK * np * 64 * sizeof(h8);
    if (half_w)
        hipLaunchKernelGGL(k_rate_conv<1>, grid, dim3(kThreads), lds, s, fp, bp, g, theta, out_frames, counts);
    else
        hipLaunchKernelGGL(k_rate_conv<2>, grid, dim3(kThreads), lds, s, fp, bp, g, theta, out_frames, counts);
    SPK_LAUNCHED("spk_conv_if_rate");
    return SPK_OK;
}

extern "C" spk_status spk_rate_pool(const uint8_t *in_frames, const int32_t *in_counts, int B, int T,
                                    int C, int Hi, int Wi, int Kh, int Kw, int stride, int pad,
                                    uint8_t *out_frames, int32_t *out_counts, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(in_frames && in_counts && out_frames && out_counts, SPK_E_ARG, "spk_rate_pool: NULL pointer");
    SPK_REQUIRE(B > 0 && T > 0 && C > 0 && Hi > 0 && Wi > 0, SPK_E_ARG, "spk_rate_pool: sizes must be positive");
    const int Ho = spk_out_extent(Hi, Kh, stride, pad), Wo = spk_out_extent(Wi, Kw, stride, pad);
    SPK_REQUIRE(Ho > 0 && Wo > 0, SPK_E_SHAPE, "spk_rate_pool: empty output (%d x %d)", Ho, Wo);
    const int64_t n = (int64_t)B * C * Ho * Wo;
    hipLaunchKernelGGL(k_rate_pool, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, spk::stream_of(stream),
                       in_frames, in_counts, B, T, C, Hi, Wi, Kh, Kw, stride, pad, Ho, Wo, out_frames,
                       out_counts);
    SPK_LAUNCHED("spk_rate_pool");
    return SPK_OK;
}

extern "C" spk_status spk_rate_features(const int32_t *counts, int64_t n, int T, float *out, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE((counts && out) || n == 0, SPK_E_ARG, "spk_rate_features: NULL pointer");
    SPK_REQUIRE(n >= 0 && T > 0, SPK_E_ARG, "spk_rate_features: n=%lld T=%d", (long long)n, T);
    if (n == 0) return SPK_OK;
    hipLaunchKernelGGL(k_rate_features, dim3((unsigned)std::min<int64_t>(4096, (n + 255) / 256)), dim3(256), 0,
                       spk::stream_of(stream), counts, n, T, out);
    SPK_LAUNCHED("spk_rate_features");
    return SPK_OK;
}
