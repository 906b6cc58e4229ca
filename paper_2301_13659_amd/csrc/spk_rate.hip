// Rate coding (Spyker §II-D.1) and the rate-coded network: integrate-and-
// fire over per-step frames (§II-E with the potential reset after a spike)
// and rate-based max pooling (§II-E.3).
//
// Under rate coding a neuron fires at many steps, so layers exchange frames
// B x T x C x H x W (one byte per neuron and step, the dense interface of
// §II-A) plus spike counts.  The convolution is an implicit GEMM per step on
// the matrix cores over a padded channels-last copy of the frames, and the
// wave walks all T steps of its tile, so the potential never leaves the
// registers: each step's products give the step's current, which is added to
// the potential, and after the step the neurons above theta spike and are
// set back to zero.
//
// The main kernel (k_rate_conv16) takes 16 output positions x 16 or 32 maps
// per wave on the 16x16x32 products.  The copy holds one byte per input
// (0x3C where it spikes, 0 elsewhere: the high byte of the half 1.0), the
// depth is walked in groups of 8 channels of one window pixel (four groups
// per product), the B fragments stay in registers and each lane keeps the
// loads of several steps ahead in flight, so a step costs the memory latency
// only once per batch of steps.  Layers whose weights do not fit a wave's
// registers take k_rate_conv: 32 x 32 tiles, B fragments in LDS, the copy
// held as halves.
#include <hip/hip_fp16.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <utility>

#include "spk_internal.h"

namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kSlack = 16;  // readable halves past the end of the packed frames
constexpr int kBatch = 16;  // slices loaded together
constexpr int kMaxKB = 12;  // depth blocks of 32 taps k_rate_conv16 holds in registers

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
// Thread: 4 consecutive values (kVec: n a multiple of 4, 16-byte vectors) or
// one, for kRateTT consecutive steps starting at blockIdx.y * kRateTT.
constexpr int kRateTT = 3;  // (10 held 40 draws per thread and ran at half the rate)

template <bool kVec>
__global__ void k_rate_frames(const float *__restrict__ x, const float *__restrict__ u, int64_t n,
                              int T, float min_value, const uint32_t *__restrict__ m,
                              uint8_t *__restrict__ frames)
{
    const int b = blockIdx.z;
    const int t0 = blockIdx.y * kRateTT;
    const float xm = __uint_as_float(m[b]);
    constexpr int L = kVec ? 4 : 1;
    const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * L;
    if (i >= n) return;
    float p[L];
#pragma unroll
    for (int e = 0; e < L; e++) {
        const float v = x[(size_t)b * n + i + e];
        p[e] = (xm > 0.0f && v > min_value) ? v / xm : 0.0f;
    }
    // every step's draws are loaded before the comparisons
    float uu[kRateTT][L];
#pragma unroll
    for (int k = 0; k < kRateTT; k++) {
        const size_t row = ((size_t)b * T + min(t0 + k, T - 1)) * n + i;
        if (kVec) {
            const float4 q = *reinterpret_cast<const float4 *>(u + row);
            uu[k][0] = q.x; uu[k][L > 1 ? 1 : 0] = q.y; uu[k][L > 2 ? 2 : 0] = q.z; uu[k][L > 3 ? 3 : 0] = q.w;
        } else {
            uu[k][0] = u[row];
        }
    }
#pragma unroll
    for (int k = 0; k < kRateTT; k++) {
        if (t0 + k >= T) break;
        const size_t row = ((size_t)b * T + t0 + k) * n + i;
        if (kVec) {
            uint32_t w = 0u;
#pragma unroll
            for (int e = 0; e < L; e++) w |= (uu[k][e] < p[e] ? 1u : 0u) << (8 * e);
            *reinterpret_cast<uint32_t *>(frames + row) = w;
        } else {
            frames[row] = uu[k][0] < p[0] ? 1 : 0;
        }
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
    // k_rate_conv16: 8-tap channel groups per pixel, groups of the window,
    // 32-tap depth blocks, 16-map column tiles
    int G8, G, KB, NT16;
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
    g.G8 = g.Cp / 8;
    g.G = Kh * Kw * g.G8;
    g.KB = (g.G + 3) / 4;
    g.NT16 = (Co + 15) / 16;
    return g;
}

// Bytes of the indicator copy of k_rate_conv16: [b][t][Hp][Wp][Cp].
size_t rate_x8_bytes(const RGeom &g) { return spk::align_up((size_t)g.B * g.T * g.Hp * g.rowb, 256); }

// k_rate_conv16's choices: 16-map column tiles per wave (NC) and weight
// products per depth block (NP), with KB * NC * NP <= 20 (B fragments in at
// most 80 registers); NC = 0 when the layer does not fit.
int rate16_nc(const RGeom &g, int np)
{
    // buffer offsets are 32-bit: the copy and the output frames below 2^31 bytes
    // (and one packing block row per frame: B*T <= 65535)
    if (g.KB > kMaxKB || (long long)g.B * g.T * g.Hp * g.rowb >= (1ll << 31) ||
        (long long)g.B * g.T * g.Co * g.HoWo >= (1ll << 31) || (long long)g.B * g.T > 65535)
        return 0;
    const int nc = g.NT16 >= 2 && np == 1 && g.KB <= 9 ? 2 : 1;
    return g.KB * nc * np <= 20 ? nc : 0;
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

// One thread per padded pixel (b, t, yp, xp) of frame bt = blockIdx.y: its Cp
// indicator bytes, 0x3C where the input spikes at that step, 0 in the
// padding and past Ci, written as 8-byte words.
__global__ void k_rate_pack8(const uint8_t *__restrict__ frames, RGeom g, uint2 *__restrict__ x8)
{
    const int i = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    const int npx = g.Hp * g.Wp;
    if (i >= npx) return;
    const int bt = (int)blockIdx.y;
    const int yp = i / g.Wp, xp = i - yp * g.Wp;
    const int iy = yp - g.pad, ix = xp - g.pad;
    const bool in = (unsigned)iy < (unsigned)g.Hi && (unsigned)ix < (unsigned)g.Wi;
    const uint8_t *src = frames + (size_t)bt * g.Ci * g.Hi * g.Wi + (size_t)(in ? iy : 0) * g.Wi + (in ? ix : 0);
    uint2 *dst = x8 + ((size_t)bt * npx + i) * (g.Cp / 8);
    for (int c0 = 0; c0 < g.Cp; c0 += 8) {
        // the 8 loads first (clamped channel, no branch around a load), then the bytes
        uint8_t v[8];
#pragma unroll
        for (int e = 0; e < 8; e++) v[e] = src[(size_t)min(c0 + e, g.Ci - 1) * g.Hi * g.Wi];
        uint32_t w[2] = {0u, 0u};
#pragma unroll
        for (int e = 0; e < 8; e++)
            if (in && c0 + e < g.Ci && v[e] != 0) w[e >> 2] |= 0x3Cu << (8 * (e & 3));
        dst[c0 / 8] = make_uint2(w[0], w[1]);
    }
}

// The same copy with one block per frame bt = blockIdx.x: the frame's
// Ci*Hi*Wi bytes are loaded into LDS as dwords (kAligned: the frames are
// 4-byte aligned) or bytes, then each thread writes the 8 bytes of a
// channel group (8 channels of a padded pixel) gathered from LDS.
template <bool kAligned>
__global__ __launch_bounds__(256) void k_rate_pack8_lds(const uint8_t *__restrict__ frames, RGeom g,
                                                        uint2 *__restrict__ x8)
{
    extern __shared__ __align__(16) uint8_t fr[];
    const int bt = (int)blockIdx.x;
    const int HW = g.Hi * g.Wi, nbytes = g.Ci * HW;
    const uint8_t *src = frames + (size_t)bt * nbytes;
    if (kAligned) {
        const uint32_t *s4 = reinterpret_cast<const uint32_t *>(src);
        for (int i = threadIdx.x; i < nbytes / 4; i += blockDim.x) reinterpret_cast<uint32_t *>(fr)[i] = s4[i];
        for (int i = (nbytes / 4) * 4 + threadIdx.x; i < nbytes; i += blockDim.x) fr[i] = src[i];
    } else {
        for (int i = threadIdx.x; i < nbytes; i += blockDim.x) fr[i] = src[i];
    }
    __syncthreads();
    const int n8 = g.Hp * g.Wp * g.G8;
    uint2 *dst = x8 + (size_t)bt * n8;
    for (int i = threadIdx.x; i < n8; i += blockDim.x) {
        const int px = i / g.G8, c0 = 8 * (i - px * g.G8);
        const int yp = px / g.Wp, xp = px - yp * g.Wp;
        const int iy = yp - g.pad, ix = xp - g.pad;
        const bool in = (unsigned)iy < (unsigned)g.Hi && (unsigned)ix < (unsigned)g.Wi;
        const int at = in ? iy * g.Wi + ix : 0;
        uint32_t w[2] = {0u, 0u};
#pragma unroll
        for (int e = 0; e < 8; e++) {
            const int c = c0 + e;
            if (in && c < g.Ci && fr[c * HW + at] != 0) w[e >> 2] |= 0x3Cu << (8 * (e & 3));
        }
        dst[i] = make_uint2(w[0], w[1]);
    }
}

// B fragments of k_rate_conv16, [ct][kb][k][lane]: lane l holds map
// 16*ct + l % 16 and the 8 taps of channel group 4*kb + l / 16 (group gi =
// pixel (ky*Kw + kx)*G8 + cg: channels 8*cg..+7 of window pixel (ky, kx));
// k = 0, 1: hi and lo halves of a float master, or k = 0 only: the half
// weights.  Zero past Co, Ci and the window.
template <int NP, bool kHalfW>
__global__ void k_rate_pack_w16(const void *__restrict__ wv, RGeom g, h8 *__restrict__ bp)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)g.NT16 * g.KB * NP * 64) return;
    const int lane = (int)(i % 64);
    const int64_t r = i / 64;
    const int k = (int)(r % NP);
    const int kb = (int)((r / NP) % g.KB);
    const int ct = (int)(r / NP / g.KB);
    const int o = 16 * ct + lane % 16;
    const int gi = 4 * kb + lane / 16;
    const int pix = gi / g.G8, cg = gi - pix * g.G8;
    const int ky = pix / g.Kw, kx = pix - ky * g.Kw;
    h8 f;
#pragma unroll
    for (int e = 0; e < 8; e++) {
        const int c = 8 * cg + e;
        float w = 0.0f;
        if (o < g.Co && gi < g.G && c < g.Ci) {
            const size_t at = (((size_t)o * g.Ci + c) * g.Kh + ky) * g.Kw + kx;
            w = kHalfW ? (float)reinterpret_cast<const _Float16 *>(wv)[at]
                       : reinterpret_cast<const float *>(wv)[at];
        }
        const _Float16 hi = (_Float16)w;
        f[e] = k == 0 ? hi : (_Float16)(w - (float)hi);
    }
    bp[i] = f;
}

// 8 indicator bytes as an A fragment: each byte the high byte of a half.
__device__ __forceinline__ h8 frag_ind(uint2 x)
{
    u4 v = {__builtin_amdgcn_perm(x.y, x.x, 0x010C000Cu), __builtin_amdgcn_perm(x.y, x.x, 0x030C020Cu),
            __builtin_amdgcn_perm(x.y, x.x, 0x050C040Cu), __builtin_amdgcn_perm(x.y, x.x, 0x070C060Cu)};
    return __builtin_bit_cast(h8, v);
}

// Block = 8 waves = 128 consecutive output positions (wave w: the 16-position
// tile 8*block + w) x NC column tiles of 16 maps, all T steps.  Lane l: A row
// (position) l % 16 and channel group 4*kb + l / 16 of depth block kb; B
// column (map) l % 16; the 16x16 results: map l % 16, positions
// 4*(l/16)..+3.  The loads of steps t+1..t+D-1 are in flight while step t is
// computed (D*KB loads at most, within the 63 the counter tracks).  Spikes go
// to LDS, [step][map][position] over D steps (two such buffers), and every D
// steps the block writes them out as rows of 128 positions per map and step,
// so the frame stores fill whole cache lines.
constexpr int kRW = 8;                    // waves per block
constexpr int kNT = 2;                    // cache policy of a buffer store: non-temporal
constexpr int kRRow = 32 * kRW + 4;       // bytes of a staged map row (128 positions, padded)

template <int KB, int NC, int NP, int D>
__global__ __launch_bounds__(64 * kRW) __attribute__((amdgpu_waves_per_eu(2)))
void k_rate_conv16(const uint8_t *__restrict__ x8, const h8 *__restrict__ bp, RGeom g, float theta,
                   uint8_t *__restrict__ out, int32_t *__restrict__ counts)
{
    extern __shared__ __align__(16) uint8_t lds[];
    const int lane = threadIdx.x & 63, wave = (int)(threadIdx.x >> 6);
    const int pblk = blockIdx.x * 16 * kRW;  // first position of the block
    const int tile = blockIdx.x * kRW + wave;
    const int ct0 = blockIdx.y * NC;
    h8 bw[NC][KB][NP];
#pragma unroll
    for (int c = 0; c < NC; c++)
#pragma unroll
        for (int kb = 0; kb < KB; kb++)
#pragma unroll
            for (int k = 0; k < NP; k++) {
                const int ct = min(ct0 + c, g.NT16 - 1);  // a missing tile's maps are never stored
                bw[c][kb][k] = bp[((size_t)(ct * KB + kb) * NP + k) * 64 + lane];
            }
    // this lane's A row: position p (the last one for rows past P, whose
    // results are not stored); its operand of depth block kb at step t is the
    // 8 bytes at x8 + t*stepb + loff[kb] (the copy is below 2^31 bytes)
    const int p = min(tile * 16 + (lane & 15), g.P - 1);
    const int b = p / g.HoWo, rem = p - b * g.HoWo;
    const int y = rem / g.Wo, x = rem - y * g.Wo;
    const uint32_t stepb = (uint32_t)g.Hp * g.rowb;
    const uint32_t pos_off = (uint32_t)b * g.T * stepb + (uint32_t)(y * g.stride) * g.rowb +
                             (uint32_t)(x * g.stride) * g.Cp;
    uint32_t loff[KB];
#pragma unroll
    for (int kb = 0; kb < KB; kb++) {
        const int gi = 4 * kb + (lane >> 4);
        const int pix = gi / g.G8, cg = gi - pix * g.G8;
        const int ky = pix / g.Kw, kx = pix - ky * g.Kw;
        loff[kb] = pos_off + (gi < g.G ? ky * g.rowb + kx * g.Cp + 8 * cg : 0);  // past the window: weights 0
    }
    // buffer loads: the step's offset is a scalar, each lane adds its own
    // (no 64-bit address per load and step)
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(x8), 0, (int)(stepb * g.T * g.B), 0x00020000);
    auto load_step = [&](int t, uint2 *dst) {
        const int so = __builtin_amdgcn_readfirstlane((int)(t * stepb));
#pragma unroll
        for (int kb = 0; kb < KB; kb++) {
            const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, (int)loff[kb], so, 0);
            dst[kb] = make_uint2(v[0], v[1]);
        }
    };
    uint2 A[D][KB];
#pragma unroll
    for (int j = 0; j < D; j++)
        if (j < g.T) load_step(j, A[j]);

    f4 V[NC];
    int cnt[NC][4];
#pragma unroll
    for (int c = 0; c < NC; c++)
#pragma unroll
        for (int e = 0; e < 4; e++) {
            V[c][e] = 0.0f;
            cnt[c][e] = 0;
        }
    const uint32_t tstep = (uint32_t)g.Co * g.HoWo;
    const __amdgpu_buffer_rsrc_t ro =
        __builtin_amdgcn_make_buffer_rsrc(out, 0, (int)(tstep * g.T * g.B), 0x00020000);
    // staged spikes: buffer h, step s, map m of the block's NC*16: row of
    // 128 position bytes at lds + ((h*D + s)*NC*16 + m)*kRRow
    const int my_col = 16 * wave + 4 * (lane >> 4);  // this lane's 4 positions in the row
    // The staged steps [t0, t0 + n) of buffer h to the frames: thread i
    // writes positions 4*(i % 32)..+3 (one dword, the same for all its rows)
    // of the (step, map) rows i / 32 + 16k; a wave covers two rows of 128
    // positions.  qoff[e]: frame offset of position e at step 0 and map 0.
    const int fdw = (int)(threadIdx.x & 31), fq = pblk + 4 * fdw;
    const bool fvec = g.vec && fq + 3 < g.P;  // 4 positions of one sample (HoWo a multiple of 4, fq too)
    uint32_t qoff[4];
#pragma unroll
    for (int e = 0; e < 4; e++) {
        const int qe = min(fq + e, g.P - 1), bi = qe / g.HoWo;
        qoff[e] = (uint32_t)bi * g.T * tstep + (uint32_t)(qe - bi * g.HoWo);
    }
    auto flush = [&](int h, int t0, int n) {
        if (fq >= g.P) return;
        const int rows = n * NC * 16;
        for (int row = (int)(threadIdx.x >> 5); row < rows; row += 2 * kRW) {
            const int st = row / (NC * 16), m = row - st * (NC * 16);
            const int o = 16 * ct0 + m;
            if (o >= g.Co) continue;
            const uint32_t v = *reinterpret_cast<const uint32_t *>(lds + (size_t)(h * D * NC * 16 + row) * kRRow + 4 * fdw);
            const uint32_t base = (uint32_t)(t0 + st) * tstep + (uint32_t)o * g.HoWo;
            // streaming (non-temporal) stores: the frames are read once, much later
            if (fvec) {
                __builtin_amdgcn_raw_buffer_store_b32(v, ro, (int)(base + qoff[0]), 0, kNT);
            } else {
#pragma unroll
                for (int e = 0; e < 4; e++)
                    if (fq + e < g.P)
                        __builtin_amdgcn_raw_buffer_store_b8((uint8_t)(v >> (8 * e)), ro, (int)(base + qoff[e]), 0, kNT);
            }
        }
    };
    int h = 0;
    for (int t0 = 0; t0 < g.T; t0 += D, h ^= 1) {
#pragma unroll
        for (int j = 0; j < D; j++) {
            const int t = t0 + j;
            if (t >= g.T) continue;
            f4 acc[NC];
#pragma unroll
            for (int c = 0; c < NC; c++) acc[c] = f4{0.0f, 0.0f, 0.0f, 0.0f};
            // the step's products at a raised wave priority, ahead of other
            // waves' fire updates and stores on the SIMD
            __builtin_amdgcn_s_setprio(2);
#pragma unroll
            for (int kb = 0; kb < KB; kb++) {
                const h8 a = frag_ind(A[j][kb]);
#pragma unroll
                for (int c = 0; c < NC; c++)
#pragma unroll
                    for (int k = 0; k < NP; k++)
                        acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bw[c][kb][k], acc[c], 0, 0, 0);
            }
            __builtin_amdgcn_s_setprio(0);
            // the operands of step t + D replace this step's
            if (t + D < g.T) load_step(t + D, A[j]);
#pragma unroll
            for (int c = 0; c < NC; c++) {
                uint32_t sp = 0u;
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    const float v = V[c][e] + acc[c][e];
                    const bool f = v > theta;
                    V[c][e] = f ? 0.0f : v;
                    cnt[c][e] += f ? 1 : 0;
                    sp |= (f ? 1u : 0u) << (8 * e);
                }
                const int m = 16 * c + (lane & 15);
                *reinterpret_cast<uint32_t *>(lds + (size_t)((h * D + j) * NC * 16 + m) * kRRow + my_col) = sp;
            }
        }
        // this batch is staged: every wave writes it out (the other buffer,
        // flushed after the previous barrier, is free for the next batch)
        __syncthreads();
        flush(h, t0, min(D, g.T - t0));
    }
    const int q0 = tile * 16 + 4 * (lane >> 4);
#pragma unroll
    for (int c = 0; c < NC; c++) {
        const int o = 16 * (ct0 + c) + (lane & 15);
        if (o >= g.Co) continue;
#pragma unroll
        for (int e = 0; e < 4; e++) {
            const int q = q0 + e;
            if (q >= g.P) continue;
            const int bi = q / g.HoWo, ri = q - bi * g.HoWo;
            counts[((size_t)bi * g.Co + o) * g.HoWo + ri] = cnt[c][e];
        }
    }
}

// Launch table of k_rate_conv16 over KB = 1..kMaxKB for (NC, NP) = (1, 1)
// and (1, 2), KB = 1..9 for (2, 1); D = steps in flight, min(8, 60 / KB).
typedef void (*Rate16Fn)(dim3, hipStream_t, const uint8_t *, const h8 *, const RGeom &, float, uint8_t *,
                         int32_t *);

template <int KB, int NC, int NP>
void launch_rate16(dim3 grid, hipStream_t s, const uint8_t *x8, const h8 *bp, const RGeom &g, float theta,
                   uint8_t *out, int32_t *counts)
{
    constexpr int D = 60 / KB < 8 ? 60 / KB : 8;
    const size_t lds = (size_t)2 * D * NC * 16 * kRRow;
    const void *fn = reinterpret_cast<const void *>(k_rate_conv16<KB, NC, NP, D>);
    if (lds > 64 * 1024) (void)hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL((k_rate_conv16<KB, NC, NP, D>), grid, dim3(64 * kRW), lds, s, x8, bp, g, theta, out,
                       counts);
}

template <int NC, int NP, int... KBs>
constexpr std::array<Rate16Fn, sizeof...(KBs)> rate16_table(std::integer_sequence<int, KBs...>)
{
    return {&launch_rate16<KBs + 1, NC, NP>...};
}

const auto kRate16_11 = rate16_table<1, 1>(std::make_integer_sequence<int, kMaxKB>{});
const auto kRate16_21 = rate16_table<2, 1>(std::make_integer_sequence<int, 9>{});
const auto kRate16_12 = rate16_table<1, 2>(std::make_integer_sequence<int, kMaxKB>{});

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

// One thread per output neuron and chunk of kPoolTT steps (blockIdx.y): the
// window's neuron with the most spikes (first in row-major order among
// equals) passes its train on; chunk 0 also writes the count.
constexpr int kPoolTT = 64;

__global__ void k_rate_pool(const uint8_t *__restrict__ in, const int32_t *__restrict__ cin, int B,
                            int T, int C, int Hi, int Wi, int Kh, int Kw, int stride, int pad, int Ho,
                            int Wo, uint8_t *__restrict__ out, int32_t *__restrict__ cout)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)B * C * Ho * Wo) return;
    const int t0 = blockIdx.y * kPoolTT;
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
    if (t0 == 0) cout[i] = best < 0 ? 0 : best;
    const int b = (int)(bc / C), c = (int)(bc - (int64_t)b * C);
    // the chunk's loads first (clamped step, winner or pixel 0), then the stores
    const int sy = by < 0 ? 0 : by, sx = by < 0 ? 0 : bx;
    uint8_t v[kPoolTT];
#pragma unroll
    for (int k = 0; k < kPoolTT; k++) {
        const int t = min(t0 + k, T - 1);
        v[k] = in[(((size_t)b * T + t) * C + c) * Hi * Wi + (size_t)sy * Wi + sx];
    }
#pragma unroll
    for (int k = 0; k < kPoolTT; k++) {
        const int t = t0 + k;
        if (t >= T) break;
        out[(((size_t)b * T + t) * C + c) * Ho * Wo + (size_t)yo * Wo + xo] = by < 0 ? 0 : v[k];
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
    const unsigned ty = (unsigned)((T + kRateTT - 1) / kRateTT);
    if (n % 4 == 0 && ((uintptr_t)u % 16) == 0 && ((uintptr_t)frames % 4) == 0)
        hipLaunchKernelGGL(k_rate_frames<true>, dim3((unsigned)((n / 4 + 255) / 256), ty, B), dim3(256), 0, s, x, u,
                           n, T, min_value, m, frames);
    else
        hipLaunchKernelGGL(k_rate_frames<false>, dim3((unsigned)((n + 255) / 256), ty, B), dim3(256), 0, s, x, u, n,
                           T, min_value, m, frames);
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
    if (rate16_nc(g, np) > 0)
        return rate_x8_bytes(g) + spk::align_up((size_t)g.NT16 * g.KB * np * 64 * sizeof(h8), 256);
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
    g.vec = (g.HoWo % 4 == 0) && ((uintptr_t)out_frames % 4 == 0);
    hipStream_t s = spk::stream_of(stream);
    const int nc = rate16_nc(g, np);
    if (nc > 0) {
        const size_t xb = rate_x8_bytes(g);
        const size_t need = xb + spk::align_up((size_t)g.NT16 * g.KB * np * 64 * sizeof(h8), 256);
        SPK_REQUIRE(ws_bytes >= need, SPK_E_WORKSPACE, "spk_conv_if_rate: workspace %zu < %zu bytes",
                    ws_bytes, need);
        SPK_REQUIRE_WS_ALIGNED(ws, "spk_conv_if_rate");
        SPK_REQUIRE((g.NT16 + nc - 1) / nc <= 65535, SPK_E_SHAPE, "spk_conv_if_rate: Co=%d too large", Co);
        uint8_t *x8 = static_cast<uint8_t *>(ws);
        h8 *bp = reinterpret_cast<h8 *>(x8 + xb);
        const size_t fbytes = (size_t)Ci * Hi * Wi;
        if (fbytes <= 48 * 1024 && (B * T) <= 0x7fffffff / 2) {
            if (fbytes % 4 == 0 && ((uintptr_t)frames % 4) == 0)
                hipLaunchKernelGGL(k_rate_pack8_lds<true>, dim3((unsigned)(B * T)), dim3(256), fbytes, s, frames, g,
                                   reinterpret_cast<uint2 *>(x8));
            else
                hipLaunchKernelGGL(k_rate_pack8_lds<false>, dim3((unsigned)(B * T)), dim3(256), fbytes, s, frames, g,
                                   reinterpret_cast<uint2 *>(x8));
        } else {
            hipLaunchKernelGGL(k_rate_pack8, dim3((unsigned)((g.Hp * g.Wp + 255) / 256), (unsigned)(B * T)), dim3(256),
                               0, s, frames, g, reinterpret_cast<uint2 *>(x8));
        }
        const int64_t nf = (int64_t)g.NT16 * g.KB * np * 64;
        if (half_w)
            hipLaunchKernelGGL((k_rate_pack_w16<1, true>), dim3((unsigned)((nf + 255) / 256)), dim3(256), 0, s, w, g, bp);
        else
            hipLaunchKernelGGL((k_rate_pack_w16<2, false>), dim3((unsigned)((nf + 255) / 256)), dim3(256), 0, s, w, g, bp);
        const int ptiles = (g.P + 15) / 16;
        const dim3 grid((unsigned)((ptiles + kRW - 1) / kRW), (unsigned)((g.NT16 + nc - 1) / nc));
        const Rate16Fn fn = np == 2 ? kRate16_12[g.KB - 1] : nc == 2 ? kRate16_21[g.KB - 1] : kRate16_11[g.KB - 1];
        fn(grid, s, x8, bp, g, theta, out_frames, counts);
        SPK_LAUNCHED("spk_conv_if_rate");
        return SPK_OK;
    }
    g.ntb = rate_ntb(g, np);
    SPK_REQUIRE(g.ntb > 0, SPK_E_UNSUPPORTED, "spk_conv_if_rate: %d weight slices do not fit LDS", g.SK);
    SPK_REQUIRE(g.NT <= 65535 * g.ntb, SPK_E_SHAPE, "spk_conv_if_rate: Co=%d too large", Co);
    const size_t xb = rate_xp_bytes(g);
    const size_t need = xb + spk::align_up((size_t)g.NT * g.SK * np * 64 * sizeof(h8), 256);
    SPK_REQUIRE(ws_bytes >= need, SPK_E_WORKSPACE, "spk_conv_if_rate: workspace %zu < %zu bytes",
                ws_bytes, need);
    SPK_REQUIRE_WS_ALIGNED(ws, "spk_conv_if_rate");
    uint16_t *fp = static_cast<uint16_t *>(ws);
    h8 *bp = reinterpret_cast<h8 *>(static_cast<uint8_t *>(ws) + xb);
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
    SPK_REQUIRE(n < (1ll << 31) && (T + kPoolTT - 1) / kPoolTT <= 65535, SPK_E_SHAPE,
                "spk_rate_pool: B*C*Ho*Wo or T too large");
    const dim3 grid((unsigned)((n + 255) / 256), (unsigned)((T + kPoolTT - 1) / kPoolTT));
    hipLaunchKernelGGL(k_rate_pool, grid, dim3(256), 0, spk::stream_of(stream), in_frames, in_counts, B, T, C,
                       Hi, Wi, Kh, Kw, stride, pad, Ho, Wo, out_frames, out_counts);
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
