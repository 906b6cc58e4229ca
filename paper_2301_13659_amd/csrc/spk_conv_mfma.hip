// spk_conv_fire on the matrix cores (Spyker §II-E.1, Eq. 2): implicit GEMM.
//
//   rows  M = output positions (b, y, x), 16 per MFMA tile
//   depth K = taps (c, ky, kx) of the kernel, 32 per MFMA step
//   cols  N = output maps o, 16 per MFMA tile
//
// The input is a uint8 first-spike-time map, so frame t is S_t = [time <= t]
// and a frame differs from the previous one only by the spikes arriving at t.
// Each wave gathers the time bytes of its A fragments once, then walks the
// steps t = 0..T-1 carrying the potentials in the MFMA accumulators:
// V_t = V_{t-1} + W * [time == t].  The indicator [time == t] is built in
// fp16 from the cached bytes (two packed-half instructions per register),
// and a (step, K-subtile) pair in which no input of the fragment arrives is
// skipped entirely (bit masks over t, reduced across the wave once).  After
// every step the epilogue compares the accumulators with theta and writes the
// first crossing (time and potential) of every neuron once.
//
// Binary spikes times fp16 weights are exact products.  Float master weights
// are split w = hi + lo with hi = f16(w), lo = f16(w - hi) (about 22
// significant bits) and take two MFMAs; half weights take one.
//
// Readout layers (theta = +inf, potentials not requested) only need V at the
// last step: a split-K GEMM on the final frame S_{T-1} = [time <= T-1] with
// deterministic partial sums in the workspace, reduced in a fixed order.
#include <hip/hip_fp16.h>

#include <algorithm>

#include "spk_internal.h"

namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr uint32_t kSelLo = 0x04010400u;  // bytes 0,1 -> halves 1024 + b
constexpr uint32_t kSelHi = 0x04030402u;  // bytes 2,3 -> halves 1024 + b
constexpr size_t kLdsLimit = 150 * 1024;
constexpr int kHaloSentinel = 16;  // bytes of 255 in front of a staged halo

struct Geom {
    int B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo;
    int K;  // Ci*Kh*Kw
    int S;  // ceil(K / 32)
    int P;  // B*Ho*Wo
};

__device__ __forceinline__ h2 as_h2(uint32_t u) { return __builtin_bit_cast(h2, u); }
__device__ __forceinline__ uint32_t as_u(h2 h) { return __builtin_bit_cast(uint32_t, h); }

// [t == tau] for two time bytes, as halves (c = 1024 + tau in both halves).
__device__ __forceinline__ uint32_t arrive2(uint32_t x, uint32_t sel, h2 c)
{
    const h2 one = {(_Float16)1.0f, (_Float16)1.0f}, zero = {(_Float16)0.0f, (_Float16)0.0f};
    h2 d = as_h2(__builtin_amdgcn_perm(0x64646464u, x, sel)) - c;  // small exact integers
    h2 a = one - d * d;                                            // 1 at d == 0, <= 0 else
    return as_u(__builtin_elementwise_min(__builtin_elementwise_max(a, zero), one));
}

// [t <= last] for two time bytes (c = 1025 + last).
__device__ __forceinline__ uint32_t upto2(uint32_t x, uint32_t sel, h2 c)
{
    const h2 one = {(_Float16)1.0f, (_Float16)1.0f}, zero = {(_Float16)0.0f, (_Float16)0.0f};
    h2 a = c - as_h2(__builtin_amdgcn_perm(0x64646464u, x, sel));
    return as_u(__builtin_elementwise_min(__builtin_elementwise_max(a, zero), one));
}

__device__ __forceinline__ h8 frag_arrive(uint32_t x0, uint32_t x1, h2 c)
{
    u4 v = {arrive2(x0, kSelLo, c), arrive2(x0, kSelHi, c), arrive2(x1, kSelLo, c),
            arrive2(x1, kSelHi, c)};
    return __builtin_bit_cast(h8, v);
}

__device__ __forceinline__ h8 frag_upto(uint32_t x0, uint32_t x1, h2 c)
{
    u4 v = {upto2(x0, kSelLo, c), upto2(x0, kSelHi, c), upto2(x1, kSelLo, c), upto2(x1, kSelHi, c)};
    return __builtin_bit_cast(h8, v);
}

template <bool kHalfW>
__device__ __forceinline__ float weight(const void *wv, const Geom &g, int o, int k)
{
    if (o >= g.Co || k >= g.K) return 0.0f;
    size_t at = (size_t)o * g.K + k;
    if (kHalfW) return (float)reinterpret_cast<const _Float16 *>(wv)[at];
    return reinterpret_cast<const float *>(wv)[at];
}

// n / d for 0 <= n < 2^31 by a 64-bit multiply-high (d >= 1, magic from the
// host): with l = ceil(log2 d) and m = ceil(2^(31+l) / d), floor(n*m / 2^(31+l))
// equals floor(n / d) for every n < 2^31.
struct FastDiv {
    uint32_t d, shift;
    uint64_t m;
};

__host__ __device__ inline FastDiv make_fastdiv(uint32_t d)
{
    uint32_t l = 0;
    while ((1ull << l) < d) l++;
    const uint64_t two = 1ull << (31 + l);
    return FastDiv{d, 31 + l, (two + d - 1) / d};
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv &f)
{
    return (uint32_t)(((uint64_t)n * f.m) >> f.shift);  // n*m < 2^63
}

// The 8 weights of one B fragment lane (taps kb..kb+7 of map o), as hi/lo
// halves.  Branch-free: out-of-range taps load an in-range weight (index
// clamped) and are zeroed afterwards, so all loads issue back to back.
template <bool kHalfW>
__device__ __forceinline__ void load_b8(const void *wv, int K, int Co, int o, int kb, h8 &hi, h8 &lo)
{
    const int oc = min(o, Co - 1);
    float w[8];
#pragma unroll
    for (int j = 0; j < 8; j++) {
        const int k = min(kb + j, K - 1);
        const size_t at = (size_t)oc * K + k;
        w[j] = kHalfW ? (float)reinterpret_cast<const _Float16 *>(wv)[at]
                      : reinterpret_cast<const float *>(wv)[at];
    }
#pragma unroll
    for (int j = 0; j < 8; j++) {
        const float v = ((o < Co) & (kb + j < K)) ? w[j] : 0.0f;
        const _Float16 h = (_Float16)v;
        hi[j] = h;
        lo[j] = (_Float16)(v - (float)h);
    }
}

// Copy input rows into the block's halo: channels [c_lo, c_lo + nc), flattened
// (sample, row) input rows [rlo, rlo + NR), full width; layout [c][row][Wi].
// Eight loads per thread are issued before their stores (indices past the
// end are clamped to the last element, their stores skipped).
__device__ __forceinline__ void stage_halo(const uint8_t *__restrict__ in, int Ci, int Hi, int Wi,
                                           FastDiv fd_wi, FastDiv fd_nr, FastDiv fd_hi, int c_lo,
                                           int nc, int rlo, int NR, uint8_t *halo)
{
    const int total = nc * NR * Wi;
    const size_t per_sample = (size_t)Ci * Hi * Wi;
    for (int base = threadIdx.x; base < total; base += 8 * blockDim.x) {
        uint32_t v[8];
#pragma unroll
        for (int j = 0; j < 8; j++) {
            const uint32_t idx = (uint32_t)min(base + j * (int)blockDim.x, total - 1);
            const uint32_t row = fdiv(idx, fd_wi), ix = idx - row * Wi;
            const uint32_t c = fdiv(row, fd_nr), r = row - c * NR;
            const uint32_t fr = rlo + r, b = fdiv(fr, fd_hi), iy = fr - b * Hi;
            v[j] = in[b * per_sample + ((c_lo + c) * Hi + iy) * Wi + ix];
        }
#pragma unroll
        for (int j = 0; j < 8; j++) {
            const int idx = base + j * blockDim.x;
            if (idx < total) halo[idx] = (uint8_t)v[j];
        }
    }
}

// The tap tables of a lane's 8 taps kb..kb+7 (kb a multiple of 8), read as
// vectors: koff (8 x int32) and kyx (8 x int16, ky << 8 | kx, -1: padding).
__device__ __forceinline__ void load_taps8(const int *koff, const int16_t *kyx, int kb, int (&kof)[8],
                                          int (&kk)[8])
{
    const int4 a = *reinterpret_cast<const int4 *>(koff + kb);
    const int4 b = *reinterpret_cast<const int4 *>(koff + kb + 4);
    const int4 c = *reinterpret_cast<const int4 *>(kyx + kb);
    kof[0] = a.x; kof[1] = a.y; kof[2] = a.z; kof[3] = a.w;
    kof[4] = b.x; kof[5] = b.y; kof[6] = b.z; kof[7] = b.w;
    const uint32_t cw[4] = {(uint32_t)c.x, (uint32_t)c.y, (uint32_t)c.z, (uint32_t)c.w};
#pragma unroll
    for (int j = 0; j < 8; j++) kk[j] = (int)(int16_t)(cw[j >> 1] >> (16 * (j & 1)));
}

// Gather the 8 time bytes of a lane's A fragment (taps kb..kb+7) for the row
// whose window origin is (iy0, ix0) in sample b; 255 outside the input.
// Branch-free: taps outside the input load byte 0 of the input (gather8) or
// the sentinel in front of the halo (gather8_lds) and are forced to 255.
__device__ __forceinline__ void gather8(const uint8_t *__restrict__ in, const Geom &g,
                                       const int *koff, const int16_t *kyx, bool valid, int b,
                                       int iy0, int ix0, int kb, uint32_t &x0, uint32_t &x1)
{
    int kof[8], kk[8];
    load_taps8(koff, kyx, kb, kof, kk);
    const size_t base = (size_t)b * g.Ci * g.Hi * g.Wi + (ptrdiff_t)iy0 * g.Wi + ix0;
    uint32_t tb[8];
    bool inb[8];
#pragma unroll
    for (int j = 0; j < 8; j++) {
        const int iy = iy0 + (kk[j] >> 8), ix = ix0 + (kk[j] & 0xFF);
        inb[j] = valid & (kk[j] >= 0) & ((unsigned)iy < (unsigned)g.Hi) & ((unsigned)ix < (unsigned)g.Wi);
        tb[j] = in[inb[j] ? base + kof[j] : 0];
    }
    uint32_t w[2] = {0, 0};
#pragma unroll
    for (int j = 0; j < 8; j++) w[j >> 2] |= (inb[j] ? tb[j] : 255u) << (8 * (j & 3));
    x0 = w[0];
    x1 = w[1];
}

__device__ __forceinline__ void gather8_lds(const uint8_t *halo, const Geom &g, const int *koff,
                                           const int16_t *kyx, bool valid, int hbase, int iy0, int ix0,
                                           int kb, uint32_t &x0, uint32_t &x1)
{
    int kof[8], kk[8];
    load_taps8(koff, kyx, kb, kof, kk);
    uint32_t tb[8];
#pragma unroll
    for (int j = 0; j < 8; j++) {
        const int iy = iy0 + (kk[j] >> 8), ix = ix0 + (kk[j] & 0xFF);
        const bool inb =
            valid & (kk[j] >= 0) & ((unsigned)iy < (unsigned)g.Hi) & ((unsigned)ix < (unsigned)g.Wi);
        tb[j] = halo[inb ? kHaloSentinel + hbase + kof[j] : 0];
    }
    uint32_t w[2] = {0, 0};
#pragma unroll
    for (int j = 0; j < 8; j++) w[j >> 2] |= tb[j] << (8 * (j & 3));
    x0 = w[0];
    x1 = w[1];
}

// Bytes of the firing kernel's scratch region: the larger of the B fragments
// of one column group and the setup arrays (lane masks, then the halo).
__host__ __device__ inline size_t fire_scratch_bytes(int S, int C, int NP, int halo_cap)
{
    const size_t b = (size_t)S * C * NP * 64 * 16;
    const size_t setup = (size_t)kWaves * S * 64 * sizeof(uint32_t) + (size_t)halo_cap;
    return ((b > setup ? b : setup) + 15) / 16 * 16;
}

// ------------------------------------------------------------ firing layers
//
// Block: 4 waves, each owning R row tiles (16 positions each).  The A side is
// set up once per block: the input halo goes to LDS, every wave gathers the
// time bytes of its fragments ([r][s][lane], 8 bytes per lane) and builds one
// activity word per step t (bit s: some row of the wave has an arrival in
// subtile s at t).  The block then loops over its column groups (C column
// tiles each): stage the group's weights as ready B fragments, walk the steps
// carrying the potentials in the MFMA accumulators, write the crossings.
template <int R, int C, bool kHiLo, bool kHalfW>
__global__ __launch_bounds__(kThreads) void k_conv_fire_mfma(
    const uint8_t *__restrict__ in, const void *__restrict__ wv, Geom g, float theta, int halo_cap,
    FastDiv fd_wi, FastDiv fd_hi, int groups_per_block, uint8_t *__restrict__ out_t,
    float *__restrict__ out_v, float *__restrict__ pot)
{
    static_assert(R * C * 4 <= 32, "one bit per accumulator entry");
    constexpr int NP = kHiLo ? 2 : 1;
    extern __shared__ __align__(16) unsigned char lds[];
    // LDS: [scratch | koff | kyx | astage | act].  The scratch region holds the
    // setup-only arrays (lane masks, input halo) first and the B fragments
    // of the current column group afterwards.
    const size_t scratch = fire_scratch_bytes(g.S, C, NP, halo_cap);
    h8 *bfrag = reinterpret_cast<h8 *>(lds);                              // [S][C][NP][64]
    uint32_t *mstage_all = reinterpret_cast<uint32_t *>(lds);              // [wave][s][64]
    uint8_t *halo = lds + (size_t)kWaves * g.S * 64 * sizeof(uint32_t);
    int *koff = reinterpret_cast<int *>(lds + scratch);
    int16_t *kyx = reinterpret_cast<int16_t *>(koff + g.S * 32);
    uint2 *astage_all = reinterpret_cast<uint2 *>(kyx + g.S * 32);         // [wave][r][s][64]
    uint32_t *act_all = reinterpret_cast<uint32_t *>(astage_all + (size_t)kWaves * R * g.S * 64);

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int HoWo = g.Ho * g.Wo;

    // input rows of the block as one run of flattened (sample, row) rows
    const int pb0 = blockIdx.x * kWaves * 16 * R;
    const int pb1 = min(g.P, pb0 + kWaves * 16 * R) - 1;
    const int q0 = pb0 / g.Wo, q1 = pb1 / g.Wo;
    const int b0 = q0 / g.Ho, y0 = q0 - b0 * g.Ho, b1 = q1 / g.Ho, y1 = q1 - b1 * g.Ho;
    const int rlo = b0 * g.Hi + max(0, y0 * g.stride - g.pad);
    const int rhi = b1 * g.Hi + max(-1, min(g.Hi - 1, y1 * g.stride - g.pad + g.Kh - 1));
    const int NR = max(1, rhi - rlo + 1);
    const bool use_halo = (long long)g.Ci * NR * g.Wi + kHaloSentinel <= halo_cap;
    if (use_halo) {
        if (threadIdx.x < kHaloSentinel) halo[threadIdx.x] = 255u;
        stage_halo(in, g.Ci, g.Hi, g.Wi, fd_wi, make_fastdiv(NR), fd_hi, 0, g.Ci, rlo, NR,
                   halo + kHaloSentinel);
    }
    {
        const int KK = g.Kh * g.Kw, HiWi = g.Hi * g.Wi;
        for (int k = threadIdx.x; k < g.S * 32; k += blockDim.x) {
            if (k < g.K) {
                int c = k / KK, r = k - c * KK, ky = r / g.Kw, kx = r - ky * g.Kw;
                koff[k] = use_halo ? (c * NR + ky) * g.Wi + kx : c * HiWi + ky * g.Wi + kx;
                kyx[k] = (int16_t)((ky << 8) | kx);
            } else {
                koff[k] = 0;
                kyx[k] = -1;
            }
        }
    }
    __syncthreads();

    // ---- A side: gather, per-lane arrival masks, activity words
    uint2 *astage = astage_all + (size_t)wave * R * g.S * 64;
    uint32_t *act = act_all + wave * 32;
    uint32_t *mstage = mstage_all + (size_t)wave * g.S * 64;
    const bool masks = g.T <= 32 && g.S <= 32;
    const int m0 = (blockIdx.x * kWaves + wave) * 16 * R;
    const int kg = (lane >> 4) * 8;  // this lane's first tap inside a subtile
    for (int s = 0; s < g.S && masks; s++) mstage[s * 64 + lane] = 0u;
#pragma unroll
    for (int r = 0; r < R; r++) {
        const int p = m0 + r * 16 + (lane & 15);
        const bool valid = p < g.P;
        const int b = valid ? p / HoWo : 0, rem = p - b * HoWo;
        const int y = rem / g.Wo, x = rem - y * g.Wo;
        const int iy0 = y * g.stride - g.pad, ix0 = x * g.stride - g.pad;
        const int hbase = (b * g.Hi + iy0 - rlo) * g.Wi + ix0;
        for (int s = 0; s < g.S; s++) {
            uint32_t x0, x1;
            if (use_halo)
                gather8_lds(halo, g, koff, kyx, valid, hbase, iy0, ix0, s * 32 + kg, x0, x1);
            else
                gather8(in, g, koff, kyx, valid, b, iy0, ix0, s * 32 + kg, x0, x1);
            uint32_t m = 0u;
#pragma unroll
            for (int j = 0; j < 8; j++) {
                const uint32_t t = ((j < 4 ? x0 : x1) >> (8 * (j & 3))) & 0xFFu;
                m |= (t < (uint32_t)g.T) ? (1u << (t & 31)) : 0u;
            }
            astage[(r * g.S + s) * 64 + lane] = make_uint2(x0, x1);
            if (masks) mstage[s * 64 + lane] |= m;
        }
    }
    if (masks) {
        // lane s ORs the 64 lane masks of subtile s; a ballot per step then
        // turns the S x T bit matrix around into activity words
        uint32_t ms = 0u;
        if (lane < g.S)
            for (int l = 0; l < 64; l++) ms |= mstage[lane * 64 + l];
        for (int t = 0; t < g.T; t++) {
            const uint64_t bal = __ballot((ms >> t) & 1u);
            if (lane == 0) act[t] = (uint32_t)bal;
        }
    }
    __syncthreads();

    const uint64_t all_s = g.S >= 64 ? ~0ull : ((1ull << g.S) - 1ull);
    const int n_groups = (g.Co + 16 * C - 1) / (16 * C);
    const int grp0 = blockIdx.y * groups_per_block;
    const int grp1 = min(n_groups, grp0 + groups_per_block);
    for (int grp = grp0; grp < grp1; grp++) {
        const int o0 = grp * 16 * C;
        // ---- B side: this group's weights as ready fragments
        __syncthreads();  // setup arrays / previous group's fragments no longer read
#pragma unroll 4
        for (int e = threadIdx.x; e < g.S * C * 64; e += blockDim.x) {
            const int l = e & 63, sc = e >> 6, c = sc % C, s = sc / C;
            const int o = o0 + c * 16 + (l & 15), kb = s * 32 + (l >> 4) * 8;
            h8 hi, lo;
            load_b8<kHalfW>(wv, g.K, g.Co, o, kb, hi, lo);
            bfrag[(sc * NP) * 64 + l] = hi;
            if (kHiLo) bfrag[(sc * NP + 1) * 64 + l] = lo;
        }
        __syncthreads();

        uint32_t valid_bits = 0;
#pragma unroll
        for (int r = 0; r < R; r++)
#pragma unroll
            for (int c = 0; c < C; c++)
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const int p = m0 + r * 16 + (lane >> 4) * 4 + i, o = o0 + c * 16 + (lane & 15);
                    if (p < g.P && o < g.Co) valid_bits |= 1u << ((r * C + c) * 4 + i);
                }
        uint32_t live = valid_bits;  // dense-potential mode: not yet fired

        f4 acc[R][C];
#pragma unroll
        for (int r = 0; r < R; r++)
#pragma unroll
            for (int c = 0; c < C; c++) acc[r][c] = f4{0.0f, 0.0f, 0.0f, 0.0f};

        for (int tau = 0; tau < g.T; tau++) {
            const _Float16 ct = (_Float16)(float)(1024 + tau);
            const h2 cc = {ct, ct};
            uint64_t sm = all_s;
            // (through uint32_t: the int the builtin returns must not sign-extend
            // subtile 31 into bits 32..63)
            if (masks) sm = (uint32_t)__builtin_amdgcn_readfirstlane(act[tau]);
            // Walk the active subtiles with the operands of the next one already
            // in flight (two register sets used in turn).
            h8 bh0[C], bl0[C], bh1[C], bl1[C];
            uint2 ax0[R], ax1[R];
            auto load_ops = [&](int s, h8 (&bh)[C], h8 (&bl)[C], uint2 (&ax)[R]) {
#pragma unroll
                for (int c = 0; c < C; c++) {
                    bh[c] = bfrag[((s * C + c) * NP) * 64 + lane];
                    if (kHiLo) bl[c] = bfrag[((s * C + c) * NP + 1) * 64 + lane];
                }
#pragma unroll
                for (int r = 0; r < R; r++) ax[r] = astage[(r * g.S + s) * 64 + lane];
            };
            auto compute = [&](const h8 (&bh)[C], const h8 (&bl)[C], const uint2 (&ax)[R]) {
                h8 af[R];
#pragma unroll
                for (int r = 0; r < R; r++) af[r] = frag_arrive(ax[r].x, ax[r].y, cc);
#pragma unroll
                for (int r = 0; r < R; r++)
#pragma unroll
                    for (int c = 0; c < C; c++)
                        acc[r][c] =
                            __builtin_amdgcn_mfma_f32_16x16x32_f16(af[r], bh[c], acc[r][c], 0, 0, 0);
                if (kHiLo) {
#pragma unroll
                    for (int r = 0; r < R; r++)
#pragma unroll
                        for (int c = 0; c < C; c++)
                            acc[r][c] =
                                __builtin_amdgcn_mfma_f32_16x16x32_f16(af[r], bl[c], acc[r][c], 0, 0, 0);
                }
            };
            if (sm) {
                int s0 = __builtin_ctzll(sm);
                sm &= sm - 1;
                load_ops(s0, bh0, bl0, ax0);
                while (true) {
                    if (sm) {
                        const int s1 = __builtin_ctzll(sm);
                        sm &= sm - 1;
                        load_ops(s1, bh1, bl1, ax1);
                        compute(bh0, bl0, ax0);
                    } else {
                        compute(bh0, bl0, ax0);
                        break;
                    }
                    if (sm) {
                        const int s2 = __builtin_ctzll(sm);
                        sm &= sm - 1;
                        load_ops(s2, bh0, bl0, ax0);
                        compute(bh1, bl1, ax1);
                    } else {
                        compute(bh1, bl1, ax1);
                        break;
                    }
                }
            }
            if (pot) {
                // dense potentials: every V_t out, crossings tracked with live bits
#pragma unroll
                for (int r = 0; r < R; r++)
#pragma unroll
                    for (int c = 0; c < C; c++)
#pragma unroll
                        for (int i = 0; i < 4; i++) {
                            const int bit = (r * C + c) * 4 + i;
                            if (!((valid_bits >> bit) & 1u)) continue;
                            const float v = acc[r][c][i];
                            const int p = m0 + r * 16 + (lane >> 4) * 4 + i, o = o0 + c * 16 + (lane & 15);
                            const int b = p / HoWo, rem = p - b * HoWo;
                            pot[((size_t)(b * g.T + tau) * g.Co + o) * HoWo + rem] = v;
                            if (v > theta && ((live >> bit) & 1u)) {
                                const size_t n = ((size_t)b * g.Co + o) * HoWo + rem;
                                out_t[n] = (uint8_t)tau;
                                out_v[n] = v;
                                live &= ~(1u << bit);
                            }
                        }
            } else {
                // fired neurons hold -inf, so the largest accumulator tells whether
                // anything new crossed theta at this step
                float mx = -INFINITY;
#pragma unroll
                for (int r = 0; r < R; r++)
#pragma unroll
                    for (int c = 0; c < C; c++)
#pragma unroll
                        for (int i = 0; i < 4; i++) mx = fmaxf(mx, acc[r][c][i]);
                if (__ballot(mx > theta)) {
#pragma unroll
                    for (int r = 0; r < R; r++)
#pragma unroll
                        for (int c = 0; c < C; c++)
#pragma unroll
                            for (int i = 0; i < 4; i++) {
                                const float v = acc[r][c][i];
                                if (v > theta) {
                                    const int bit = (r * C + c) * 4 + i;
                                    if ((valid_bits >> bit) & 1u) {
                                        const int p = m0 + r * 16 + (lane >> 4) * 4 + i;
                                        const int o = o0 + c * 16 + (lane & 15);
                                        const int b = p / HoWo, rem = p - b * HoWo;
                                        const size_t n = ((size_t)b * g.Co + o) * HoWo + rem;
                                        out_t[n] = (uint8_t)tau;
                                        out_v[n] = v;
                                    }
                                    acc[r][c][i] = -INFINITY;
                                }
                            }
                }
            }
        }
        // neurons that never fired: NEVER and the last potential
#pragma unroll
        for (int r = 0; r < R; r++)
#pragma unroll
            for (int c = 0; c < C; c++)
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const int bit = (r * C + c) * 4 + i;
                    const float v = acc[r][c][i];
                    const bool fired = pot ? !((live >> bit) & 1u) : (v == -INFINITY);
                    if (((valid_bits >> bit) & 1u) && !fired) {
                        const int p = m0 + r * 16 + (lane >> 4) * 4 + i, o = o0 + c * 16 + (lane & 15);
                        const int b = p / HoWo, rem = p - b * HoWo;
                        const size_t n = ((size_t)b * g.Co + o) * HoWo + rem;
                        out_t[n] = (uint8_t)spk::kNever;
                        out_v[n] = v;
                    }
                }
    }
}

// ----------------------------------------------------------- readout layers
//
// Only V at the last step is needed: a GEMM on the final frame
// [time <= T-1].  Block = 4 waves x R row tiles over C column tiles and one
// K split (a run of subtiles); the split's weights are staged in LDS as B
// fragments, A fragments are gathered straight into registers.  Partial sums
// go to part[split][Co][P] and are reduced in split order.
template <int R, int C, bool kHiLo, bool kHalfW>
__global__ __launch_bounds__(kThreads) void k_conv_readout_mfma(
    const uint8_t *__restrict__ in, const void *__restrict__ wv, Geom g, int s_per_split,
    int halo_cap, FastDiv fd_wi, FastDiv fd_hi, float *__restrict__ part)
{
    constexpr int NP = kHiLo ? 2 : 1;
    extern __shared__ __align__(16) unsigned char lds[];
    const int split = blockIdx.z;
    const int s0 = split * s_per_split, ns = min(g.S, s0 + s_per_split) - s0;
    h8 *bfrag = reinterpret_cast<h8 *>(lds);                              // [ns][C][NP][64]
    int *koff = reinterpret_cast<int *>(lds + (size_t)s_per_split * C * NP * 64 * sizeof(h8));
    int16_t *kyx = reinterpret_cast<int16_t *>(koff + s_per_split * 32);
    uint8_t *halo = reinterpret_cast<uint8_t *>(kyx + s_per_split * 32);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int o0 = blockIdx.y * 16 * C;
    const int KK = g.Kh * g.Kw, HiWi = g.Hi * g.Wi, HoWo = g.Ho * g.Wo;

    // the split's input channels and the block's input rows
    const int k_first = s0 * 32, k_last = min(g.K, (s0 + ns) * 32) - 1;
    const int c_lo = k_first / KK, nc = k_last / KK - c_lo + 1;
    const int pb0 = blockIdx.x * kWaves * 16 * R;
    const int pb1 = min(g.P, pb0 + kWaves * 16 * R) - 1;
    const int q0 = pb0 / g.Wo, q1 = pb1 / g.Wo;
    const int b0 = q0 / g.Ho, y0 = q0 - b0 * g.Ho, b1 = q1 / g.Ho, y1 = q1 - b1 * g.Ho;
    const int rlo = b0 * g.Hi + max(0, y0 * g.stride - g.pad);
    const int rhi = b1 * g.Hi + max(-1, min(g.Hi - 1, y1 * g.stride - g.pad + g.Kh - 1));
    const int NR = max(1, rhi - rlo + 1);
    const bool use_halo = (long long)nc * NR * g.Wi + kHaloSentinel <= halo_cap;
    if (use_halo) {
        if (threadIdx.x < kHaloSentinel) halo[threadIdx.x] = 255u;
        stage_halo(in, g.Ci, g.Hi, g.Wi, fd_wi, make_fastdiv(NR), fd_hi, c_lo, nc, rlo, NR,
                   halo + kHaloSentinel);
    }
    for (int kl = threadIdx.x; kl < ns * 32; kl += blockDim.x) {
        const int k = s0 * 32 + kl;
        if (k < g.K) {
            int c = k / KK, rr = k - c * KK, ky = rr / g.Kw, kx = rr - ky * g.Kw;
            koff[kl] = use_halo ? ((c - c_lo) * NR + ky) * g.Wi + kx : c * HiWi + ky * g.Wi + kx;
            kyx[kl] = (int16_t)((ky << 8) | kx);
        } else {
            koff[kl] = 0;
            kyx[kl] = -1;
        }
    }
#pragma unroll 4
    for (int e = threadIdx.x; e < ns * C * 64; e += blockDim.x) {
        const int l = e & 63, sc = e >> 6, c = sc % C, s = sc / C;
        const int o = o0 + c * 16 + (l & 15), kb = (s0 + s) * 32 + (l >> 4) * 8;
        h8 hi, lo;
        load_b8<kHalfW>(wv, g.K, g.Co, o, kb, hi, lo);
        bfrag[(sc * NP) * 64 + l] = hi;
        if (kHiLo) bfrag[(sc * NP + 1) * 64 + l] = lo;
    }
    __syncthreads();

    const int m0 = (blockIdx.x * kWaves + wave) * 16 * R;
    const float last = (float)(1025 + g.T - 1);
    const h2 cc = {(_Float16)last, (_Float16)last};
    int rb[R], riy[R], rix[R], rh[R];
    bool rvalid[R];
#pragma unroll
    for (int r = 0; r < R; r++) {
        const int p = m0 + r * 16 + (lane & 15);
        rvalid[r] = p < g.P;
        const int b = rvalid[r] ? p / HoWo : 0, rem = p - b * HoWo;
        const int y = rem / g.Wo, x = rem - y * g.Wo;
        rb[r] = b;
        riy[r] = y * g.stride - g.pad;
        rix[r] = x * g.stride - g.pad;
        rh[r] = (b * g.Hi + riy[r] - rlo) * g.Wi + rix[r];
    }
    f4 acc[R][C];
#pragma unroll
    for (int r = 0; r < R; r++)
#pragma unroll
        for (int c = 0; c < C; c++) acc[r][c] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    for (int s = 0; s < ns; s++) {
        h8 bh[C], bl[C];
#pragma unroll
        for (int c = 0; c < C; c++) {
            bh[c] = bfrag[((s * C + c) * NP) * 64 + lane];
            if (kHiLo) bl[c] = bfrag[((s * C + c) * NP + 1) * 64 + lane];
        }
#pragma unroll
        for (int r = 0; r < R; r++) {
            uint32_t x0, x1;
            if (use_halo)
                gather8_lds(halo, g, koff, kyx, rvalid[r], rh[r], riy[r], rix[r], s * 32 + (lane >> 4) * 8,
                            x0, x1);
            else
                gather8(in, g, koff, kyx, rvalid[r], rb[r], riy[r], rix[r], s * 32 + (lane >> 4) * 8, x0,
                        x1);
            const h8 av8 = frag_upto(x0, x1, cc);
#pragma unroll
            for (int c = 0; c < C; c++)
                acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av8, bh[c], acc[r][c], 0, 0, 0);
            if (kHiLo) {
#pragma unroll
                for (int c = 0; c < C; c++)
                    acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av8, bl[c], acc[r][c], 0, 0, 0);
            }
        }
    }
#pragma unroll
    for (int r = 0; r < R; r++)
#pragma unroll
        for (int c = 0; c < C; c++)
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int p = m0 + r * 16 + (lane >> 4) * 4 + i, o = o0 + c * 16 + (lane & 15);
                if (p < g.P && o < g.Co) part[((size_t)split * g.Co + o) * g.P + p] = acc[r][c][i];
            }
}

__global__ void k_readout_reduce(const float *__restrict__ part, Geom g, int splits,
                                 uint8_t *__restrict__ out_t, float *__restrict__ out_v)
{
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;  // o * P + p
    const long long n = (long long)g.Co * g.P;
    if (i >= n) return;
    float v = 0.0f;
    for (int s = 0; s < splits; s++) v += part[(size_t)s * n + i];
    const int o = (int)(i / g.P), p = (int)(i - (long long)o * g.P);
    const int HoWo = g.Ho * g.Wo, b = p / HoWo, rem = p - b * HoWo;
    const size_t at = ((size_t)b * g.Co + o) * HoWo + rem;
    out_t[at] = (uint8_t)spk::kNever;
    out_v[at] = v;
}

// ------------------------------------------------------------ dispatch

struct Plan {
    int R, C;
    size_t lds;
    int halo;  // bytes of input halo staged in LDS (0: gather from global memory)
};

// LDS bytes of the firing kernel for a given halo size (0: no halo).
size_t fire_lds(const Geom &g, int R, int C, bool hilo, int halo)
{
    return fire_scratch_bytes(g.S, C, hilo ? 2 : 1, halo) +
           (size_t)g.S * 32 * (sizeof(int) + sizeof(int16_t)) +
           (size_t)kWaves * R * g.S * 64 * sizeof(uint2) + (size_t)kWaves * 32 * sizeof(uint32_t);
}

// Largest input halo (bytes) of any block of kWaves*16*R positions; mirrors
// the row range the kernel computes.
long long max_halo(const Geom &g, int R)
{
    const int per = kWaves * 16 * R;
    long long best = 0;
    for (int pb0 = 0; pb0 < g.P; pb0 += per) {
        const int pb1 = std::min(g.P, pb0 + per) - 1;
        const int q0 = pb0 / g.Wo, q1 = pb1 / g.Wo;
        const int b0 = q0 / g.Ho, y0 = q0 - b0 * g.Ho, b1 = q1 / g.Ho, y1 = q1 - b1 * g.Ho;
        const int rlo = b0 * g.Hi + std::max(0, y0 * g.stride - g.pad);
        const int rhi = b1 * g.Hi + std::max(-1, std::min(g.Hi - 1, y1 * g.stride - g.pad + g.Kh - 1));
        best = std::max(best, (long long)g.Ci * std::max(1, rhi - rlo + 1) * g.Wi);
    }
    return best;
}

bool plan_fire(const Geom &g, bool hilo, Plan &pl)
{
    // Candidate tiles per wave (row tiles R x column tiles C), best first;
    // R*C <= 4 keeps the accumulators small enough for 3+ waves per SIMD.
    // First choice: a plan whose LDS, input halo included, lets two blocks
    // share a CU; then any plan with the halo; then one that gathers from
    // global memory (no halo).
    static const int cand[][2] = {{2, 2}, {1, 4}, {2, 1}, {1, 2}, {1, 1}};
    const int col_tiles = (g.Co + 15) / 16;
    for (int pass = 0; pass < 3; pass++) {
        const size_t cap = pass == 0 ? 80 * 1024 : kLdsLimit;
        for (const auto &rc : cand) {
            const int R = rc[0], C = rc[1];
            if (C > 1 && col_tiles < C) continue;          // no empty column tiles
            const int halo = pass < 2 && g.P > 0 ? (int)(max_halo(g, R) + kHaloSentinel) : 0;
            const size_t lds = fire_lds(g, R, C, hilo, halo);
            if (lds <= cap) {
                pl = Plan{R, C, lds, halo};
                return true;
            }
        }
    }
    return false;
}

template <typename K>
void allow_lds(K kern, size_t lds)
{
    if (lds > 64 * 1024)
        (void)hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
}

template <int R, int C>
spk_status launch_fire_rc(bool half_w, const uint8_t *in, const void *w, const Geom &g, float th,
                          uint8_t *ot, float *ov, float *pot, const Plan &pl, hipStream_t s)
{
    // Column groups per block: the A-side setup is shared by a block's groups,
    // so give each block as many as keeps >= ~1024 blocks in flight.
    const int pos_blocks = spk::ceil_div(g.P, kWaves * 16 * R);
    const int n_groups = spk::ceil_div(g.Co, 16 * C);
    int per = n_groups;
    while (per > 1 && (long long)pos_blocks * spk::ceil_div(n_groups, per) < 1024) per = (per + 1) / 2;
    dim3 grid(pos_blocks, spk::ceil_div(n_groups, per));
    if (half_w) {
        auto kern = k_conv_fire_mfma<R, C, false, true>;
        allow_lds(kern, pl.lds);
        hipLaunchKernelGGL(kern, grid, dim3(kThreads), pl.lds, s, in, w, g, th, pl.halo,
                           make_fastdiv(g.Wi), make_fastdiv(g.Hi), per, ot, ov, pot);
    } else {
        auto kern = k_conv_fire_mfma<R, C, true, false>;
        allow_lds(kern, pl.lds);
        hipLaunchKernelGGL(kern, grid, dim3(kThreads), pl.lds, s, in, w, g, th, pl.halo,
                           make_fastdiv(g.Wi), make_fastdiv(g.Hi), per, ot, ov, pot);
    }
    return spk::check_launch("spk_conv_fire");
}

constexpr int kRoR = 2;

int readout_splits(int S) { return S >= 128 ? 8 : (S >= 32 ? 4 : (S >= 8 ? 2 : 1)); }

// Largest halo (bytes) of any readout block: its rows times the channels a
// K split of `per` subtiles can touch.
long long max_halo_readout(const Geom &g, int R, int per)
{
    const int KK = g.Kh * g.Kw;
    const int nc = std::min(g.Ci, (per * 32 + KK - 1) / KK + 1);
    return max_halo(g, R) / std::max(1, g.Ci) * nc;
}

template <int C>
spk_status launch_readout_c(bool half_w, const uint8_t *in, const void *w, const Geom &g,
                            float *part, int splits, hipStream_t s)
{
    const int per = (g.S + splits - 1) / splits;
    size_t lds = (size_t)per * C * (half_w ? 1 : 2) * 64 * sizeof(h8) +
                 (size_t)per * 32 * (sizeof(int) + sizeof(int16_t));
    int halo = 0;
    const long long need = max_halo_readout(g, kRoR, per) + kHaloSentinel;
    if (lds + need <= kLdsLimit) halo = (int)need;
    lds += spk::align_up((size_t)halo, 16);
    dim3 grid(spk::ceil_div(g.P, kWaves * 16 * kRoR), spk::ceil_div(g.Co, 16 * C), splits);
    if (half_w) {
        auto kern = k_conv_readout_mfma<kRoR, C, false, true>;
        allow_lds(kern, lds);
        hipLaunchKernelGGL(kern, grid, dim3(kThreads), lds, s, in, w, g, per, halo, make_fastdiv(g.Wi),
                           make_fastdiv(g.Hi), part);
    } else {
        auto kern = k_conv_readout_mfma<kRoR, C, true, false>;
        allow_lds(kern, lds);
        hipLaunchKernelGGL(kern, grid, dim3(kThreads), lds, s, in, w, g, per, halo, make_fastdiv(g.Wi),
                           make_fastdiv(g.Hi), part);
    }
    return spk::check_launch("spk_conv_fire");
}

}  // namespace

namespace spk {

bool conv_mfma_supported(int Ci, int Kh, int Kw, int Co, bool half_w, bool readout)
{
    if (Kh > 127 || Kw > 127) return false;  // taps are packed as (ky << 8 | kx) in int16
    Geom g{};
    g.K = Ci * Kh * Kw;
    g.S = (g.K + 31) / 32;
    g.Co = Co;
    g.P = 0;  // shape-only question: no halo sizing (it needs the real geometry)
    if (readout) {
        const int per = (g.S + readout_splits(g.S) - 1) / readout_splits(g.S);
        return (size_t)per * 2 * 64 * sizeof(h8) <= kLdsLimit;
    }
    Plan pl;
    return plan_fire(g, !half_w, pl);
}

size_t conv_mfma_workspace(int B, int Ho, int Wo, int Co, int K, bool readout)
{
    if (!readout) return 0;
    return align_up((size_t)readout_splits((K + 31) / 32) * Co * B * Ho * Wo * sizeof(float), 256);
}

spk_status conv_fire_mfma(const uint8_t *in, int B, int T, int Ci, int Hi, int Wi, const void *w,
                          bool half_w, int Co, int Kh, int Kw, int stride, int pad, int Ho, int Wo,
                          float theta, uint8_t *out_t, float *out_v, float *pot, void *ws,
                          hipStream_t s)
{
    Geom g{B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo, Ci * Kh * Kw, 0, B * Ho * Wo};
    g.S = (g.K + 31) / 32;
    const bool readout = !(theta <= 3.4e38f) && !pot;
    if (readout) {
        const int splits = readout_splits(g.S);
        float *part = reinterpret_cast<float *>(ws);
        spk_status st = g.Co <= 16 ? launch_readout_c<1>(half_w, in, w, g, part, splits, s)
                                   : launch_readout_c<2>(half_w, in, w, g, part, splits, s);
        if (st != SPK_OK) return st;
        const long long n = (long long)g.Co * g.P;
        hipLaunchKernelGGL(k_readout_reduce, dim3(ceil_div(n, 256)), dim3(256), 0, s, part, g,
                           splits, out_t, out_v);
        return check_launch("spk_conv_fire");
    }
    Plan pl;
    if (!plan_fire(g, !half_w, pl)) {
        set_error("spk_conv_fire: no matrix-core plan for K=%d", g.K);
        return SPK_E_UNSUPPORTED;
    }
    switch (pl.R * 10 + pl.C) {
    case 11: return launch_fire_rc<1, 1>(half_w, in, w, g, theta, out_t, out_v, pot, pl, s);
    case 12: return launch_fire_rc<1, 2>(half_w, in, w, g, theta, out_t, out_v, pot, pl, s);
    case 14: return launch_fire_rc<1, 4>(half_w, in, w, g, theta, out_t, out_v, pot, pl, s);
    case 21: return launch_fire_rc<2, 1>(half_w, in, w, g, theta, out_t, out_v, pot, pl, s);
    default: return launch_fire_rc<2, 2>(half_w, in, w, g, theta, out_t, out_v, pot, pl, s);
    }
}

}  // namespace spk
