// spk_inhibit_winners: lateral inhibition and convolutional k-WTA (Spyker §II-F.3).
//
// Pointwise inhibition is one coalesced sweep over the spike-time and
// potential maps: one thread per location (b, y, x) walks the C maps and
// keeps the earliest neuron (then the higher potential, then the lower map).
// Its survivor is written as an 8-byte record (time|map, potential) to the
// workspace, and optionally the inhibited time map.  Winner selection then
// runs one workgroup per sample: up to k greedy rounds of an arg-min over the
// surviving records.  Up to 8192 candidates per sample stay in registers;
// larger maps keep the suppressed maps and locations as bit sets in LDS and
// sweep the records each round.  Readout layers (no threshold) and calls
// without pointwise inhibition rank the neurons themselves instead of
// per-location records.
#include <algorithm>

#include "spk_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kMaxPos = 1 << 19;      // H*W per sample (64 KB location bit set)
constexpr int kMaxMaps = 1 << 16;     // C (8 KB map bit set)
constexpr int kMaxK = 4096;

struct Rec {
    uint32_t tc;  // time << 24 | map; time == NEVER: no survivor here
    float v;
};

__device__ __forceinline__ uint32_t order_desc(float v)
{
    if (v == 0.0f) v = 0.0f;
    uint32_t u = __float_as_uint(v);
    uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ~asc;
}

// Block = 64 consecutive locations x kGroups waves; wave g walks the maps
// c = g, g + kGroups, ... for its 64 locations (coalesced loads per map), and
// the kGroups partial winners meet in LDS.
constexpr int kGroups = 16;

__device__ __forceinline__ bool earlier(int ta, float va, int ca, int tb, float vb, int cb)
{
    if (ta != tb) return ta < tb;
    if (va != vb) return va > vb;
    return ca < cb;
}

__global__ __launch_bounds__(64 * kGroups) void k_pointwise(const uint8_t *times,
                                                            const float *__restrict__ vkey, int C,
                                                            int HW, long long total,
                                                            Rec *__restrict__ recs,
                                                            uint8_t *inhibited)
{
    __shared__ int s_t[kGroups][64], s_c[kGroups][64];
    __shared__ float s_v[kGroups][64];
    const int lane = threadIdx.x & 63, grp = threadIdx.x >> 6;
    const long long i = (long long)blockIdx.x * 64 + lane;  // b*HW + p
    const bool ok = i < total;
    const long long b = ok ? i / HW : 0, p = i - b * HW;
    const size_t base = (size_t)b * C * HW + p;
    int bt = spk::kNever, bc = -1;
    float bv = 0.0f;
    if (ok) {
        // maps in batches of 4: the loads of a batch are issued before any is used
        auto take = [&](int c, int t, float v) {
            if (t != spk::kNever && (t < bt || (t == bt && v > bv))) {
                bt = t;
                bv = v;
                bc = c;
            }
        };
        int c = grp;
        for (; c + 3 * kGroups < C; c += 4 * kGroups) {
            int t[4];
            float v[4];
#pragma unroll
            for (int u = 0; u < 4; u++) {
                t[u] = times[base + (size_t)(c + u * kGroups) * HW];
                v[u] = vkey[base + (size_t)(c + u * kGroups) * HW];
            }
#pragma unroll
            for (int u = 0; u < 4; u++) take(c + u * kGroups, t[u], v[u]);
        }
        for (; c < C; c += kGroups) take(c, times[base + (size_t)c * HW], vkey[base + (size_t)c * HW]);
    }
    s_t[grp][lane] = bt;
    s_v[grp][lane] = bv;
    s_c[grp][lane] = bc;
    __syncthreads();
    if (grp == 0) {
        for (int q = 1; q < kGroups; q++) {
            const int t = s_t[q][lane], c = s_c[q][lane];
            const float v = s_v[q][lane];
            if (c >= 0 && (bc < 0 || earlier(t, v, c, bt, bv, bc))) {
                bt = t;
                bv = v;
                bc = c;
            }
        }
        s_t[0][lane] = bt;
        s_c[0][lane] = bc;
        if (ok && recs) recs[i] = Rec{((uint32_t)bt << 24) | (uint32_t)(bc < 0 ? 0 : bc), bv};
    }
    if (inhibited) {
        __syncthreads();
        const int wt = s_t[0][lane], wc = s_c[0][lane];
        if (ok)
            for (int c = grp; c < C; c += kGroups)
                inhibited[base + (size_t)c * HW] = (c == wc) ? (uint8_t)wt : (uint8_t)spk::kNever;
    }
}

// The same sweep with L consecutive locations per lane (H*W a multiple of
// L = 4 or 8): each load of a wave brings 64*L time bytes and 256*L bytes of
// potentials.  Block (x, y) takes the maps [y*c_per, (y+1)*c_per); its G
// waves split them (c = g, g + G, ...), with U maps' loads in flight at a
// time, and meet in LDS.  kNT: the loads and the map's stores are
// non-temporal (large layers, whose data is touched once; a small layer's
// maps are still in the caches from the conv and go on to the pooling).  One
// split (gridDim.y == 1, part == nullptr) gives the result of k_pointwise;
// with several, each block writes its winner per location to
// part[y][location] and k_pw_merge finishes.
constexpr int kG4 = 8;   // waves of a block, and
constexpr int kU = 4;    // maps in flight per wave, of the usual form
constexpr int kU8 = 3;   // (three with L = 8: 60 registers, four blocks per CU);
constexpr int kGW = 16;  // those of the wide form (L = 4) for layers with
constexpr int kUW = 8;   // few location blocks

template <int L> struct TimesVec;
template <> struct TimesVec<4> { typedef uint32_t type; };
template <> struct TimesVec<8> { typedef uint2 type; };

template <int L>
__device__ __forceinline__ uint32_t time_at(const typename TimesVec<L>::type &t, int q)
{
    if constexpr (L == 4) return (t >> (8 * q)) & 0xFF;
    else return ((q < 4 ? t.x : t.y) >> (8 * (q & 3))) & 0xFF;
}

template <int L, int G, int U, bool kNT>
__global__ __launch_bounds__(64 * G) void k_pointwise_v(const uint8_t *times,
                                                          const float *__restrict__ vkey, int C,
                                                          int HW, long long total, int c_per,
                                                          Rec *__restrict__ part,
                                                          Rec *__restrict__ recs, uint8_t *inhibited)
{
    typedef typename TimesVec<L>::type TV;
    constexpr int NL = 64 * L;  // locations of a block
    __shared__ uint32_t s_tc[G][NL];  // time << 24 | map (time NEVER: none)
    __shared__ float s_v[G][NL];
    const int lane = threadIdx.x & 63, grp = threadIdx.x >> 6;
    const long long i0 = (long long)blockIdx.x * NL + L * lane;  // b*HW + p, p % L == 0
    const bool ok = i0 < total;
    const long long b = ok ? i0 / HW : 0, p = i0 - b * HW;
    const size_t base = (size_t)b * C * HW + p;
    // per location: time << 24 | map of the best so far (time NEVER: none),
    // one register instead of two, and its potential
    uint32_t btc[L];
    float bv[L];
#pragma unroll
    for (int q = 0; q < L; q++) {
        btc[q] = ~0u;
        bv[q] = 0.0f;
    }
    if (ok) {
        auto take = [&](int c, const TV &t4, const float4 *v4) {
#pragma unroll
            for (int q = 0; q < L; q++) {
                const int t = (int)time_at<L>(t4, q);
                const float4 &vq = v4[q >> 2];
                const float v = (q & 3) == 0 ? vq.x : (q & 3) == 1 ? vq.y : (q & 3) == 2 ? vq.z : vq.w;
                const int bt = (int)(btc[q] >> 24);
                if (t != spk::kNever && (t < bt || (t == bt && v > bv[q]))) {
                    btc[q] = ((uint32_t)t << 24) | (uint32_t)c;
                    bv[q] = v;
                }
            }
        };
        const int c_lo = (int)blockIdx.y * c_per, c_hi = min(C, c_lo + c_per);
        // a batch past c_hi loads map c_hi - 1 again (no branch around a load)
        // and skips it
        for (int c = c_lo + grp; c < c_hi; c += U * G) {
            TV t[U];
            float4 v[U][L / 4];
#pragma unroll
            for (int u = 0; u < U; u++) {
                const size_t at = base + (size_t)min(c + u * G, c_hi - 1) * HW;
                // kNT: read once, streaming (non-temporal) loads
                typedef float nf4 __attribute__((ext_vector_type(4)));
                typedef uint32_t nu2 __attribute__((ext_vector_type(2)));
                if constexpr (!kNT)
                    t[u] = *reinterpret_cast<const TV *>(times + at);
                else if constexpr (L == 4)
                    t[u] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t *>(times + at));
                else
                    t[u] = __builtin_bit_cast(TV, __builtin_nontemporal_load(reinterpret_cast<const nu2 *>(times + at)));
#pragma unroll
                for (int r = 0; r < L / 4; r++)
                    v[u][r] = kNT ? __builtin_bit_cast(float4, __builtin_nontemporal_load(
                                                                   reinterpret_cast<const nf4 *>(vkey + at + 4 * r)))
                                  : *reinterpret_cast<const float4 *>(vkey + at + 4 * r);
            }
#pragma unroll
            for (int u = 0; u < U; u++)
                if (c + u * G < c_hi) take(c + u * G, t[u], v[u]);
        }
    }
#pragma unroll
    for (int q = 0; q < L; q++) {
        s_tc[grp][L * lane + q] = btc[q];
        s_v[grp][L * lane + q] = bv[q];
    }
    __syncthreads();
    // the block's locations, one thread each, merge the G partial winners as
    // a minimum of 64-bit keys ordered as `earlier` (no branches)
    for (int j = threadIdx.x; j < NL; j += blockDim.x) {
        uint64_t best = ~0ull;
        float v0 = 0.0f;
        for (int g = 0; g < G; g++) {
            const uint32_t tc = s_tc[g][j];
            const float v = s_v[g][j];
            const uint64_t key = (tc >> 24) == (uint32_t)spk::kNever
                                     ? ~0ull
                                     : ((uint64_t)(tc >> 24) << 56) | ((uint64_t)order_desc(v) << 24) |
                                           (uint64_t)(tc & 0xFFFFFFu);
            const bool better = key < best;
            best = better ? key : best;
            v0 = better ? v : v0;
        }
        const bool any = best != ~0ull;
        const uint32_t tc0 = any ? (uint32_t)(best >> 56) << 24 | (uint32_t)(best & 0xFFFFFFu)
                                 : (uint32_t)spk::kNever << 24;
        s_tc[0][j] = tc0;
        const long long i = (long long)blockIdx.x * NL + j;
        const Rec r{tc0, any ? v0 : 0.0f};
        if (part) {
            if (i < total) part[(size_t)blockIdx.y * total + i] = r;
        } else if (recs && i < total) {
            recs[i] = r;
        }
    }
    if (inhibited && !part) {
        __syncthreads();
        if (ok) {
            int wt[L], wc[L];
#pragma unroll
            for (int q = 0; q < L; q++) {
                const uint32_t tc = s_tc[0][L * lane + q];
                wt[q] = (int)(tc >> 24);
                wc[q] = wt[q] == (int)spk::kNever ? -1 : (int)(tc & 0xFFFFFFu);
            }
            for (int c = grp; c < C; c += G) {
                uint32_t o[2] = {0u, 0u};
#pragma unroll
                for (int q = 0; q < L; q++)
                    o[q >> 2] |= (uint32_t)(c == wc[q] ? wt[q] : spk::kNever) << (8 * (q & 3));
                typedef uint32_t nu2 __attribute__((ext_vector_type(2)));
                uint8_t *dst = inhibited + base + (size_t)c * HW;
                if constexpr (!kNT && L == 4)
                    *reinterpret_cast<uint32_t *>(dst) = o[0];
                else if constexpr (!kNT)
                    *reinterpret_cast<uint2 *>(dst) = make_uint2(o[0], o[1]);
                else if constexpr (L == 4)
                    __builtin_nontemporal_store(o[0], reinterpret_cast<uint32_t *>(dst));
                else
                    __builtin_nontemporal_store(nu2{o[0], o[1]}, reinterpret_cast<nu2 *>(dst));
            }
        }
    }
}

// Winners of the map splits, merged per location as a minimum of keys that
// order records as `earlier` does (a total order on distinct maps, so the
// order of the splits does not matter), four locations per thread (H*W a
// multiple of 4).  Block (x, y) writes the inhibited time bytes of maps
// [y*c_chunk, (y+1)*c_chunk); blocks with y == 0 also write the records.
__global__ __launch_bounds__(kThreads) void k_pw_merge(const Rec *__restrict__ part, int S,
                                                       long long total, int C, int HW, int c_chunk,
                                                       Rec *__restrict__ recs, uint8_t *inhibited)
{
    const long long i0 = ((long long)blockIdx.x * kThreads + threadIdx.x) * 4;
    if (i0 >= total) return;
    // A record as one 64-bit key, smaller = earlier: time, then the potential
    // in descending order, then the map; a split without a survivor gives
    // the largest key.  The merge is a minimum, with no branches.
    uint64_t best[4];
    float bv[4];
#pragma unroll
    for (int q = 0; q < 4; q++) {
        best[q] = ~0ull;
        bv[q] = 0.0f;
    }
    // eight splits' loads in flight at a time; a batch past S repeats split
    // S - 1, which leaves a minimum unchanged
    for (int y0 = 0; y0 < S; y0 += 8) {
        uint4 w[8][2];
#pragma unroll
        for (int u = 0; u < 8; u++) {
            const uint4 *pp = reinterpret_cast<const uint4 *>(part + (size_t)min(y0 + u, S - 1) * total + i0);
            w[u][0] = pp[0];
            w[u][1] = pp[1];
        }
#pragma unroll
        for (int u = 0; u < 8; u++) {
            const uint4 a = w[u][0], b = w[u][1];
            const uint32_t tc[4] = {a.x, a.z, b.x, b.z}, vb[4] = {a.y, a.w, b.y, b.w};
#pragma unroll
            for (int q = 0; q < 4; q++) {
                const uint32_t t = tc[q] >> 24;
                const uint64_t key = t == (uint32_t)spk::kNever
                                         ? ~0ull
                                         : ((uint64_t)t << 56) |
                                               ((uint64_t)order_desc(__uint_as_float(vb[q])) << 24) |
                                               (uint64_t)(tc[q] & 0xFFFFFFu);
                const bool better = key < best[q];
                best[q] = better ? key : best[q];
                bv[q] = better ? __uint_as_float(vb[q]) : bv[q];
            }
        }
    }
    int t0[4], c0[4];
    float v0[4];
#pragma unroll
    for (int q = 0; q < 4; q++) {
        const bool any = best[q] != ~0ull;
        t0[q] = any ? (int)(best[q] >> 56) : (int)spk::kNever;
        c0[q] = any ? (int)(best[q] & 0xFFFFFFu) : -1;
        v0[q] = any ? bv[q] : 0.0f;
    }
    if (blockIdx.y == 0 && recs) {
#pragma unroll
        for (int q = 0; q < 4; q++)
            recs[i0 + q] = Rec{((uint32_t)t0[q] << 24) | (uint32_t)(c0[q] < 0 ? 0 : c0[q]), v0[q]};
    }
    if (inhibited) {
        const long long b = i0 / HW, p = i0 - b * HW;
        const int c_lo = (int)blockIdx.y * c_chunk, c_hi = min(C, c_lo + c_chunk);
        for (int c = c_lo; c < c_hi; c++) {
            uint32_t o = 0u;
#pragma unroll
            for (int q = 0; q < 4; q++) o |= (uint32_t)(c == c0[q] ? t0[q] : (int)spk::kNever) << (8 * q);
            *reinterpret_cast<uint32_t *>(inhibited + ((size_t)b * C + c) * HW + p) = o;
        }
    }
}

// How a location sweep is laid out: L locations per lane (0: the scalar
// kernel), G waves per block with U maps in flight per wave, X location
// blocks and S map splits of c_per maps each.  A wave issues the loads of U
// maps together, so a block whose waves have several such batches waits
// several memory latencies.  Layers with few location blocks take the wide
// form (16 waves, 8 maps in flight); when even that leaves more than two
// batches per wave, the maps are split so that each wave has one.
struct PwPlan {
    int L, G, U;
    long long X;
    int S, c_per;
};

PwPlan pw_plan(long long total, int C, int HW, bool aligned, bool may_split)
{
    PwPlan pl{0, kGroups, 1, spk::ceil_div(total, 64), 1, C};
    if (!aligned || HW % 4 != 0) return pl;
    pl.L = HW % 8 == 0 ? 8 : 4;
    pl.G = kG4;
    pl.U = pl.L == 8 ? kU8 : kU;
    pl.X = spk::ceil_div(total, 64 * pl.L);
    if (spk::ceil_div(total, 64 * 4) < 256) {
        pl.L = 4;
        pl.G = kGW;
        pl.U = kUW;
        pl.X = spk::ceil_div(total, 64 * 4);
    }
    if (may_split && pl.X < 1024 && C > 2 * pl.G * pl.U) {
        pl.c_per = pl.G * pl.U;
        pl.S = spk::ceil_div(C, pl.c_per);
    }
    return pl;
}

size_t pw_part_bytes(long long total, int C, int HW)
{
    const PwPlan pl = pw_plan(total, C, HW, true, true);
    return pl.S > 1 ? spk::align_up((size_t)pl.S * total * sizeof(Rec), 256) : 0;
}

// Launch of the location sweep: vectorized when H*W and the arrays allow,
// split over the maps when a workspace for the partial winners is given.
void launch_pointwise(const uint8_t *times, const float *vkey, int C, int HW, long long total, Rec *recs,
                      uint8_t *inhibited, Rec *part, hipStream_t s)
{
    const bool al = (uintptr_t)times % 8 == 0 && (uintptr_t)vkey % 16 == 0 && (uintptr_t)inhibited % 8 == 0;
    const PwPlan pl = pw_plan(total, C, HW, al, part != nullptr);
    Rec *pp = pl.S > 1 ? part : nullptr;
    const dim3 grid((unsigned)pl.X, pl.S);
    if (pl.L == 8)
        hipLaunchKernelGGL((k_pointwise_v<8, kG4, kU8, true>), grid, dim3(64 * kG4), 0, s, times, vkey, C, HW, total,
                           pl.c_per, pp, recs, inhibited);
    else if (pl.L == 4 && pl.G == kGW)
        hipLaunchKernelGGL((k_pointwise_v<4, kGW, kUW, false>), grid, dim3(64 * kGW), 0, s, times, vkey, C, HW, total,
                           pl.c_per, pp, recs, inhibited);
    else if (pl.L == 4)
        hipLaunchKernelGGL((k_pointwise_v<4, kG4, kU, true>), grid, dim3(64 * kG4), 0, s, times, vkey, C, HW, total,
                           pl.c_per, pp, recs, inhibited);
    else
        hipLaunchKernelGGL(k_pointwise, dim3((unsigned)pl.X), dim3(64 * kGroups), 0, s, times, vkey, C, HW,
                           total, recs, inhibited);
    if (pp) {
        const long long xm = spk::ceil_div(total, 4 * kThreads);
        const int chunks = (int)std::min<long long>(C, spk::ceil_div(1024, xm));
        const int c_chunk = (int)spk::ceil_div(C, chunks);
        hipLaunchKernelGGL(k_pw_merge, dim3((unsigned)xm, (unsigned)spk::ceil_div(C, c_chunk)), dim3(kThreads),
                           0, s, pp, pl.S, total, C, HW, c_chunk, recs, inhibited);
    }
}

// Wave-wide minima with row shifts and row broadcasts (DPP) instead of LDS
// permutes.  Lanes without a source keep the identity (all ones); every lane
// gets the result.
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_or_ones(uint32_t x)
{
    return (uint32_t)__builtin_amdgcn_update_dpp((int)0xFFFFFFFF, (int)x, CTRL, ROWS, 0xf, false);
}

template <int CTRL, int ROWS>
__device__ __forceinline__ uint64_t dpp_or_ones64(uint64_t x)
{
    const uint32_t lo = dpp_or_ones<CTRL, ROWS>((uint32_t)x);
    const uint32_t hi = dpp_or_ones<CTRL, ROWS>((uint32_t)(x >> 32));
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x)
{
    x = min(x, dpp_or_ones64<0x111, 0xf>(x));  // row_shr:1
    x = min(x, dpp_or_ones64<0x112, 0xf>(x));  // row_shr:2
    x = min(x, dpp_or_ones64<0x114, 0xf>(x));  // row_shr:4
    x = min(x, dpp_or_ones64<0x118, 0xf>(x));  // row_shr:8
    x = min(x, dpp_or_ones64<0x142, 0xa>(x));  // row_bcast:15
    x = min(x, dpp_or_ones64<0x143, 0xc>(x));  // row_bcast:31
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), 63);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x)
{
    x = min(x, dpp_or_ones<0x111, 0xf>(x));
    x = min(x, dpp_or_ones<0x112, 0xf>(x));
    x = min(x, dpp_or_ones<0x114, 0xf>(x));
    x = min(x, dpp_or_ones<0x118, 0xf>(x));
    x = min(x, dpp_or_ones<0x142, 0xa>(x));
    x = min(x, dpp_or_ones<0x143, 0xc>(x));
    return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

// Lexicographic (hi, lo) minimum across the block; returns the winner to all.
__device__ void block_argmin(uint64_t &hi, uint32_t &lo, uint64_t *s_hi, uint32_t *s_lo)
{
    for (int o = 32; o > 0; o >>= 1) {
        uint64_t h2 = __shfl_xor(hi, o, 64);
        uint32_t l2 = __shfl_xor(lo, o, 64);
        if (h2 < hi || (h2 == hi && l2 < lo)) {
            hi = h2;
            lo = l2;
        }
    }
    const int wid = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        s_hi[wid] = hi;
        s_lo[wid] = lo;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < (int)(blockDim.x >> 6); w++)
            if (s_hi[w] < s_hi[0] || (s_hi[w] == s_hi[0] && s_lo[w] < s_lo[0])) {
                s_hi[0] = s_hi[w];
                s_lo[0] = s_lo[w];
            }
    }
    __syncthreads();
    hi = s_hi[0];
    lo = s_lo[0];
    __syncthreads();
}

struct WtaArgs {
    int C, H, W, T, k, radius, readout, by_record;
};

// 1024 threads: one block per sample is all the grid has, so each sweep of
// the candidates is spread over as many lanes as a block holds.
constexpr int kSelT = 1024;

__global__ __launch_bounds__(kSelT) void k_select(const uint8_t *__restrict__ times,
                                                     const float *__restrict__ vkey,
                                                     const Rec *__restrict__ recs, WtaArgs a,
                                                     int stage_recs, spk_winner *__restrict__ winners,
                                                     int32_t *__restrict__ n_winners)
{
    extern __shared__ uint32_t bits[];  // [positions][maps] dead bits, then staged records
    __shared__ uint64_t s_hi[kSelT / 64];
    __shared__ uint32_t s_lo[kSelT / 64];
    const int b = blockIdx.x;
    const int HW = a.H * a.W;
    const int pw = (HW + 31) / 32, cw = (a.C + 31) / 32;
    uint32_t *pos_dead = bits, *map_dead = bits + pw;
    Rec *srec = reinterpret_cast<Rec *>(bits + ((pw + cw + 1) & ~1));
    for (int i = threadIdx.x; i < pw + cw; i += blockDim.x) bits[i] = 0;
    const Rec *rb = recs + (size_t)b * HW;
    if (a.by_record && stage_recs) {
        for (int p = threadIdx.x; p < HW; p += blockDim.x) srec[p] = rb[p];
        rb = srec;
    }
    __syncthreads();
    const uint64_t kNone = ~0ull;
    int count = 0;
    for (int round = 0; round < a.k; round++) {
        uint64_t hi = kNone;
        uint32_t lo = ~0u;
        // candidates in batches of kScan per thread: a batch's loads are all
        // issued before any is tested
        constexpr int kScan = 8;
        if (a.by_record) {
            for (int p0 = threadIdx.x; p0 < HW; p0 += kScan * (int)blockDim.x) {
                Rec rr[kScan];
#pragma unroll
                for (int u = 0; u < kScan; u++) rr[u] = rb[min(p0 + u * (int)blockDim.x, HW - 1)];
#pragma unroll
                for (int u = 0; u < kScan; u++) {
                    const int p = p0 + u * (int)blockDim.x;
                    if (p >= HW || (pos_dead[p >> 5] & (1u << (p & 31)))) continue;
                    const uint32_t t = rr[u].tc >> 24, c = rr[u].tc & 0xFFFFFFu;
                    if (t == (uint32_t)spk::kNever || (map_dead[c >> 5] & (1u << (c & 31)))) continue;
                    const uint64_t h = ((uint64_t)t << 32) | order_desc(rr[u].v);
                    const uint32_t l = c * (uint32_t)HW + (uint32_t)p;
                    if (h < hi || (h == hi && l < lo)) {
                        hi = h;
                        lo = l;
                    }
                }
            }
        } else {
            const size_t base = (size_t)b * a.C * HW;
            const int n = a.C * HW;
            for (int i0 = threadIdx.x; i0 < n; i0 += kScan * (int)blockDim.x) {
                uint32_t tt[kScan];
                float vv[kScan];
#pragma unroll
                for (int u = 0; u < kScan; u++) {
                    const int i = min(i0 + u * (int)blockDim.x, n - 1);
                    tt[u] = times[base + i];
                    vv[u] = vkey[base + i];
                }
#pragma unroll
                for (int u = 0; u < kScan; u++) {
                    const int i = i0 + u * (int)blockDim.x;
                    if (i >= n) continue;
                    const int c = i / HW, p = i - c * HW;
                    if (pos_dead[p >> 5] & (1u << (p & 31))) continue;
                    if (map_dead[c >> 5] & (1u << (c & 31))) continue;
                    const uint32_t t = tt[u];
                    if (!a.readout && t == (uint32_t)spk::kNever) continue;
                    const uint64_t h = ((uint64_t)(a.readout ? 0u : t) << 32) | order_desc(vv[u]);
                    if (h < hi || (h == hi && (uint32_t)i < lo)) {
                        hi = h;
                        lo = (uint32_t)i;
                    }
                }
            }
        }
        block_argmin(hi, lo, s_hi, s_lo);
        if (hi == kNone) break;
        const int c = (int)(lo / (uint32_t)HW), p = (int)(lo % (uint32_t)HW);
        const int y = p / a.W, x = p - y * a.W;
        if (threadIdx.x == 0) {
            spk_winner wn;
            wn.c = c;
            wn.y = y;
            wn.x = x;
            wn.t = a.readout ? a.T - 1 : (int)(hi >> 32);
            wn.v = vkey[(size_t)b * a.C * HW + (size_t)c * HW + p];
            winners[(size_t)b * a.k + count] = wn;
            map_dead[c >> 5] |= 1u << (c & 31);
        }
        const int r = a.radius, side = 2 * r + 1;
        for (int i = threadIdx.x; i < side * side; i += blockDim.x) {
            const int yy = y - r + i / side, xx = x - r + i % side;
            if (yy >= 0 && yy < a.H && xx >= 0 && xx < a.W) {
                const int q = yy * a.W + xx;
                atomicOr(&pos_dead[q >> 5], 1u << (q & 31));
            }
        }
        count++;
        __syncthreads();
    }
    for (int s = count + threadIdx.x; s < a.k; s += blockDim.x)
        winners[(size_t)b * a.k + s] = spk_winner{-1, -1, -1, -1, 0.0f};
    if (threadIdx.x == 0) n_winners[b] = count;
}

// Winner selection with the candidates of one sample held in registers: NW
// waves, NPL candidates per thread (candidate i at thread i % (64*NW), slot
// i / (64*NW)).  A round is a register arg-min, a wave reduction (DPP) and,
// with several waves, one exchange through LDS; the lane that owns the
// winner writes it, and every lane retires its own candidates that share the
// winner's map or lie in its window.
// The k rounds of a sample's winner selection on candidates held in
// registers (NPL per thread, NW waves): candidate keys kh = time << 32 |
// order_desc(v) (kNone: not a candidate), ties to the lower kl = map*HW +
// position; cc, yx, vv: its map, y << 16 | x and potential.
template <int NPL, int NW, bool kPacked>
__device__ __forceinline__ void select_rounds(uint64_t (&kh)[NPL], const uint32_t (&kl)[NPL],
                                              const int (&cc)[NPL], const int (&yx)[NPL],
                                              const float (&vv)[NPL], const WtaArgs &a, int HW, int b,
                                              uint64_t (&s_hi)[2][NW], uint32_t (&s_lo)[2][NW],
                                              spk_winner *__restrict__ winners,
                                              int32_t *__restrict__ n_winners)
{
    const uint64_t kNone = ~0ull;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int count = 0;
    for (int round = 0; round < a.k; round++) {
        uint64_t bh = kNone;
        uint32_t bl = ~0u;
        if constexpr (kPacked) {
            // keys t << 56 | order << 24 | index: one 64-bit minimum
#pragma unroll
            for (int j = 0; j < NPL; j++) bh = kh[j] < bh ? kh[j] : bh;
            bh = wave_min_u64(bh);
        } else {
#pragma unroll
            for (int j = 0; j < NPL; j++)
                if (kh[j] < bh || (kh[j] == bh && kl[j] < bl)) {
                    bh = kh[j];
                    bl = kl[j];
                }
            // the smallest key, then the smallest index among the lanes holding it
            const uint64_t wh = wave_min_u64(bh);
            bl = wave_min_u32(bh == wh ? bl : ~0u);
            bh = wh;
        }
        if (NW > 1) {
            const int slot = round & 1;
            if (lane == 0) {
                s_hi[slot][wave] = bh;
                s_lo[slot][wave] = bl;
            }
            __syncthreads();
#pragma unroll
            for (int w = 0; w < NW; w++) {
                const uint64_t h2 = s_hi[slot][w];
                const uint32_t l2 = s_lo[slot][w];
                if (h2 < bh || (!kPacked && h2 == bh && l2 < bl)) {
                    bh = h2;
                    bl = l2;
                }
            }
        }
        if (bh == kNone) break;
        uint32_t order = (uint32_t)bh;  // order_desc of the winner's potential
        int tw = (int)(bh >> 32);       // its time
        if constexpr (kPacked) {
            bl = (uint32_t)bh & 0xFFFFFFu;
            order = (uint32_t)(bh >> 24);
            tw = (int)(bh >> 56);
        }
        const int wc = (int)(bl / (uint32_t)HW), wp = (int)(bl - (uint32_t)wc * (uint32_t)HW);
        const int wy = wp / a.W, wx = wp - wy * a.W;
        if (tid == 0) {
            // the winner's potential from its key (the map of order_desc back to the float bits)
            const uint32_t asc = ~order;
            const uint32_t u = (asc & 0x80000000u) ? (asc & 0x7FFFFFFFu) : ~asc;
            spk_winner wn;
            wn.c = wc;
            wn.y = wy;
            wn.x = wx;
            wn.t = a.readout ? a.T - 1 : tw;
            wn.v = __uint_as_float(u);
            winners[(size_t)b * a.k + count] = wn;
        }
        // a candidate is suppressed by the winner's map, or by lying within
        // the radius: with both coordinates packed as 16-bit halves,
        // (y - wy + r) and (x - wx + r), taken modulo 2^16, are both at most 2r
        const uint32_t base = ((uint32_t)(wy - a.radius) << 16) | (uint32_t)((wx - a.radius) & 0xFFFF);
        const uint32_t lim = 0x00010001u * (uint32_t)(2 * a.radius);
#pragma unroll
        for (int j = 0; j < NPL; j++) {
            typedef unsigned short us2 __attribute__((ext_vector_type(2)));
            const us2 e = __builtin_bit_cast(us2, (uint32_t)yx[j]) - __builtin_bit_cast(us2, base);
            const us2 over = __builtin_elementwise_sub_sat(e, __builtin_bit_cast(us2, lim));
            const bool near = __builtin_bit_cast(uint32_t, over) == 0u;
            if (cc[j] == wc || near) kh[j] = kNone;
        }
        count++;
    }
    for (int s = count + tid; s < a.k; s += 64 * NW)
        winners[(size_t)b * a.k + s] = spk_winner{-1, -1, -1, -1, 0.0f};
    if (tid == 0) n_winners[b] = count;
}

// kPacked: candidate indices below 2^24, so (time, potential order, index) fit
// one 64-bit key.
template <int NPL, int NW, bool kRec, bool kPacked>
__global__ __launch_bounds__(64 * NW) void k_select_reg(const uint8_t *__restrict__ times,
                                                        const float *__restrict__ vkey,
                                                        const Rec *__restrict__ recs, WtaArgs a,
                                                        spk_winner *__restrict__ winners,
                                                        int32_t *__restrict__ n_winners)
{
    __shared__ uint64_t s_hi[2][NW];
    __shared__ uint32_t s_lo[2][NW];
    const int b = blockIdx.x;
    const int HW = a.H * a.W;
    const int n = kRec ? HW : a.C * HW;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint64_t kNone = ~0ull;
    uint64_t kh[NPL];
    uint32_t kl[NPL];
    int cc[NPL], yx[NPL];
    float vv[NPL];
    // every candidate load first (clamped index, no branch), then the keys
    uint32_t tq[NPL];
#pragma unroll
    for (int j = 0; j < NPL; j++) {
        const int ii = min(tid + j * 64 * NW, n - 1);
        if (kRec) {
            const Rec r = recs[(size_t)b * HW + ii];
            tq[j] = r.tc;
            vv[j] = r.v;
        } else {
            const size_t at = (size_t)b * a.C * HW + ii;
            tq[j] = times[at];
            vv[j] = vkey[at];
        }
    }
#pragma unroll
    for (int j = 0; j < NPL; j++) {
        const int i = tid + j * 64 * NW;
        const int ii = min(i, n - 1);
        int t, c, pos;
        if (kRec) {
            t = (int)(tq[j] >> 24);
            c = (int)(tq[j] & 0xFFFFFFu);
            pos = ii;
        } else {
            t = (int)tq[j];
            c = ii / HW;
            pos = ii - c * HW;
        }
        const bool alive = i < n && (a.readout || t != spk::kNever);
        const uint32_t tk = a.readout ? 0u : (uint32_t)t;
        kh[j] = !alive ? kNone
                : kPacked ? (((uint64_t)tk << 56) | ((uint64_t)order_desc(vv[j]) << 24) |
                             (uint64_t)((uint32_t)c * (uint32_t)HW + (uint32_t)pos))
                          : (((uint64_t)tk << 32) | order_desc(vv[j]));
        kl[j] = (uint32_t)c * (uint32_t)HW + (uint32_t)pos;
        cc[j] = c;
        const int y = pos / a.W;
        yx[j] = (y << 16) | (pos - y * a.W);
    }
    select_rounds<NPL, NW, kPacked>(kh, kl, cc, yx, vv, a, HW, b, s_hi, s_lo, winners, n_winners);
}

template <int NPL, int NW>
void launch_select_reg(int B, hipStream_t s, const uint8_t *times, const float *vkey,
                       const Rec *recs, const WtaArgs &a, spk_winner *winners, int32_t *n_winners)
{
    const bool packed = (long long)a.C * a.H * a.W <= (1ll << 24);
    auto run = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3(B), dim3(64 * NW), 0, s, times, vkey, recs, a, winners, n_winners);
    };
    if (a.by_record) {
        if (packed) run(k_select_reg<NPL, NW, true, true>);
        else run(k_select_reg<NPL, NW, true, false>);
    } else {
        if (packed) run(k_select_reg<NPL, NW, false, true>);
        else run(k_select_reg<NPL, NW, false, false>);
    }
}

}  // namespace

extern "C" size_t spk_inhibit_winners_workspace_size(int B, int C, int H, int W)
{
    if (B <= 0 || C <= 0 || H <= 0 || W <= 0) return 0;
    const long long total = (long long)B * H * W;
    return spk::align_up((size_t)total * sizeof(Rec), 256) + pw_part_bytes(total, C, H * W);
}

extern "C" spk_status spk_inhibit_winners(const uint8_t *times, const float *vkey, int B, int C,
                                          int H, int W, int T, int pointwise, int k, int radius,
                                          int readout, uint8_t *inhibited, spk_winner *winners,
                                          int32_t *n_winners, void *ws, size_t ws_bytes,
                                          spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(times && vkey && n_winners && (winners || k == 0), SPK_E_ARG,
                "spk_inhibit_winners: NULL pointer");
    SPK_REQUIRE(B > 0 && C > 0 && H > 0 && W > 0 && k >= 0 && radius >= 0, SPK_E_ARG,
                "spk_inhibit_winners: B=%d C=%d H=%d W=%d k=%d radius=%d", B, C, H, W, k, radius);
    SPK_REQUIRE(T >= 1 && T <= SPK_MAX_T, SPK_E_SHAPE, "spk_inhibit_winners: T=%d not in [1, %d]",
                T, SPK_MAX_T);
    SPK_REQUIRE((long long)H * W <= kMaxPos && C <= kMaxMaps && k <= kMaxK &&
                    (long long)C * H * W < (1LL << 31),
                SPK_E_SHAPE, "spk_inhibit_winners: H*W <= %d, C <= %d, k <= %d required", kMaxPos,
                kMaxMaps, kMaxK);
    SPK_REQUIRE(!(readout && pointwise), SPK_E_UNSUPPORTED,
                "spk_inhibit_winners: readout ranks all neurons; pointwise must be 0");
    SPK_REQUIRE(B <= 65535 || !pointwise, SPK_E_SHAPE, "spk_inhibit_winners: B > 65535");
    const size_t need = pointwise ? spk_inhibit_winners_workspace_size(B, C, H, W) : 0;
    SPK_REQUIRE(ws_bytes >= need && (need == 0 || ws), SPK_E_WORKSPACE,
                "spk_inhibit_winners: workspace of %zu bytes needed, %zu given", need, ws_bytes);
    SPK_REQUIRE_WS_ALIGNED(ws, "spk_inhibit_winners");
    hipStream_t s = spk::stream_of(stream);
    const int HW = H * W;
    Rec *recs = (Rec *)ws;
    WtaArgs a{C, H, W, T, k, radius, readout, pointwise};
    if (pointwise) {
        const long long total = (long long)B * HW;
        Rec *part = reinterpret_cast<Rec *>(reinterpret_cast<char *>(ws) +
                                            spk::align_up((size_t)total * sizeof(Rec), 256));
        launch_pointwise(times, vkey, C, HW, total, recs, inhibited, part, s);
        SPK_LAUNCHED("spk_inhibit_winners");
    } else if (inhibited && inhibited != times) {
        SPK_REQUIRE(hipMemcpyAsync(inhibited, times, (size_t)B * C * HW, hipMemcpyDeviceToDevice,
                                   s) == hipSuccess,
                    SPK_E_HIP, "spk_inhibit_winners: copy of the time map failed");
    }
    // candidates per sample: one record per location after pointwise
    // inhibition, else every neuron
    const long long n_cand = pointwise ? (long long)HW : (long long)C * HW;
    if (k > 0 && n_cand <= 64 * 4) {
        launch_select_reg<4, 1>(B, s, times, vkey, recs, a, winners, n_winners);
    } else if (k > 0 && n_cand <= 256 * 4) {
        launch_select_reg<4, 4>(B, s, times, vkey, recs, a, winners, n_winners);
    } else if (k > 0 && n_cand <= 256 * 16) {
        launch_select_reg<16, 4>(B, s, times, vkey, recs, a, winners, n_winners);
    } else if (k > 0 && n_cand <= 256 * 20) {
        launch_select_reg<20, 4>(B, s, times, vkey, recs, a, winners, n_winners);
    } else if (k > 0 && n_cand <= 512 * 16) {
        launch_select_reg<16, 8>(B, s, times, vkey, recs, a, winners, n_winners);
    }
    if (k > 0 && n_cand <= 512 * 16) {
        SPK_LAUNCHED("spk_inhibit_winners");
        return SPK_OK;
    }
    size_t lds = (((size_t)(HW + 31) / 32 + (C + 31) / 32 + 1) & ~(size_t)1) * sizeof(uint32_t);
    // records re-read every round are staged in LDS when there are several rounds
    const int stage = pointwise && k > 1 && lds + (size_t)HW * sizeof(Rec) <= 96 * 1024;
    if (stage) lds += (size_t)HW * sizeof(Rec);
    if (lds > 64 * 1024)
        (void)hipFuncSetAttribute(reinterpret_cast<const void *>(k_select),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(k_select, dim3(B), dim3(k > 0 ? kSelT : 64), lds, s, times, vkey, recs, a,
                       stage, winners, n_winners);
    SPK_LAUNCHED("spk_inhibit_winners");
    return SPK_OK;
}

extern "C" spk_status spk_inhibit(const uint8_t *times, const float *vkey, int B, int C, int H, int W,
                                  uint8_t *inhibited, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(times && vkey && inhibited, SPK_E_ARG, "spk_inhibit: NULL pointer");
    SPK_REQUIRE(B > 0 && C > 0 && H > 0 && W > 0, SPK_E_ARG, "spk_inhibit: sizes must be positive");
    SPK_REQUIRE((long long)C * H * W < (1LL << 31) && (long long)B * H * W < (1LL << 40), SPK_E_SHAPE,
                "spk_inhibit: C*H*W >= 2^31");
    const int HW = H * W;
    const long long total = (long long)B * HW;
    hipStream_t s = spk::stream_of(stream);
    launch_pointwise(times, vkey, C, HW, total, nullptr, inhibited, nullptr, s);
    SPK_LAUNCHED("spk_inhibit");
    return SPK_OK;
}
