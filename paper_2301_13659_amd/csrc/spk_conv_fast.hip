// spk_conv_fire, firing layers on the matrix cores with register-resident
// operands (Spyker §II-E.1 Eq. 2, first-spike firing of §II-D.3).
//
// Two small passes first rewrite the operands into the order the MFMA
// fragments consume (both in the caller's workspace):
//
//  - the time map becomes padded channels-last: Xp[b][iy][ix][c] over the
//    zero-padded extent (Hi + 2 pad) x (Wi + 2 pad), padding = 255 (never
//    fires).  For a fixed kernel row ky, the taps (kx, c) of an output
//    position are then one contiguous run of Kw*Ci bytes;
//  - the depth K is ordered (ky, j) with j = kx*Ci + c, each run padded to a
//    multiple of 8 (R8), so the 8 taps of a fragment lane are 8 consecutive
//    bytes of Xp.  The weights are packed in that order as ready B fragments
//    (hi/lo halves of the float master, or the half weights), zero on the
//    padding taps, so padding bytes never matter.
//
// The firing kernel: a block of 4 waves owns one column tile (16 maps); each
// wave keeps the B fragments of all its K subtiles in registers for the whole
// block.  The block walks row groups (4 waves x R row tiles of 16 positions):
// it stages the contiguous Xp byte range of the group in LDS, every wave pulls
// the 8 time bytes of each of its A fragments into registers, then runs the
// T steps on registers only.  A step either recomputes the potential from the
// cumulative frame, V_t = W * [time <= t] (two packed-half operations per pair
// of taps), or, when the wave's inputs arrive sparsely, adds the newly
// arriving spikes, V_t = V_{t-1} + W * [time == t], skipping subtiles with no
// arrival.  After each step the crossings of theta are recorded in registers;
// times and potentials are written once at the end.
#include <hip/hip_fp16.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <tuple>

#include "spk_internal.h"

namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kSlack = 64;                  // readable bytes past the end of Xp / the halo
constexpr int kHaloMax = 48 * 1024;         // LDS bytes for a staged row group
constexpr uint32_t kSelLo = 0x04010400u;    // bytes 0,1 -> halves 1024 + b
constexpr uint32_t kSelHi = 0x04030402u;    // bytes 2,3 -> halves 1024 + b

struct FGeom {
    int B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo;
    int Cin;     // channels of the input and weights (Ci: channels of Xp, Cin or more)
    int ind;     // 1: Xp holds the readout's indicator bytes (see make_ro_geom), 0: times
    int Hp, Wp;  // padded input extent
    int run;     // Kw*Ci: bytes of one kernel row's taps
    int R8;      // run rounded up to a multiple of 8
    int K;       // Kh*R8: packed depth
    int S;       // ceil(K / 32): MFMA subtiles
    int P;       // B*Ho*Wo: output positions
    int NT;      // ceil(Co / 16): column tiles
    int rowb;    // Wp*Ci: bytes of one padded input row
    int S16;     // ceil(K / 16): subtiles of the 32x32x16 kernel
    int NT32;    // ceil(Co / 32): its column tiles
};

FGeom make_geom(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride, int pad,
                int Ho, int Wo)
{
    FGeom g{};
    g.B = B; g.T = T; g.Ci = Ci; g.Hi = Hi; g.Wi = Wi; g.Co = Co; g.Kh = Kh; g.Kw = Kw;
    g.stride = stride; g.pad = pad; g.Ho = Ho; g.Wo = Wo;
    g.Cin = Ci;
    g.ind = 0;
    g.Hp = Hi + 2 * pad;
    g.Wp = Wi + 2 * pad;
    g.run = Kw * Ci;
    g.R8 = (g.run + 7) / 8 * 8;
    g.K = Kh * g.R8;
    g.S = (g.K + 31) / 32;
    g.P = B * Ho * Wo;
    g.NT = (Co + 15) / 16;
    g.rowb = g.Wp * Ci;
    g.S16 = (g.K + 15) / 16;
    g.NT32 = (Co + 31) / 32;
    return g;
}

// Geometry of a readout layer's Xp.  Its channels are padded to an odd
// multiple of 8: the 8 taps of a fragment lane are then always 8 aligned
// bytes, and the 8-byte LDS reads of neighbouring positions (Ci bytes apart)
// fall on different banks.  Its bytes are indicators of the last frame, 0x3C
// for a time <= T-1 and 0 for later, never and padding: placed in the high
// byte of a half (byte permutes) they are the halves 1.0 and 0 of the A
// operand.
int ro_channels(int Ci)
{
    const int c8 = (Ci + 7) / 8;
    return 8 * (c8 | 1);
}

FGeom make_ro_geom(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride, int pad,
                   int Ho, int Wo)
{
    FGeom g = make_geom(B, T, ro_channels(Ci), Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo);
    g.Cin = Ci;
    g.ind = 1;
    return g;
}

size_t xp_bytes(const FGeom &g)
{
    return spk::align_up((size_t)g.B * g.Hp * g.rowb + kSlack, 256);
}

// B fragment bytes for either fragment shape (the larger of the two).
size_t bp_bytes(const FGeom &g, int np)
{
    const size_t a = (size_t)g.NT * g.S, b = (size_t)g.NT32 * g.S16;
    return (a > b ? a : b) * np * 64 * sizeof(h8);
}

__device__ __forceinline__ h2 as_h2(uint32_t u) { return __builtin_bit_cast(h2, u); }
__device__ __forceinline__ uint32_t as_u(h2 h) { return __builtin_bit_cast(uint32_t, h); }

// [t <= last] for two time bytes, as halves (c = 1025 + last in both halves):
// c - (1024 + t) is a small exact integer, >= 1 iff t <= last.
__device__ __forceinline__ uint32_t upto2(uint32_t x, uint32_t sel, h2 c)
{
    const h2 one = {(_Float16)1.0f, (_Float16)1.0f}, zero = {(_Float16)0.0f, (_Float16)0.0f};
    h2 a = c - as_h2(__builtin_amdgcn_perm(0x64646464u, x, sel));
    return as_u(__builtin_elementwise_min(__builtin_elementwise_max(a, zero), one));
}

// [t == tau] for two time bytes (c = 1024 + tau): 1 - d^2 is 1 at d == 0 and
// <= 0 elsewhere.
__device__ __forceinline__ uint32_t arrive2(uint32_t x, uint32_t sel, h2 c)
{
    const h2 one = {(_Float16)1.0f, (_Float16)1.0f}, zero = {(_Float16)0.0f, (_Float16)0.0f};
    h2 d = as_h2(__builtin_amdgcn_perm(0x64646464u, x, sel)) - c;
    h2 a = one - d * d;
    return as_u(__builtin_elementwise_min(__builtin_elementwise_max(a, zero), one));
}

__device__ __forceinline__ h8 frag_upto(uint2 x, h2 c)
{
    u4 v = {upto2(x.x, kSelLo, c), upto2(x.x, kSelHi, c), upto2(x.y, kSelLo, c), upto2(x.y, kSelHi, c)};
    return __builtin_bit_cast(h8, v);
}

// A fragment of 8 indicator bytes (0x3C or 0): each byte becomes the high
// byte of a half, 0x3C00 = 1.0 or 0.
__device__ __forceinline__ h8 frag_ind(uint2 x)
{
    u4 v = {__builtin_amdgcn_perm(x.y, x.x, 0x010C000Cu), __builtin_amdgcn_perm(x.y, x.x, 0x030C020Cu),
            __builtin_amdgcn_perm(x.y, x.x, 0x050C040Cu), __builtin_amdgcn_perm(x.y, x.x, 0x070C060Cu)};
    return __builtin_bit_cast(h8, v);
}

__device__ __forceinline__ h8 frag_arrive(uint2 x, h2 c)
{
    u4 v = {arrive2(x.x, kSelLo, c), arrive2(x.x, kSelHi, c), arrive2(x.y, kSelLo, c),
            arrive2(x.y, kSelHi, c)};
    return __builtin_bit_cast(h8, v);
}

// 8 bytes at any byte offset of LDS, from three aligned dwords.
__device__ __forceinline__ uint2 lds_read8(const uint8_t *base, int at)
{
    const uint32_t *w = reinterpret_cast<const uint32_t *>(base + (at & ~3));
    const uint32_t w0 = w[0], w1 = w[1], w2 = w[2];
    const uint32_t sh = (uint32_t)(at & 3);
    return make_uint2(__builtin_amdgcn_alignbyte(w1, w0, sh), __builtin_amdgcn_alignbyte(w2, w1, sh));
}

// OR over the 64 lanes of a wave, with row shifts and row broadcasts (DPP)
// rather than LDS permutes; every lane gets the result.
__device__ __forceinline__ uint32_t wave_or(uint32_t x)
{
    x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false);  // row_shr:1
    x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false);  // row_shr:2
    x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false);  // row_shr:4
    x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false);  // row_shr:8
    x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);  // row_bcast:15
    x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);  // row_bcast:31
    return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

// Sum over the 64 lanes of a wave (DPP, as wave_or).
__device__ __forceinline__ int wave_sum(int x)
{
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);
    return __builtin_amdgcn_readlane(x, 63);
}

// Number of the 4 time bytes of x below T.
__device__ __forceinline__ int spikes4(uint32_t x, int T)
{
    int n = 0;
#pragma unroll
    for (int e = 0; e < 4; e++) n += ((x >> (8 * e)) & 0xFFu) < (uint32_t)T ? 1 : 0;
    return n;
}

// Bit t for each of the 8 time bytes, with every time >= 31 (late or never)
// folded onto bit 31; the caller keeps bits below T.
__device__ __forceinline__ uint32_t time_bits(uint2 x)
{
    uint32_t m = 0u;
#pragma unroll
    for (int e = 0; e < 8; e++) {
        const uint32_t t = ((e < 4 ? x.x : x.y) >> (8 * (e & 3))) & 0xFFu;
        m |= 1u << min(t, 31u);
    }
    return m;
}

// Copy n 16-byte words from global memory to LDS with the whole block, as
// direct loads into LDS (no registers): every word of the copy is in flight
// at once.  The caller's barrier waits for them.
__device__ __forceinline__ void copy_to_lds(uint8_t *dst, const uint8_t *src, int n)
{
    typedef __attribute__((address_space(3))) void lds_void;
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6), lane = (int)threadIdx.x & 63;
    for (int w0 = wave * 64; w0 < n; w0 += (int)blockDim.x)
        if (w0 + lane < n)
            __builtin_amdgcn_global_load_lds(src + (size_t)(w0 + lane) * 16,
                                             (lds_void *)(dst + (size_t)w0 * 16), 16, 0, 0);
}

// ------------------------------------------------------------------ packing

// Blocks [0, nb_in): one padded input row each, (b, py): the row's time bytes
// go through LDS from channel rows (coalesced reads) to channels-last order
// (coalesced writes), a pooled input row pooled there from its staged window
// rows; the last block also fills the readable slack.  A pooled input whose
// rows are too wide to stage runs a grid-stride pass over the Xp bytes
// instead.
// Blocks [nb_in, nb_in + maps): one output map o each (maps = the column tiles'
// width, the padding maps written as zeros): its weights are staged in LDS
// and written as B fragments in the packed tap order, as hi/lo halves
// (NP = 2) or halves (NP = 1).  kBig: fragments of the 32x32x16 shape (lane:
// map l % 32, taps 8*(l/32)..+7 of a 16-tap subtile), else of the 16x16x32
// shape (map l % 16, taps 8*(l/16)..+7 of a 32-tap subtile).
template <int NP, bool kHalfW, bool kBig>
__global__ __launch_bounds__(256) void k_pack(const uint8_t *__restrict__ in,
                                              const void *__restrict__ wv, FGeom g, int nb_in,
                                              uint8_t *__restrict__ xp, h8 *__restrict__ bp,
                                              spk::PoolIn pool)
{
    extern __shared__ __align__(16) uint8_t sm[];
    // empty cells: never fires (times), or indicator 0
    const uint8_t fill = g.ind ? (uint8_t)0 : (uint8_t)spk::kNever;
    if ((int)blockIdx.x < nb_in && pool.src && pool.stage < 0) {
        // pooled input too wide to stage: each thread writes Xp bytes
        // (b, py, px, c), the pooling window read from the unpooled map; the
        // Xp body is below 2^31 bytes
        const uint32_t body = (uint32_t)g.B * g.Hp * g.rowb, total = body + kSlack;
        for (uint32_t e = blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (uint32_t)nb_in * blockDim.x) {
            uint8_t v = fill;
            if (e < body) {
                const uint32_t rowi = e / (uint32_t)g.rowb, within = e - rowi * (uint32_t)g.rowb;
                const int b = (int)(rowi / (uint32_t)g.Hp), py = (int)(rowi - (uint32_t)b * g.Hp);
                const int px = (int)(within / (uint32_t)g.Ci), c = (int)within - px * g.Ci;
                const int iy = py - g.pad, ix = px - g.pad;
                if ((unsigned)iy < (unsigned)g.Hi && (unsigned)ix < (unsigned)g.Wi && c < g.Cin) {
                    const long long plane = (long long)b * g.Cin + c;
                    const uint32_t t = spk::pool_cell(pool, plane, iy, ix);
                    if (pool.pooled) pool.pooled[(plane * g.Hi + iy) * g.Wi + ix] = (uint8_t)t;
                    v = g.ind ? (t < (uint32_t)g.T ? (uint8_t)0x3C : (uint8_t)0) : (uint8_t)t;
                }
            }
            xp[e] = v;
        }
        return;
    }
    if ((int)blockIdx.x < nb_in) {
        const int b = blockIdx.x / g.Hp, py = blockIdx.x - b * g.Hp;
        const int iy = py - g.pad;
        uint8_t *row = xp + ((size_t)b * g.Hp + py) * g.rowb;
        // rows of a multiple of 8 bytes start 8-byte aligned: 8-byte fills and stores
        const bool wide = (g.rowb & 7) == 0;
        const uint64_t fill8 = 0x0101010101010101ull * fill;
        auto store_row = [&](auto get8, auto get1) {
            if (wide) {
                for (int e = threadIdx.x; e < g.rowb / 8; e += blockDim.x)
                    reinterpret_cast<uint64_t *>(row)[e] = get8(e);
            } else {
                for (int e = threadIdx.x; e < g.rowb; e += blockDim.x) row[e] = get1(e);
            }
        };
        if ((unsigned)iy < (unsigned)g.Hi) {
            if (wide) {
                for (int e = threadIdx.x; e < g.rowb / 8; e += blockDim.x) reinterpret_cast<uint64_t *>(sm)[e] = fill8;
            } else {
                for (int e = threadIdx.x; e < g.rowb; e += blockDim.x) sm[e] = fill;
            }
            __syncthreads();
            const int n = g.Cin * g.Wi, step = (int)blockDim.x;
            auto put = [&](int e, uint8_t v) {
                const int c = e / g.Wi, x = e - c * g.Wi;
                sm[(x + g.pad) * g.Ci + c] = g.ind ? (v < g.T ? (uint8_t)0x3C : (uint8_t)0) : v;
            };
            if (pool.src) {
                // the input row is pooled here (and kept when asked for)
                spk::pool_row(pool, (long long)b * g.Cin, g.Cin, g.Hi, g.Wi, iy,
                              reinterpret_cast<uint32_t *>(sm + pool.stage),
                              [&](int c, int x, uint8_t v) { put(c * g.Wi + x, v); });
            } else {
                const uint8_t *src = in + (size_t)b * g.Cin * g.Hi * g.Wi + (size_t)iy * g.Wi;
                auto get = [&](int e) {
                    const int c = e / g.Wi, x = e - c * g.Wi;
                    return src[(size_t)c * g.Hi * g.Wi + x];
                };
                int e = threadIdx.x;
                for (; e + 3 * step < n; e += 4 * step) {
                    const uint8_t a = get(e), bb = get(e + step), c = get(e + 2 * step), d = get(e + 3 * step);
                    put(e, a);
                    put(e + step, bb);
                    put(e + 2 * step, c);
                    put(e + 3 * step, d);
                }
                for (; e < n; e += step) put(e, get(e));
            }
            __syncthreads();
            store_row([&](int e) { return reinterpret_cast<const uint64_t *>(sm)[e]; }, [&](int e) { return sm[e]; });
        } else {
            store_row([&](int) { return fill8; }, [&](int) { return fill; });
        }
        if ((int)blockIdx.x == nb_in - 1)
            for (int e = threadIdx.x; e < kSlack; e += blockDim.x) row[g.rowb + e] = fill;
        return;
    }
    // map of this block: the maps are dealt to the XCDs in contiguous runs
    // (block L runs on XCD L % 8), so the blocks whose 16-byte fragment
    // stores share a cache line mostly share an L2 and the line leaves it whole
    const int n_maps = (int)gridDim.x - nb_in, wb = (int)blockIdx.x - nb_in;
    const int xcd = wb & 7, per_x = n_maps >> 3, extra = n_maps & 7;
    const int o = xcd * per_x + min(xcd, extra) + (wb >> 3);
    const int taps = g.Cin * g.Kh * g.Kw;
    float *wl = reinterpret_cast<float *>(sm);
    {
        const int oc = min(o, g.Co - 1);
        auto wget = [&](int e) {
            const size_t at = (size_t)oc * taps + e;
            return kHalfW ? (float)reinterpret_cast<const _Float16 *>(wv)[at]
                          : reinterpret_cast<const float *>(wv)[at];
        };
        const bool real = o < g.Co;  // padding maps: zeros
        const int step = (int)blockDim.x;
        // 16 loads per thread in flight: a deep map's taps arrive in one or two round trips
        for (int e0 = threadIdx.x; e0 < taps; e0 += 16 * step) {
            float v[16];
#pragma unroll
            for (int u = 0; u < 16; u++) v[u] = wget(min(e0 + u * step, taps - 1));  // clamped: no branches
#pragma unroll
            for (int u = 0; u < 16; u++)
                if (e0 + u * step < taps) wl[e0 + u * step] = real ? v[u] : 0.0f;
        }
    }
    __syncthreads();
    // this map's lanes: kBig 2 per 16-tap subtile, else 4 per 32-tap subtile
    const int per = kBig ? 2 : 4, NS = kBig ? g.S16 : g.S;
    const int nt = kBig ? o / 32 : o / 16, col = kBig ? o & 31 : o & 15;
    for (int f = threadIdx.x; f < NS * per; f += blockDim.x) {
        const int s = f / per, h = f - s * per;
        const int lane = col + (kBig ? 32 : 16) * h;
        const int kb = (s * per + h) * 8;
        h8 hi, lo;
        // tap kb = ky*R8 + j, j = kx*Ci + c; the 8 taps step through (ky, j, kx, c);
        // channels c >= Cin (padding of a readout's Xp) have no weight.
        // The 8 LDS addresses first (padding taps read word 0), then the
        // reads together, then the conversions: no branch around a read.
        int ky = kb / g.R8, j = kb - ky * g.R8;
        int kx = j / g.Ci, c = j - kx * g.Ci;
        int at[8];
        bool live[8];
#pragma unroll
        for (int e = 0; e < 8; e++) {
            live[e] = ky < g.Kh && j < g.run && c < g.Cin;
            at[e] = live[e] ? (c * g.Kh + ky) * g.Kw + kx : 0;
            if (++j == g.R8) {
                j = 0;
                ky++;
                kx = 0;
                c = 0;
            } else if (++c == g.Ci) {
                c = 0;
                kx++;
            }
        }
        float wv8[8];
#pragma unroll
        for (int e = 0; e < 8; e++) wv8[e] = wl[at[e]];
#pragma unroll
        for (int e = 0; e < 8; e++) {
            const float w = live[e] ? wv8[e] : 0.0f;
            const _Float16 hw = (_Float16)w;
            hi[e] = hw;
            lo[e] = (_Float16)(w - (float)hw);
        }
        const size_t ts = (size_t)nt * NS + s;
        bp[(ts * NP) * 64 + lane] = hi;
        if (NP == 2) bp[(ts * NP + 1) * 64 + lane] = lo;
    }
}

// Pooled readout input in whole planes, for maps whose planes are small: block
// (b, chunk of kPlaneC channels of Xp) reads the chunk's planes of the
// unpooled map (one contiguous run of bytes) into LDS, pools every cell of
// the chunk (a thread per (channel, cell), kept in pool.pooled when that is
// set) into an LDS tile [cell][channel], then writes every padded pixel's run
// of the chunk's channels, 8 channels per 8-byte store.  The map is read once,
// in full cache lines, instead of in window-row pieces per output row.
// Channels of the chunk past Cin, and the padding, hold the fill (0: not
// fired); block 0 also fills the readable slack.  Needs Xp channels (g.Ci) a
// multiple of 8 (make_ro_geom's are).
constexpr int kPlaneC = 32;

__host__ __device__ inline int align_up16(int n) { return (n + 15) & ~15; }

__host__ __device__ inline bool planes_fit(const FGeom &g, const spk::PoolIn &p)
{
    return g.ind && g.Ci % 8 == 0 && (long long)kPlaneC * (p.H0 * p.W0 + g.Hi * g.Wi) <= 48 * 1024;
}

__global__ __launch_bounds__(256) void k_pack_planes(FGeom g, spk::PoolIn pool, uint8_t *__restrict__ xp)
{
    extern __shared__ __align__(16) uint8_t sm[];
    const int nch = (g.Ci + kPlaneC - 1) / kPlaneC;
    const int b = blockIdx.x / nch, c0 = (blockIdx.x - b * nch) * kPlaneC;
    const int cn = min(kPlaneC, g.Cin - c0);  // real channels of the chunk (<= 0: none)
    const int plane = pool.H0 * pool.W0, cells = g.Hi * g.Wi;
    uint8_t *tile = sm + align_up16(kPlaneC * plane);  // [cell][kPlaneC] indicator bytes
    if (cn > 0) {
        const uint8_t *src = pool.src + ((long long)b * g.Cin + c0) * plane;
        const int n = cn * plane;
        if ((((uintptr_t)src) & 3) == 0) {
            // all of a thread's loads (up to 8 dwords) in flight before any store
            const int n4 = n >> 2;
            for (int e0 = threadIdx.x; e0 < n4; e0 += 8 * (int)blockDim.x) {
                uint32_t v[8];
#pragma unroll
                for (int u = 0; u < 8; u++) {
                    const int e = e0 + u * (int)blockDim.x;
                    v[u] = e < n4 ? reinterpret_cast<const uint32_t *>(src)[e] : 0u;
                }
#pragma unroll
                for (int u = 0; u < 8; u++) {
                    const int e = e0 + u * (int)blockDim.x;
                    if (e < n4) reinterpret_cast<uint32_t *>(sm)[e] = v[u];
                }
            }
            for (int e = 4 * n4 + threadIdx.x; e < n; e += blockDim.x) sm[e] = src[e];
        } else {
            for (int e = threadIdx.x; e < n; e += blockDim.x) sm[e] = src[e];
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < kPlaneC * cells; e += blockDim.x) {
        const int c = e / cells, cell = e - c * cells;
        uint8_t v = 0;
        if (c < cn) {
            const int iy = cell / g.Wi, ix = cell - iy * g.Wi;
            const int y0 = iy * pool.stride - pool.pad, x0 = ix * pool.stride - pool.pad;
            const int ylo = max(y0, 0), yhi = min(y0 + pool.kh, pool.H0);
            const int xlo = max(x0, 0), xhi = min(x0 + pool.kw, pool.W0);
            const uint8_t *pl = sm + c * plane;
            uint32_t m = (uint32_t)spk::kNever;
            if (pool.kh <= 3 && pool.kw <= 3) {
                // windows up to 3 x 3: the nine reads together (cells outside
                // the window or the map read the window's first cell; an empty
                // window, all in the padding, never fires)
                const bool any = ylo < yhi && xlo < xhi;
                const int first = any ? ylo * pool.W0 + xlo : 0;
                uint32_t t[9];
#pragma unroll
                for (int u = 0; u < 9; u++) {
                    const int y = ylo + u / 3, x = xlo + u % 3;
                    t[u] = pl[(y < yhi && x < xhi) ? y * pool.W0 + x : first];
                }
#pragma unroll
                for (int u = 0; u < 9; u++) m = min(m, t[u]);
                if (!any) m = (uint32_t)spk::kNever;
            } else {
                for (int y = ylo; y < yhi; y++)
                    for (int x = xlo; x < xhi; x++) m = min(m, (uint32_t)pl[y * pool.W0 + x]);
            }
            if (pool.pooled) pool.pooled[((long long)b * g.Cin + c0 + c) * cells + cell] = (uint8_t)m;
            v = m < (uint32_t)g.T ? (uint8_t)0x3C : (uint8_t)0;
        }
        tile[cell * kPlaneC + c] = v;
    }
    __syncthreads();
    const int ngrp = min(kPlaneC, g.Ci - c0) / 8;
    for (int e = threadIdx.x; e < g.Hp * g.Wp * ngrp; e += blockDim.x) {
        const int pix = e / ngrp, q = e - pix * ngrp;
        const int py = pix / g.Wp, px = pix - py * g.Wp;
        const int iy = py - g.pad, ix = px - g.pad;
        uint2 v = make_uint2(0u, 0u);
        if ((unsigned)iy < (unsigned)g.Hi && (unsigned)ix < (unsigned)g.Wi)
            v = *reinterpret_cast<const uint2 *>(tile + (iy * g.Wi + ix) * kPlaneC + q * 8);
        *reinterpret_cast<uint2 *>(xp + ((size_t)(b * g.Hp + py) * g.Wp + px) * g.Ci + c0 + q * 8) = v;
    }
    if (blockIdx.x == 0)
        for (int e = threadIdx.x; e < kSlack; e += blockDim.x) xp[(size_t)g.B * g.Hp * g.rowb + e] = 0;
}

// Launch of the packing pass for a fragment shape.  in_rows: pack the input
// (nb_in blocks); weights: pack the B fragments (one block per map).
void launch_pack(const uint8_t *in, const void *w, bool half_w, bool big, const FGeom &g,
                 uint8_t *xp, h8 *bp, hipStream_t s, bool in_rows = true, bool weights = true,
                 const spk::PoolIn *pool = nullptr)
{
    // a pooled input row stages its window rows past the row buffer when
    // they fit; otherwise its cells are pooled one by one
    spk::PoolIn pl = pool ? *pool : spk::PoolIn{};
    pl.stage = -1;
    const size_t stage_at = spk::align_up((size_t)g.rowb, 16);
    if (pool && stage_at + spk::pool_stage_bytes(pl, g.Cin) <= 64 * 1024) pl.stage = (int)stage_at;
    // input blocks: one per padded row, or 1024 Xp bytes each (cells pooled one by one)
    const int nb_in = !in_rows ? 0
                      : pool && pl.stage < 0 ? spk::ceil_div((long long)g.B * g.Hp * g.rowb + kSlack, 1024)
                                             : g.B * g.Hp;
    const int maps = weights ? (big ? g.NT32 * 32 : g.NT * 16) : 0;
    size_t lds = std::max(in_rows ? (size_t)g.rowb : (size_t)0,
                          weights ? (size_t)g.Cin * g.Kh * g.Kw * sizeof(float) : (size_t)0);
    const dim3 grid(nb_in + maps), blk(256);
    if (pool && in_rows)
        lds = std::max(weights ? (size_t)g.Cin * g.Kh * g.Kw * sizeof(float) : (size_t)0,
                       pl.stage >= 0 ? stage_at + spk::pool_stage_bytes(pl, g.Cin) : (size_t)0);
    if (big) {
        if (half_w) hipLaunchKernelGGL((k_pack<1, true, true>), grid, blk, lds, s, in, w, g, nb_in, xp, bp, pl);
        else hipLaunchKernelGGL((k_pack<2, false, true>), grid, blk, lds, s, in, w, g, nb_in, xp, bp, pl);
    } else {
        if (half_w) hipLaunchKernelGGL((k_pack<1, true, false>), grid, blk, lds, s, in, w, g, nb_in, xp, bp, pl);
        else hipLaunchKernelGGL((k_pack<2, false, false>), grid, blk, lds, s, in, w, g, nb_in, xp, bp, pl);
    }
}

// -------------------------------------------------------------------- firing

// Byte range of Xp holding the input rows of output positions [p0, p1].
__host__ __device__ inline void group_range(const FGeom &g, int p0, int p1, long long &h0,
                                            long long &h1)
{
    const int HoWo = g.Ho * g.Wo;
    const int b0 = p0 / HoWo, y0 = (p0 - b0 * HoWo) / g.Wo;
    const int b1 = p1 / HoWo, y1 = (p1 - b1 * HoWo) / g.Wo;
    h0 = ((long long)b0 * g.Hp + (long long)y0 * g.stride) * g.rowb;
    h1 = ((long long)b1 * g.Hp + (long long)y1 * g.stride + g.Kh) * g.rowb;
}

// SM: the layer's subtile count (exact); kR: row tiles per wave.
template <int SM, int NP, int kR>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
void k_fire_fast(const uint8_t *__restrict__ xp, const h8 *__restrict__ bp, FGeom g, float theta,
                 int iters, int vec_store, uint8_t *__restrict__ out_t, float *__restrict__ out_v)
{
    constexpr int kRows = kWaves * kR * 16;  // positions per block iteration
    extern __shared__ __align__(16) uint8_t halo[];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nt = blockIdx.y;
    const int o = nt * 16 + (lane & 15);
    const int HoWo = g.Ho * g.Wo;
    const int Q8 = g.R8 / 8;  // fragment octets per kernel row

    // Xp offset of each lane group's octet in each subtile (relative to the
    // row's window origin), once per block: kernel row ky, byte j0 of its run
    __shared__ int s_off[SM * 4];
    __shared__ uint32_t s_bits[kWaves];
    __shared__ int s_count[kWaves];
    if (threadIdx.x < SM * 4) {
        const int q = threadIdx.x;  // = s * 4 + lane group
        const int ky = q / Q8, jq = q - ky * Q8;
        s_off[q] = (ky < g.Kh ? ky : 0) * g.rowb + jq * 8;  // octets past K: any byte (B is zero)
    }

    // B fragments of the column tile, all subtiles, in registers
    h8 bw[SM][NP];
#pragma unroll
    for (int s = 0; s < SM; s++) {
#pragma unroll
        for (int q = 0; q < NP; q++) bw[s][q] = bp[((size_t)(nt * SM + s) * NP + q) * 64 + lane];
    }

    for (int it = 0; it < iters; it++) {
        const int pb0 = (blockIdx.x * iters + it) * kRows;
        if (pb0 >= g.P) break;
        const int pb1 = min(g.P, pb0 + kRows) - 1;
        long long h0, h1;
        group_range(g, pb0, pb1, h0, h1);
        const long long a0 = h0 & ~15ll;
        const int nvec = (int)((h1 - a0 + 15) >> 4) + 1;  // 16-byte words, one past the end
        __syncthreads();  // the previous group's halo is no longer read
        // copy the group's Xp bytes, noting which steps they fire at and how
        // many of them fire at all (over a superset of the group's taps)
        const uint32_t tmask = g.T >= 32 ? ~0u : ((1u << g.T) - 1u);
        {
            const uint4 *src = reinterpret_cast<const uint4 *>(xp + a0);
            uint4 *dst = reinterpret_cast<uint4 *>(halo);
            uint32_t hb = 0u;
            int hc = 0;
            int i = threadIdx.x;
            for (; i + kThreads < nvec; i += 2 * kThreads) {
                const uint4 v = src[i], u = src[i + kThreads];
                dst[i] = v;
                dst[i + kThreads] = u;
                hb |= time_bits(make_uint2(v.x, v.y)) | time_bits(make_uint2(v.z, v.w)) |
                      time_bits(make_uint2(u.x, u.y)) | time_bits(make_uint2(u.z, u.w));
                hc += spikes4(v.x, g.T) + spikes4(u.x, g.T);  // density from a quarter of the bytes
            }
            for (; i < nvec; i += kThreads) {
                const uint4 v = src[i];
                dst[i] = v;
                hb |= time_bits(make_uint2(v.x, v.y)) | time_bits(make_uint2(v.z, v.w));
                hc += spikes4(v.x, g.T);
            }
            hb = wave_or(hb);
            hc = wave_sum(hc);
            if (lane == 0) {
                s_bits[wave] = hb;
                s_count[wave] = hc;
            }
        }
        __syncthreads();
        uint32_t all = 0u;
        int spikes = 0;
#pragma unroll
        for (int w = 0; w < kWaves; w++) {
            all |= s_bits[w];
            spikes += s_count[w];
        }
        all &= tmask;
        const int tmin = all ? __builtin_ctz(all) : g.T;
        const int tmax = all ? 31 - __builtin_clz(all) : -1;
        const int span = tmax >= tmin ? tmax - tmin + 1 : 1;
        // Expected arrivals per (step, subtile) of a wave: 16*kR rows x 32 taps
        // at the group's spike density, spread over the active steps.  Below
        // about one, enough subtiles are empty at a step for the arrival form
        // (1.5x the work of a cumulative step per computed subtile) to win.
        const float lambda = (float)(16 * kR * 32) * (float)spikes / ((float)nvec * 4.0f * (float)span);
        const bool delta = lambda < 1.1f;

        // ---- A side: 8 time bytes per (row tile, subtile) into registers
        uint2 ab[kR][SM];
#pragma unroll
        for (int r = 0; r < kR; r++) {
            const int p = pb0 + (wave * kR + r) * 16 + (lane & 15);
            const int pc = min(p, g.P - 1);
            const int b = pc / HoWo, rem = pc - b * HoWo;
            const int y = rem / g.Wo, x = rem - y * g.Wo;
            const int base = (int)(((long long)b * g.Hp + (long long)y * g.stride) * g.rowb +
                                   (long long)x * g.stride * g.Ci - a0);
#pragma unroll
            for (int s = 0; s < SM; s++) ab[r][s] = lds_read8(halo, base + s_off[s * 4 + (lane >> 4)]);
        }
        // Arrival-time masks per subtile, OR over the wave, for the arrival
        // form only.  A mask may hold extra bits (padding taps, late times
        // folded onto bit 31 when T == 32): an extra subtile adds zeros.
        uint32_t ms[SM];
#pragma unroll
        for (int s = 0; s < SM; s++) ms[s] = 0u;
        if (delta) {
#pragma unroll
            for (int s = 0; s < SM; s++) {
                uint32_t m = 0u;
#pragma unroll
                for (int r = 0; r < kR; r++) m |= time_bits(ab[r][s]);
                ms[s] = wave_or(m) & tmask;
            }
        }

        uint32_t valid = 0u;
#pragma unroll
        for (int r = 0; r < kR; r++)
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int p = pb0 + (wave * kR + r) * 16 + (lane >> 4) * 4 + i;
                if (p < g.P && o < g.Co) valid |= 1u << (r * 4 + i);
            }
        // Fired and valid neurons, as lane masks per accumulator element
        // (scalar registers); the per-lane times and key potentials are only
        // touched at steps where something new fires.
        uint64_t vmask[kR * 4], fmask[kR * 4];
#pragma unroll
        for (int e = 0; e < kR * 4; e++) {
            vmask[e] = __ballot((valid >> e) & 1u);
            fmask[e] = 0ull;
        }
        uint32_t tf[kR] = {};
        float vk[kR][4] = {};
        f4 acc[kR];
#pragma unroll
        for (int r = 0; r < kR; r++) acc[r] = f4{0.0f, 0.0f, 0.0f, 0.0f};

        for (int tau = 0; tau < g.T; tau++) {
            if (delta) {
                const uint32_t cb = 0x6400u + (uint32_t)tau;  // half 1024 + tau
                const h2 cc = as_h2(cb | (cb << 16));
#pragma unroll
                for (int s = 0; s < SM; s++) {
                    if ((ms[s] >> tau) & 1u) {
                        h8 a[kR];
#pragma unroll
                        for (int r = 0; r < kR; r++) a[r] = frag_arrive(ab[r][s], cc);
#pragma unroll
                        for (int q = 0; q < NP; q++)
#pragma unroll
                            for (int r = 0; r < kR; r++)
                                acc[r] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[r], bw[s][q], acc[r], 0, 0, 0);
                    }
                }
            } else if (tau >= tmin && tau <= tmax) {
                const uint32_t cb = 0x6401u + (uint32_t)tau;  // half 1025 + tau
                const h2 cc = as_h2(cb | (cb << 16));
#pragma unroll
                for (int r = 0; r < kR; r++) acc[r] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int s = 0; s < SM; s++) {
                    h8 a[kR];
#pragma unroll
                    for (int r = 0; r < kR; r++) a[r] = frag_upto(ab[r][s], cc);
#pragma unroll
                    for (int q = 0; q < NP; q++)
#pragma unroll
                        for (int r = 0; r < kR; r++)
                            acc[r] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[r], bw[s][q], acc[r], 0, 0, 0);
                }
            }
            // crossings of theta at this step (first crossing only)
            uint64_t any = 0ull, nm[kR * 4];
#pragma unroll
            for (int r = 0; r < kR; r++)
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const int e = r * 4 + i;
                    nm[e] = __ballot(acc[r][i] > theta) & vmask[e] & ~fmask[e];
                    any |= nm[e];
                }
            if (any) {
                const uint64_t me = 1ull << lane;
#pragma unroll
                for (int r = 0; r < kR; r++)
#pragma unroll
                    for (int i = 0; i < 4; i++) {
                        const int e = r * 4 + i;
                        if (nm[e] & me) {
                            vk[r][i] = acc[r][i];
                            tf[r] = (tf[r] & ~(0xFFu << (8 * i))) | ((uint32_t)tau << (8 * i));
                        }
                        fmask[e] |= nm[e];
                    }
            }
            if (tau >= tmax) break;  // no later arrival: the potentials stay as they are
        }
        uint32_t fired = 0u;
#pragma unroll
        for (int e = 0; e < kR * 4; e++) fired |= ((fmask[e] >> lane) & 1ull) ? (1u << e) : 0u;

        // times and key potentials: t_f and V[t_f], or NEVER and V[T-1]
#pragma unroll
        for (int r = 0; r < kR; r++) {
            uint32_t tb = 0u;
            float v[4];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const bool f = (fired >> (r * 4 + i)) & 1u;
                v[i] = f ? vk[r][i] : acc[r][i];
                tb |= (f ? ((tf[r] >> (8 * i)) & 0xFFu) : (uint32_t)spk::kNever) << (8 * i);
            }
            const int p0 = pb0 + (wave * kR + r) * 16 + (lane >> 4) * 4;
            if (vec_store) {
                // 4 positions of one sample, 4-aligned (Ho*Wo % 4 == 0)
                if ((valid >> (r * 4)) & 1u) {
                    const int b = p0 / HoWo, rem = p0 - b * HoWo;
                    const size_t n = ((size_t)b * g.Co + o) * HoWo + rem;
                    *reinterpret_cast<uint32_t *>(out_t + n) = tb;
                    *reinterpret_cast<float4 *>(out_v + n) = make_float4(v[0], v[1], v[2], v[3]);
                }
            } else {
#pragma unroll
                for (int i = 0; i < 4; i++)
                    if ((valid >> (r * 4 + i)) & 1u) {
                        const int p = p0 + i;
                        const int b = p / HoWo, rem = p - b * HoWo;
                        const size_t n = ((size_t)b * g.Co + o) * HoWo + rem;
                        out_t[n] = (uint8_t)(tb >> (8 * i));
                        out_v[n] = v[i];
                    }
            }
        }
    }
}

typedef float f16v __attribute__((ext_vector_type(16)));

// The 32x32x16 form of the firing kernel (the 16x16x32 instruction runs at
// half the rate on this chip): a wave owns 32 positions x 32 maps, B
// fragments of all SK subtiles (16 taps each) stay in registers, and so do
// the 8 time bytes per subtile of the wave's A fragments; their conversion to
// halves is redone at each step rather than kept, which saves registers.
// Accumulator element e of lane l is position row 8*(e/4) + 4*(l/32) + e%4,
// map l % 32.
template <int SK, int NP>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
void k_fire32(const uint8_t *__restrict__ xp, const h8 *__restrict__ bp, FGeom g, float theta,
              int iters, int vec_store, uint8_t *__restrict__ out_t, float *__restrict__ out_v)
{
    constexpr int kRows = kWaves * 32;  // positions per block iteration
    // LDS: [time bytes of every wave's A fragments: wave][subtile][lane] | halo]
    extern __shared__ __align__(16) uint8_t lds[];
    uint2 *astage = reinterpret_cast<uint2 *>(lds) + (size_t)(threadIdx.x >> 6) * SK * 64;
    uint8_t *halo = lds + (size_t)kWaves * SK * 64 * sizeof(uint2);
    __shared__ int s_off[SK * 2];
    __shared__ uint32_t s_bits[kWaves];
    __shared__ int s_count[kWaves];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nt = blockIdx.y;
    const int o = nt * 32 + (lane & 31);
    const int HoWo = g.Ho * g.Wo;
    const int Q8 = g.R8 / 8;
    if (threadIdx.x < SK * 2) {
        const int q = threadIdx.x;  // = s * 2 + lane half
        const int ky = q / Q8, jq = q - ky * Q8;
        s_off[q] = (ky < g.Kh ? ky : 0) * g.rowb + jq * 8;  // octets past K: any byte (B is zero)
    }
    h8 bw[SK][NP];
#pragma unroll
    for (int s = 0; s < SK; s++)
#pragma unroll
        for (int q = 0; q < NP; q++) bw[s][q] = bp[((size_t)(nt * SK + s) * NP + q) * 64 + lane];

    for (int it = 0; it < iters; it++) {
        const int pb0 = (blockIdx.x * iters + it) * kRows;
        if (pb0 >= g.P) break;
        const int pb1 = min(g.P, pb0 + kRows) - 1;
        long long h0, h1;
        group_range(g, pb0, pb1, h0, h1);
        const long long a0 = h0 & ~15ll;
        const int nvec = (int)((h1 - a0 + 15) >> 4) + 1;  // 16-byte words, one past the end
        const uint32_t tmask = g.T >= 32 ? ~0u : ((1u << g.T) - 1u);
        __syncthreads();  // the previous group's halo is no longer read
        {
            const uint4 *src = reinterpret_cast<const uint4 *>(xp + a0);
            uint4 *dst = reinterpret_cast<uint4 *>(halo);
            uint32_t hb = 0u;
            int hc = 0;
            int i = threadIdx.x;
            for (; i + kThreads < nvec; i += 2 * kThreads) {
                const uint4 v = src[i], u = src[i + kThreads];
                dst[i] = v;
                dst[i + kThreads] = u;
                hb |= time_bits(make_uint2(v.x, v.y)) | time_bits(make_uint2(v.z, v.w)) |
                      time_bits(make_uint2(u.x, u.y)) | time_bits(make_uint2(u.z, u.w));
                hc += spikes4(v.x, g.T) + spikes4(u.x, g.T);  // density from a quarter of the bytes
            }
            for (; i < nvec; i += kThreads) {
                const uint4 v = src[i];
                dst[i] = v;
                hb |= time_bits(make_uint2(v.x, v.y)) | time_bits(make_uint2(v.z, v.w));
                hc += spikes4(v.x, g.T);
            }
            hb = wave_or(hb);
            hc = wave_sum(hc);
            if (lane == 0) {
                s_bits[wave] = hb;
                s_count[wave] = hc;
            }
        }
        __syncthreads();
        uint32_t all = 0u;
        int spikes = 0;
#pragma unroll
        for (int w = 0; w < kWaves; w++) {
            all |= s_bits[w];
            spikes += s_count[w];
        }
        all &= tmask;
        const int tmin = all ? __builtin_ctz(all) : g.T;
        const int tmax = all ? 31 - __builtin_clz(all) : -1;
        const int span = tmax >= tmin ? tmax - tmin + 1 : 1;
        // expected arrivals per (step, subtile): 32 rows x 16 taps
        const float lambda = 512.0f * (float)spikes / ((float)nvec * 4.0f * (float)span);
        const bool delta = lambda < 1.1f;

        uint32_t ms[SK];
        {
            uint2 ab[SK];
            const int p = pb0 + wave * 32 + (lane & 31);
            const int pc = min(p, g.P - 1);
            const int b = pc / HoWo, rem = pc - b * HoWo;
            const int y = rem / g.Wo, x = rem - y * g.Wo;
            const int base = (int)(((long long)b * g.Hp + (long long)y * g.stride) * g.rowb +
                                   (long long)x * g.stride * g.Ci - a0);
#pragma unroll
            for (int s = 0; s < SK; s++) ab[s] = lds_read8(halo, base + s_off[s * 2 + (lane >> 5)]);
#pragma unroll
            for (int s = 0; s < SK; s++) ms[s] = 0u;
            if (delta) {
#pragma unroll
                for (int s = 0; s < SK; s++) ms[s] = wave_or(time_bits(ab[s])) & tmask;
            }
            // each lane reads back only what it wrote: no barrier needed
#pragma unroll
            for (int s = 0; s < SK; s++) astage[s * 64 + lane] = ab[s];
        }

        uint32_t valid = 0u;
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const int p = pb0 + wave * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
            valid |= (p < g.P && o < g.Co) ? (1u << e) : 0u;
        }
        uint32_t fired = 0u;
        uint32_t tf[4] = {0u, 0u, 0u, 0u};
        float vk[16];
#pragma unroll
        for (int e = 0; e < 16; e++) vk[e] = 0.0f;
        f16v acc;
#pragma unroll
        for (int e = 0; e < 16; e++) acc[e] = 0.0f;

        for (int tau = 0; tau < g.T; tau++) {
            // keeps the staged bytes in LDS: they are read again at every step
            asm volatile("" ::: "memory");
            if (delta) {
                const uint32_t cb = 0x6400u + (uint32_t)tau;  // half 1024 + tau
                const h2 cc = as_h2(cb | (cb << 16));
#pragma unroll
                for (int s = 0; s < SK; s++) {
                    if ((ms[s] >> tau) & 1u) {
                        const h8 a = frag_arrive(astage[s * 64 + lane], cc);
#pragma unroll
                        for (int q = 0; q < NP; q++)
                            acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bw[s][q], acc, 0, 0, 0);
                    }
                }
            } else if (tau >= tmin && tau <= tmax) {
                const uint32_t cb = 0x6401u + (uint32_t)tau;  // half 1025 + tau
                const h2 cc = as_h2(cb | (cb << 16));
#pragma unroll
                for (int e = 0; e < 16; e++) acc[e] = 0.0f;
#pragma unroll
                for (int s = 0; s < SK; s++) {
                    const h8 a = frag_upto(astage[s * 64 + lane], cc);
#pragma unroll
                    for (int q = 0; q < NP; q++)
                        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bw[s][q], acc, 0, 0, 0);
                }
            }
            // crossings of theta at this step (first crossing only)
            uint32_t now = 0u;
#pragma unroll
            for (int e = 0; e < 16; e++) now |= (acc[e] > theta) ? (1u << e) : 0u;
            now &= valid & ~fired;
            if (__ballot(now != 0u)) {
#pragma unroll
                for (int e = 0; e < 16; e++)
                    if ((now >> e) & 1u) {
                        vk[e] = acc[e];
                        tf[e >> 2] = (tf[e >> 2] & ~(0xFFu << (8 * (e & 3)))) | ((uint32_t)tau << (8 * (e & 3)));
                    }
                fired |= now;
            }
            if (tau >= tmax) break;  // no later arrival: the potentials stay as they are
        }

        // times and key potentials: t_f and V[t_f], or NEVER and V[T-1]
#pragma unroll
        for (int g4 = 0; g4 < 4; g4++) {
            uint32_t tb = 0u;
            float v[4];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int e = g4 * 4 + i;
                const bool f = (fired >> e) & 1u;
                v[i] = f ? vk[e] : acc[e];
                tb |= (f ? ((tf[g4] >> (8 * i)) & 0xFFu) : (uint32_t)spk::kNever) << (8 * i);
            }
            const int p0 = pb0 + wave * 32 + 8 * g4 + 4 * (lane >> 5);
            if (vec_store) {
                // 4 positions of one sample, 4-aligned (Ho*Wo % 4 == 0)
                if (p0 < g.P && o < g.Co) {
                    const int b = p0 / HoWo, rem = p0 - b * HoWo;
                    const size_t n = ((size_t)b * g.Co + o) * HoWo + rem;
                    *reinterpret_cast<uint32_t *>(out_t + n) = tb;
                    *reinterpret_cast<float4 *>(out_v + n) = make_float4(v[0], v[1], v[2], v[3]);
                }
            } else {
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const int p = p0 + i;
                    if (p < g.P && o < g.Co) {
                        const int b = p / HoWo, rem = p - b * HoWo;
                        const size_t n = ((size_t)b * g.Co + o) * HoWo + rem;
                        out_t[n] = (uint8_t)(tb >> (8 * i));
                        out_v[n] = v[i];
                    }
                }
            }
        }
    }
}

// ------------------------------------------------------------------ readout
//
// Readout layers (theta = +inf) need only V at the last step: one GEMM on the
// final frame [time <= T-1], split over K, on the indicator bytes of
// make_ro_geom (an A fragment is four byte permutes).  A block of 4 waves owns a column
// tile (32 maps) and a run of 4*kRoKC subtiles; wave w keeps the B fragments
// of subtiles w*kRoKC.. in registers.  The block walks row groups of 32
// positions: the Xp bytes that a group and its K run touch are staged in LDS
// (the next group's bytes are fetched into registers while this group's
// products run, when they fit kRoPre words per thread), each wave reads all
// of its A octets and then runs its products back to back, and the four
// partial tiles are added in LDS in wave order and written to
// part[split][map][position] with each map's 32 positions in one coalesced
// store.  k_readout_sum adds the splits in order.
constexpr int kRoKC = 16;
constexpr int kRoSteps = kWaves * kRoKC;
constexpr int kRoStride = 33;                                     // partial tiles: [wave][row][map], padded
constexpr int kRoRed = kWaves * 32 * kRoStride * (int)sizeof(float);  // LDS of the partial tiles
constexpr int kRoPre = 8;                                         // prefetched 16-byte words per thread

__host__ __device__ inline void ro_range(const FGeom &g, int p0, int p1, int sp, long long &h0,
                                         long long &h1)
{
    const int HoWo = g.Ho * g.Wo;
    const int kb0 = sp * kRoSteps * 16, kb1 = min(g.K, (sp + 1) * kRoSteps * 16);
    const int ky_lo = min(kb0 / g.R8, g.Kh - 1), ky_hi = min((kb1 - 1) / g.R8, g.Kh - 1);
    const int b0 = p0 / HoWo, y0 = (p0 - b0 * HoWo) / g.Wo;
    const int b1 = p1 / HoWo, y1 = (p1 - b1 * HoWo) / g.Wo;
    h0 = ((long long)b0 * g.Hp + (long long)y0 * g.stride + ky_lo) * g.rowb;
    h1 = ((long long)b1 * g.Hp + (long long)y1 * g.stride + ky_hi + 1) * g.rowb;
}

// Staged range of row group rg: first 16-aligned byte a0 and 16-byte words.
__device__ __forceinline__ void ro_words(const FGeom &g, int rg, int sp, long long &a0, int &nvec)
{
    const int p0 = rg * 32, p1 = min(g.P, p0 + 32) - 1;
    long long h0, h1;
    ro_range(g, p0, p1, sp, h0, h1);
    a0 = h0 & ~15ll;
    nvec = (int)((h1 - a0 + 15) >> 4) + 1;
}

// kPre: the staged range of every group fits kRoPre words per thread and the
// next group's words are loaded into registers during this group's products;
// otherwise each group is copied straight into LDS before its products.
template <int NP, bool kPre>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
void k_readout32(const uint8_t *__restrict__ xp, const h8 *__restrict__ bp, FGeom g, int iters,
                 int n_groups, int nx, float *__restrict__ part)
{
    // LDS: [partial tiles: wave][position row][map] | halo]
    extern __shared__ __align__(16) uint8_t lds[];
    float *red = reinterpret_cast<float *>(lds);
    uint8_t *halo = lds + kRoRed;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    // Work items j = (split, column tile) major, run of row groups minor.
    // Blocks go to the 8 XCDs in turn (block L to XCD L % 8); XCD k takes a
    // contiguous share of the items, so it reads the B fragments of only
    // about 1/8 of the (split, tile) pairs and they stay in its L2.
    const int n_items = (int)gridDim.x, xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
    const int per = n_items >> 3, extra = n_items & 7;
    const int j = xcd * per + min(xcd, extra) + slot;
    const int bx = j % nx, pair = j / nx;
    const int nt = pair % g.NT32, sp = pair / g.NT32;
    const int sw0 = sp * kRoSteps + wave * kRoKC;            // this wave's first subtile
    const int nsw = max(0, min(kRoKC, g.S16 - sw0));          // and how many it has
    const int HoWo = g.Ho * g.Wo;
    const int Q8 = g.R8 / 8;
    const int kb0 = sp * kRoSteps * 16;
    const int ky_lo = min(kb0 / g.R8, g.Kh - 1);
    const int rg0 = bx * iters;
    const int rg_end = min(n_groups, rg0 + iters);

    // the first group's words are requested before the B fragments
    u4 pre[kPre ? kRoPre : 1];
    auto fetch = [&](int rg, long long &a0, int &nvec) {
        ro_words(g, rg, sp, a0, nvec);
        const u4 *src = reinterpret_cast<const u4 *>(xp + a0);
#pragma unroll
        for (int u = 0; u < (kPre ? kRoPre : 1); u++) {
            const int i = (int)threadIdx.x + u * kThreads;
            if (i < nvec) pre[u] = src[i];
        }
    };
    auto commit = [&](int nvec) {
        u4 *dst = reinterpret_cast<u4 *>(halo);
#pragma unroll
        for (int u = 0; u < (kPre ? kRoPre : 1); u++) {
            const int i = (int)threadIdx.x + u * kThreads;
            if (i < nvec) dst[i] = pre[u];
        }
    };
    long long a0 = 0;
    int nvec = 0;
    if (kPre && rg0 < rg_end) fetch(rg0, a0, nvec);

    // B fragments; the subtiles past the wave's share (past S16) are zero,
    // so their products add nothing and every wave runs the same
    // straight-line code
    h8 bw[kRoKC][NP];
#pragma unroll
    for (int s = 0; s < kRoKC; s++) {
        const int sc = min(sw0 + s, g.S16 - 1);
#pragma unroll
        for (int q = 0; q < NP; q++) {
            const h8 v = bp[((size_t)(nt * g.S16 + sc) * NP + q) * 64 + lane];
            bw[s][q] = s < nsw ? v : (h8)(_Float16)0.0f;
        }
    }
    // Per subtile: the octet's offset from a position's window origin, the
    // same for every row group.  Octets past K read a row of the halo (their
    // weights are zero).
    int offs[kRoKC];
    {
        const int q0 = 2 * sw0 + (lane >> 5);
        int ky = q0 / Q8, jq = q0 - ky * Q8;
#pragma unroll
        for (int s = 0; s < kRoKC; s++) {
            offs[s] = ky < g.Kh ? ky * g.rowb + jq * 8 : ky_lo * g.rowb;
            jq += 2;
            while (jq >= Q8) {
                jq -= Q8;
                ky++;
            }
        }
    }
    if (kPre && rg0 < rg_end) {
        commit(nvec);
        __syncthreads();
    }

    for (int rg = rg0; rg < rg_end; rg++) {
        const int p0 = rg * 32;
        long long a0n = 0;
        int nvn = 0;
        if (kPre) {
            // the next group's words travel while this group's products run
            if (rg + 1 < rg_end) fetch(rg + 1, a0n, nvn);
        } else {
            ro_words(g, rg, sp, a0, nvec);
            __syncthreads();  // the previous group's halo and partial tiles are no longer read
            copy_to_lds(halo, xp + a0, nvec);
            __syncthreads();
        }

        // all of the wave's octets are read before the products start
        uint2 ab[kRoKC];
        {
            const int p = p0 + (lane & 31);
            const int pc = min(p, g.P - 1);
            const int b = pc / HoWo, rem = pc - b * HoWo;
            const int y = rem / g.Wo, x = rem - y * g.Wo;
            const int base = (int)(((long long)b * g.Hp + (long long)y * g.stride) * g.rowb +
                                   (long long)x * g.stride * g.Ci - a0);
            // every octet starts at a multiple of 8 (channels padded to 8)
#pragma unroll
            for (int s = 0; s < kRoKC; s++)
                ab[s] = *reinterpret_cast<const uint2 *>(halo + base + offs[s]);
        }
        f16v acc;
#pragma unroll
        for (int e = 0; e < 16; e++) acc[e] = 0.0f;
#pragma unroll
        for (int s = 0; s < kRoKC; s++) {
            const h8 a = frag_ind(ab[s]);
#pragma unroll
            for (int q = 0; q < NP; q++)
                acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bw[s][q], acc, 0, 0, 0);
        }
        // element (e, l): position row 8*(e/4) + 4*(l/32) + e%4, map l % 32
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const int r = 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
            red[(wave * 32 + r) * kRoStride + (lane & 31)] = acc[e];
        }
        __syncthreads();
        for (int i = threadIdx.x; i < 1024; i += kThreads) {
            const int o_l = i >> 5, r = i & 31;
            const int at = r * kRoStride + o_l, wst = 32 * kRoStride;
            const float v = ((red[at] + red[wst + at]) + red[2 * wst + at]) + red[3 * wst + at];
            const int p = p0 + r, o = nt * 32 + o_l;
            if (p < g.P && o < g.Co) part[((size_t)sp * g.Co + o) * g.P + p] = v;
        }
        if (kPre && rg + 1 < rg_end) {
            // every wave is past its halo reads (the barrier above): the next
            // group's words replace them
            commit(nvn);
            a0 = a0n;
            nvec = nvn;
        }
        if (kPre) __syncthreads();  // next halo in place; partial tiles free
    }
}

// V = sum of the splits in order; readout neurons never fire.
__global__ void k_readout_sum(const float *__restrict__ part, FGeom g, int splits,
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

// Kernel variants.  Both keep the B fragments of all subtiles in registers:
// the 32x32x16 one (S16 subtiles: 2*S16 + 4*NP*S16 registers of operands) up
// to 19 float or 31 half subtiles, else the 16x16x32 one (R*S*4 + NP*S*4,
// R = 2 row tiles per wave, or 1 for deeper layers) up to 15 float or 24 half
// subtiles.
enum Variant { kNone = 0, kV32 = 1, kV16 = 2 };

Variant variant_of(const FGeom &g, bool half_w)
{
    if (g.S16 <= (half_w ? 31 : 19)) return kV32;
    if (g.S <= (half_w ? 24 : 15)) return kV16;
    return kNone;
}

constexpr int rows_per_wave(int S, int NP) { return S <= (NP == 2 ? 9 : 12) ? 2 : 1; }

int group_rows(const FGeom &g, bool half_w)
{
    if (variant_of(g, half_w) == kV32) return kWaves * 32;
    return kWaves * rows_per_wave(g.S, half_w ? 1 : 2) * 16;
}

long long max_group_bytes(const FGeom &g, bool half_w)
{
    const int rows = group_rows(g, half_w);
    long long best = 0;
    for (long long p0 = 0; p0 < g.P; p0 += rows) {
        const int p1 = (int)std::min<long long>(g.P, p0 + rows) - 1;
        long long h0, h1;
        group_range(g, (int)p0, p1, h0, h1);
        best = std::max(best, h1 - (h0 & ~15ll));
    }
    return best;
}

size_t halo_lds(long long group_bytes) { return spk::align_up((size_t)group_bytes + 32, 16); }

// LDS bytes of the largest row group of a geometry, remembered per geometry
// (the exact maximum walks every group once).
size_t group_lds(const FGeom &g, bool half_w)
{
    typedef std::tuple<int, int, int, int, int, int, int, int, int, int> Key;
    static std::mutex mu;
    static std::map<Key, size_t> memo;
    const Key key{g.B, g.Ci, g.Hi, g.Wi, g.Kh, g.Kw, g.stride, g.pad, g.Ho, (int)half_w};
    {
        std::lock_guard<std::mutex> lock(mu);
        auto it = memo.find(key);
        if (it != memo.end()) return it->second;
    }
    const size_t v = halo_lds(max_group_bytes(g, half_w));
    std::lock_guard<std::mutex> lock(mu);
    if (memo.size() > 4096) memo.clear();
    memo[key] = v;
    return v;
}

template <int SM, int NP>
void launch_fire(const uint8_t *xp, const h8 *bp, const FGeom &g, float theta, int iters,
                 int vec_store, size_t lds, uint8_t *ot, float *ov, hipStream_t s)
{
    constexpr int R = rows_per_wave(SM, NP);
    const int groups = spk::ceil_div(g.P, kWaves * R * 16);
    dim3 grid(spk::ceil_div(groups, iters), g.NT);
    hipLaunchKernelGGL((k_fire_fast<SM, NP, R>), grid, dim3(kThreads), lds, s, xp, bp, g, theta,
                       iters, vec_store, ot, ov);
}

typedef void (*FireLauncher)(const uint8_t *, const h8 *, const FGeom &, float, int, int, size_t,
                             uint8_t *, float *, hipStream_t);

#define SPK_FIRE_2(S) &launch_fire<S, 2>
#define SPK_FIRE_1(S) &launch_fire<S, 1>
const FireLauncher kFireF32[16] = {
    nullptr,        SPK_FIRE_2(1),  SPK_FIRE_2(2),  SPK_FIRE_2(3),  SPK_FIRE_2(4),  SPK_FIRE_2(5),
    SPK_FIRE_2(6),  SPK_FIRE_2(7),  SPK_FIRE_2(8),  SPK_FIRE_2(9),  SPK_FIRE_2(10), SPK_FIRE_2(11),
    SPK_FIRE_2(12), SPK_FIRE_2(13), SPK_FIRE_2(14), SPK_FIRE_2(15)};
const FireLauncher kFireF16[25] = {
    nullptr,        SPK_FIRE_1(1),  SPK_FIRE_1(2),  SPK_FIRE_1(3),  SPK_FIRE_1(4),  SPK_FIRE_1(5),
    SPK_FIRE_1(6),  SPK_FIRE_1(7),  SPK_FIRE_1(8),  SPK_FIRE_1(9),  SPK_FIRE_1(10), SPK_FIRE_1(11),
    SPK_FIRE_1(12), SPK_FIRE_1(13), SPK_FIRE_1(14), SPK_FIRE_1(15), SPK_FIRE_1(16), SPK_FIRE_1(17),
    SPK_FIRE_1(18), SPK_FIRE_1(19), SPK_FIRE_1(20), SPK_FIRE_1(21), SPK_FIRE_1(22), SPK_FIRE_1(23),
    SPK_FIRE_1(24)};
#undef SPK_FIRE_2
#undef SPK_FIRE_1

template <int SK, int NP>
void launch_fire32(const uint8_t *xp, const h8 *bp, const FGeom &g, float theta, int iters,
                   int vec_store, size_t lds, uint8_t *ot, float *ov, hipStream_t s)
{
    const int groups = spk::ceil_div(g.P, kWaves * 32);
    dim3 grid(spk::ceil_div(groups, iters), g.NT32);
    hipLaunchKernelGGL((k_fire32<SK, NP>), grid, dim3(kThreads), lds, s, xp, bp, g, theta, iters,
                       vec_store, ot, ov);
}

#define SPK_F32_2(S) &launch_fire32<S, 2>
#define SPK_F32_1(S) &launch_fire32<S, 1>
const FireLauncher kFire32F32[20] = {
    nullptr,        SPK_F32_2(1),  SPK_F32_2(2),  SPK_F32_2(3),  SPK_F32_2(4),  SPK_F32_2(5),
    SPK_F32_2(6),   SPK_F32_2(7),  SPK_F32_2(8),  SPK_F32_2(9),  SPK_F32_2(10), SPK_F32_2(11),
    SPK_F32_2(12),  SPK_F32_2(13), SPK_F32_2(14), SPK_F32_2(15), SPK_F32_2(16), SPK_F32_2(17),
    SPK_F32_2(18),  SPK_F32_2(19)};
const FireLauncher kFire32F16[32] = {
    nullptr,        SPK_F32_1(1),  SPK_F32_1(2),  SPK_F32_1(3),  SPK_F32_1(4),  SPK_F32_1(5),
    SPK_F32_1(6),   SPK_F32_1(7),  SPK_F32_1(8),  SPK_F32_1(9),  SPK_F32_1(10), SPK_F32_1(11),
    SPK_F32_1(12),  SPK_F32_1(13), SPK_F32_1(14), SPK_F32_1(15), SPK_F32_1(16), SPK_F32_1(17),
    SPK_F32_1(18),  SPK_F32_1(19), SPK_F32_1(20), SPK_F32_1(21), SPK_F32_1(22), SPK_F32_1(23),
    SPK_F32_1(24),  SPK_F32_1(25), SPK_F32_1(26), SPK_F32_1(27), SPK_F32_1(28), SPK_F32_1(29),
    SPK_F32_1(30),  SPK_F32_1(31)};
#undef SPK_F32_2
#undef SPK_F32_1

int ro_splits(const FGeom &g) { return (g.S16 + kRoSteps - 1) / kRoSteps; }

// Largest staged byte range of any (row group, split), remembered per geometry.
size_t ro_halo(const FGeom &g)
{
    typedef std::tuple<int, int, int, int, int, int, int, int, int> Key;
    static std::mutex mu;
    static std::map<Key, size_t> memo;
    const Key key{g.B, g.Ci, g.Hi, g.Wi, g.Kh, g.Kw, g.stride, g.pad, g.Ho};
    {
        std::lock_guard<std::mutex> lock(mu);
        auto it = memo.find(key);
        if (it != memo.end()) return it->second;
    }
    long long best = 0;
    const int splits = ro_splits(g);
    for (long long p0 = 0; p0 < g.P; p0 += 32) {
        const int p1 = (int)std::min<long long>(g.P, p0 + 32) - 1;
        for (int sp = 0; sp < splits; sp++) {
            long long h0, h1;
            ro_range(g, (int)p0, p1, sp, h0, h1);
            best = std::max(best, h1 - (h0 & ~15ll));
        }
    }
    const size_t v = halo_lds(best);
    std::lock_guard<std::mutex> lock(mu);
    if (memo.size() > 4096) memo.clear();
    memo[key] = v;
    return v;
}

constexpr size_t kRoLdsMax = 96 * 1024;

// The packing pass stages one padded input row or one map's weights in LDS.
bool pack_fits(const FGeom &g)
{
    return (long long)g.rowb <= 64 * 1024 && (long long)g.Cin * g.Kh * g.Kw * 4 <= 64 * 1024;
}

}  // namespace

namespace spk {

bool conv_fast_supported(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride,
                         int pad, int Ho, int Wo, bool half_w, bool readout, bool potentials)
{
    if (readout || potentials || T < 1 || T > 32 || B < 1 || Ci < 1 || Co < 1 || Ho < 1 || Wo < 1) return false;
    const long long Hp = Hi + 2ll * pad, Wp = Wi + 2ll * pad;
    if ((long long)B * Ho * Wo >= (1ll << 31) || (long long)B * Hp * Wp * Ci + kSlack >= (1ll << 31))
        return false;
    if ((long long)Kw * Ci > (1 << 16) || Kh > (1 << 12)) return false;
    const FGeom g = make_geom(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo);
    if (variant_of(g, half_w) == kNone || !pack_fits(g)) return false;
    if ((long long)g.rowb * g.Kh > kHaloMax) return false;  // cheap pre-check
    return group_lds(g, half_w) <= (size_t)kHaloMax;  // + at most 31 KB of staged bytes
}

size_t conv_fast_workspace(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride,
                           int pad, int Ho, int Wo)
{
    const FGeom g = make_geom(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo);
    return xp_bytes(g) + bp_bytes(g, 2);
}

bool readout_fast_supported(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw,
                            int stride, int pad, int Ho, int Wo)
{
    if (T < 1 || T > SPK_MAX_T || B < 1 || Ci < 1 || Co < 1 || Ho < 1 || Wo < 1) return false;
    const long long Hp = Hi + 2ll * pad, Wp = Wi + 2ll * pad, Cp = ro_channels(Ci);
    if ((long long)B * Ho * Wo >= (1ll << 31) || (long long)B * Hp * Wp * Cp + kSlack >= (1ll << 31))
        return false;
    if ((long long)Kw * Cp > (1 << 16) || Kh > (1 << 12)) return false;
    const FGeom g = make_ro_geom(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo);
    if (!pack_fits(g) || (long long)ro_splits(g) * Co * g.P >= (1ll << 31)) return false;
    if ((long long)g.rowb * (g.Kh + 2) * 2 > (long long)kRoLdsMax) return false;  // cheap pre-check
    return ro_halo(g) + kRoRed <= kRoLdsMax;
}

size_t readout_fast_workspace(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw,
                              int stride, int pad, int Ho, int Wo)
{
    const FGeom g = make_ro_geom(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo);
    return xp_bytes(g) + spk::align_up(bp_bytes(g, 2), 256) +
           (size_t)ro_splits(g) * Co * g.P * sizeof(float);
}

spk_status readout_fast(const uint8_t *in, int B, int T, int Ci, int Hi, int Wi, const void *w,
                        bool half_w, int Co, int Kh, int Kw, int stride, int pad, int Ho, int Wo,
                        uint8_t *out_t, float *out_v, void *ws, hipStream_t s, const void *packed_w,
                        const PoolIn *pool)
{
    const FGeom g = make_ro_geom(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo);
    uint8_t *xp = reinterpret_cast<uint8_t *>(ws);
    h8 *bp = packed_w ? const_cast<h8 *>(reinterpret_cast<const h8 *>(packed_w))
                      : reinterpret_cast<h8 *>(reinterpret_cast<char *>(ws) + xp_bytes(g));
    float *part = reinterpret_cast<float *>(reinterpret_cast<char *>(ws) + xp_bytes(g) +
                                            spk::align_up(bp_bytes(g, 2), 256));
    if (pool && planes_fit(g, *pool)) {
        // the pooled input in whole planes; the weights, when not given packed, in their own pass
        const size_t lds = align_up16(kPlaneC * pool->H0 * pool->W0) + (size_t)kPlaneC * g.Hi * g.Wi;
        hipLaunchKernelGGL(k_pack_planes, dim3(g.B * ((g.Ci + kPlaneC - 1) / kPlaneC)), dim3(256), lds, s,
                           g, *pool, xp);
        SPK_LAUNCHED("spk_conv_fire");
        if (!packed_w) launch_pack(in, w, half_w, true, g, xp, bp, s, false, true);
    } else {
        launch_pack(in, w, half_w, true, g, xp, bp, s, true, packed_w == nullptr, pool);
    }
    SPK_LAUNCHED("spk_conv_fire");

    const int splits = ro_splits(g);
    const int n_groups = spk::ceil_div(g.P, 32);
    // about 512 blocks: one round at two blocks per CU, B fragments reused
    // over several row groups
    int iters = (int)std::max<long long>(1, spk::ceil_div((long long)n_groups * g.NT32 * splits, 512));
    iters = std::min(iters, n_groups);
    const size_t halo = ro_halo(g);
    const bool pre = halo / 16 <= (size_t)kRoPre * kThreads;
    const size_t lds = halo + kRoRed;
    const int nx = spk::ceil_div(n_groups, iters);
    const dim3 grid(nx * g.NT32 * splits);
    auto run = [&](auto kern) {
        if (lds > 64 * 1024)
            (void)hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        hipLaunchKernelGGL(kern, grid, dim3(kThreads), lds, s, xp, bp, g, iters, n_groups, nx, part);
    };
    if (half_w) {
        if (pre) run(k_readout32<1, true>);
        else run(k_readout32<1, false>);
    } else {
        if (pre) run(k_readout32<2, true>);
        else run(k_readout32<2, false>);
    }
    SPK_LAUNCHED("spk_conv_fire");
    const long long n = (long long)g.Co * g.P;
    hipLaunchKernelGGL(k_readout_sum, dim3(spk::ceil_div(n, 256)), dim3(256), 0, s, part, g, splits,
                       out_t, out_v);
    return check_launch("spk_conv_fire");
}

size_t readout_packed_bytes(int Co, int Ci, int Kh, int Kw, bool half_w)
{
    const FGeom g = make_ro_geom(1, 1, Ci, Kh, Kw, Co, Kh, Kw, 1, 0, 1, 1);
    return (size_t)g.NT32 * g.S16 * (half_w ? 1 : 2) * 64 * sizeof(h8);
}

spk_status readout_pack_weights(const void *w, bool half_w, int Co, int Ci, int Kh, int Kw,
                                void *packed, hipStream_t s)
{
    const FGeom g = make_ro_geom(1, 1, Ci, Kh, Kw, Co, Kh, Kw, 1, 0, 1, 1);
    launch_pack(nullptr, w, half_w, true, g, nullptr, reinterpret_cast<h8 *>(packed), s, false, true);
    return check_launch("spk_conv_pack_weights");
}

spk_status conv_fire_fast(const uint8_t *in, int B, int T, int Ci, int Hi, int Wi, const void *w,
                          bool half_w, int Co, int Kh, int Kw, int stride, int pad, int Ho, int Wo,
                          float theta, uint8_t *out_t, float *out_v, void *ws, hipStream_t s)
{
    const FGeom g = make_geom(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo);
    uint8_t *xp = reinterpret_cast<uint8_t *>(ws);
    h8 *bp = reinterpret_cast<h8 *>(reinterpret_cast<char *>(ws) + xp_bytes(g));
    const Variant v = variant_of(g, half_w);
    launch_pack(in, w, half_w, v == kV32, g, xp, bp, s);
    SPK_LAUNCHED("spk_conv_fire");

    // Row groups per block: keep about 640 blocks in flight (two per CU with
    // some slack) so that each wave's register B fragments serve several groups.
    const int groups = spk::ceil_div(g.P, group_rows(g, half_w));
    const int col_tiles = v == kV32 ? g.NT32 : g.NT;
    int iters = (int)std::max<long long>(1, (long long)groups * col_tiles / 640);
    iters = std::min(iters, groups);
    size_t lds = group_lds(g, half_w);
    if (v == kV32) lds += (size_t)kWaves * g.S16 * 64 * sizeof(uint2);
    const int vec_store = (g.Ho * g.Wo) % 4 == 0 && ((uintptr_t)out_t & 3) == 0 &&
                          ((uintptr_t)out_v & 15) == 0;
    const FireLauncher launch = v == kV32 ? (half_w ? kFire32F16[g.S16] : kFire32F32[g.S16])
                                          : (half_w ? kFireF16[g.S] : kFireF32[g.S]);
    launch(xp, bp, g, theta, iters, vec_store, lds, out_t, out_v, s);
    return check_launch("spk_conv_fire");
}

}  // namespace spk
