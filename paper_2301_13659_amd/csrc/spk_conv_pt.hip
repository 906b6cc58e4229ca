// spk_conv_fire, firing layers with T <= 32: one matrix-core product per
// tile computes the potentials of every time step at once (Spyker §II-E.1
// Eq. 2; first-spike firing of §II-D.3 and §II-E).
//
// Under rank-order coding frame t is the cumulative S_t = [time <= t], so
// V_t = W * S_t for every step independently.  The implicit GEMM here puts
// (position, step) pairs on the MFMA rows: a 32x32x16 tile holds 32 / TP
// output positions x TP steps (TP = 8, 16 or 32 >= T; rows past T - 1 repeat
// step T - 1) against 32 maps, and its 16-tap depth slices walk the kernel
// window.  The A fragment of row (p, t) is [time <= t] over 8 taps, one
// packed-half subtraction with clamping per pair of taps.  The first crossing
// of theta and the potential that goes with it are read off the finished
// tile, with no state carried across steps.
//
// Operands (in the caller's workspace, written by k_pack_pt):
//  - Xp: the time map as padded channels-last bytes, Xp[b][iy][ix][c] over
//    (Hi + 2 pad) x (Wi + 2 pad) x Cp, each time clamped to T (T and above
//    never fire within the window; padding and the channels past Ci hold T).
//    Cp is Ci rounded up to 8 when that adds no depth, so window runs start
//    aligned;
//  - the depth is ordered (ky, j), j = kx*Cp + c, each kernel row's run of
//    Kw*Cp taps padded to a multiple of 16, so a 16-tap slice never straddles
//    two kernel rows and its offset from the window origin is
//    ky*rowbytes + 16*jq for every position;
//  - the weights as ready B fragments in that order: hi/lo halves of the
//    float master (two products per slice) or the half weights; zero on
//    padding taps.
//
// Work split: a block (4 waves) keeps the B fragments of one 32-map column
// tile in registers and walks one contiguous range of positions in groups of
// 64.  Ranges divide the positions evenly over about two blocks per CU, so
// every SIMD gets the same work; the blocks of one range sit on one XCD and
// share its L2 for the input bytes.  A group's input rows are loaded into
// registers one group ahead and stored to LDS as the halves 1024 + t that the
// A fragments subtract from (with a flag per 16 bytes that says whether any
// of them fires).  Results go through LDS so that each map's run of positions
// is written with coalesced stores.  In a sparse group, the 16-tap slices in
// which no input of the tile fires are skipped.
#include <hip/hip_fp16.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <tuple>

#include "spk_internal.h"

namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kG = 64;                         // positions per group
constexpr int kStageStride = kG + 1;           // staged results: [map][position], padded
constexpr int kRange = 16 * 1024;              // Xp bytes of a group's input rows (at most)
constexpr int kSlackPT = 64;                   // readable bytes past the end of Xp
constexpr uint32_t kSelLo = 0x04010400u;       // bytes 0,1 -> halves 1024 + b
constexpr uint32_t kSelHi = 0x04030402u;       // bytes 2,3 -> halves 1024 + b

// LDS: [staged V x 2 | staged t x 2 | position table x 3 | word counts per
// wave | fire flag per 16 input bytes | input as halves (2 bytes per input
// byte, sized per launch to the largest group's range, so small images leave
// room for more blocks)]
constexpr size_t kStvOff = 0;
constexpr size_t kSttOff = kStvOff + 2 * 32 * kStageStride * sizeof(float);
constexpr size_t kTabOff = (kSttOff + 2 * 32 * kStageStride + 15) / 16 * 16;
constexpr size_t kTabBytes = 3 * kG * 3 * sizeof(int);
constexpr size_t kCntOff = kTabOff + kTabBytes;
constexpr size_t kFlagOff = kCntOff + 2 * (kThreads / 64) * sizeof(int);
constexpr size_t kHalOff = (kFlagOff + kRange / 16 + 15) / 16 * 16;

// Layers with few maps take their output positions in blocks of by x bx
// (1 x 1 otherwise): a tile's 32 columns are then (position of the block,
// map) pairs, so four maps fill a tile with 2 x 4 positions instead of
// leaving 28 of its 32 columns empty.  A block is one position of a virtual
// layer with by*bx*Co maps, a window of Khv x Kwv input pixels (the union of
// its positions' windows) and strides by*stride, bx*stride; the weight of
// virtual map (jy, jx, o) at virtual tap (c, kyv, kxv) is W[o, c, kyv -
// jy*stride, kxv - jx*stride] inside the real window and 0 outside it.
struct PGeom {
    int B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo;
    int by, bx;    // output positions per block
    int Hv, Wv;    // blocks: ceil(Ho / by) x ceil(Wo / bx)
    int Khv, Kwv;  // input window of a block
    int Cv;        // virtual maps: by * bx * Co
    int Cp;    // channels per padded pixel of Xp
    int Hp, Wp;
    int rowb;  // Wp * Cp: bytes of one padded input row
    int slack; // readable bytes past the last padded row
    int run;   // Kwv * Cp: taps of one kernel row
    int Q16;   // ceil(run / 16): 16-tap slices per kernel row
    int SK;    // Khv * Q16: slices of the layer
    int SKp;   // slices of the kernel instance (>= SK; the extra ones are zero)
    int P;     // B * Hv * Wv blocks (positions when the blocks are 1 x 1)
    int NT;    // ceil(Cv / 32)
    int hw;    // input words (16 bytes) the LDS halves of a launch hold
    int TP;    // steps per position in a tile: 8, 16 or 32
    int lgTP;
};

int choose_cp(int Ci, int Kw)
{
    const int c8 = (Ci + 7) / 8 * 8;
    return (Kw * c8 + 15) / 16 == (Kw * Ci + 15) / 16 ? c8 : Ci;
}

PGeom make_pgeom_blocked(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride,
                         int pad, int Ho, int Wo, int by, int bx)
{
    PGeom g{};
    g.B = B; g.T = T; g.Ci = Ci; g.Hi = Hi; g.Wi = Wi; g.Co = Co; g.Kh = Kh; g.Kw = Kw;
    g.stride = stride; g.pad = pad; g.Ho = Ho; g.Wo = Wo;
    g.by = by; g.bx = bx;
    g.Hv = (Ho + by - 1) / by;
    g.Wv = (Wo + bx - 1) / bx;
    g.Khv = (by - 1) * stride + Kh;
    g.Kwv = (bx - 1) * stride + Kw;
    g.Cv = by * bx * Co;
    g.Cp = choose_cp(Ci, g.Kwv);
    g.Hp = Hi + 2 * pad;
    g.Wp = Wi + 2 * pad;
    g.rowb = g.Wp * g.Cp;
    // a block past the last row or column reads up to by*stride rows and a
    // row's width beyond the padded input (only for its positions that are
    // past the output, whose weights there are zero)
    g.slack = kSlackPT + (by > 1 || bx > 1 ? (by * stride + 1) * g.rowb : 0);
    g.run = g.Kwv * g.Cp;
    g.Q16 = (g.run + 15) / 16;
    g.SK = g.Khv * g.Q16;
    g.SKp = g.SK;
    g.P = B * g.Hv * g.Wv;
    g.NT = (g.Cv + 31) / 32;
    g.TP = T <= 8 ? 8 : (T <= 16 ? 16 : 32);
    g.lgTP = T <= 8 ? 3 : (T <= 16 ? 4 : 5);
    return g;
}

// Geometry of a layer: 1 x 1 blocks, or for layers of at most 16 maps the
// block shape with the least work (slices x blocks x column tiles) among
// those that fill at most 32 columns and whose slices still fit the
// in-register kernels (18 with float weights, 36 with half weights), when it
// saves at least a fifth of the work.
PGeom make_pgeom(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride, int pad,
                 int Ho, int Wo, bool half_w)
{
    const PGeom one = make_pgeom_blocked(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo, 1, 1);
    if (Co > 16) return one;
    static const int kShapes[][2] = {{1, 2}, {2, 1}, {2, 2}, {1, 4}, {4, 1}, {2, 4},
                                     {4, 2}, {4, 4}, {2, 8}, {8, 2}, {4, 8}, {8, 4}};
    const int limit = half_w ? 36 : 18;
    const long long base = (long long)one.SK * one.NT * one.P;
    PGeom best = one;
    long long best_work = base;
    for (const auto &sh : kShapes) {
        if (sh[0] * sh[1] * Co > 32 || sh[0] > Ho || sh[1] > Wo) continue;
        const PGeom g = make_pgeom_blocked(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo, sh[0], sh[1]);
        if (g.SK > limit) continue;
        const long long work = (long long)g.SK * g.NT * g.P;
        if (work < best_work) {
            best = g;
            best_work = work;
        }
    }
    return best_work * 5 <= base * 4 ? best : one;
}

// Alignment of every window run in the staged halves: 16, 8, 4 or 2 bytes.
int read_mode(int Cp) { return Cp % 8 == 0 ? 3 : (Cp % 4 == 0 ? 2 : (Cp % 2 == 0 ? 1 : 0)); }

size_t xp_bytes(const PGeom &g) { return spk::align_up((size_t)g.B * g.Hp * g.rowb + g.slack, 256); }
size_t bp_bytes(const PGeom &g, int np) { return (size_t)g.NT * g.SKp * np * 64 * sizeof(h8); }

__device__ __forceinline__ h2 as_h2(uint32_t u) { return __builtin_bit_cast(h2, u); }
__device__ __forceinline__ uint32_t as_u(h2 h) { return __builtin_bit_cast(uint32_t, h); }

// [t <= last] for two staged halves 1024 + t (c = 1025 + last in both):
// c - (1024 + t) is a small exact integer, >= 1 iff t <= last; clamp to [0, 1].
__device__ __forceinline__ uint32_t upto2(uint32_t x, h2 c)
{
    const h2 one = {(_Float16)1.0f, (_Float16)1.0f}, zero = {(_Float16)0.0f, (_Float16)0.0f};
    h2 a = c - as_h2(x);
    return as_u(__builtin_elementwise_min(__builtin_elementwise_max(a, zero), one));
}

__device__ __forceinline__ h8 frag_upto(u4 x, h2 c)
{
    u4 v = {upto2(x[0], c), upto2(x[1], c), upto2(x[2], c), upto2(x[3], c)};
    return __builtin_bit_cast(h8, v);
}

// 8 staged halves (16 bytes) at byte offset at from base (16-aligned); kMode
// gives the alignment every window run has: 3 = 16, 2 = 8, 1 = 4, 0 = 2 bytes.
template <int kMode>
__device__ __forceinline__ u4 lds_read16(const uint8_t *base, int at)
{
    if (kMode == 3) return *reinterpret_cast<const u4 *>(base + at);
    if (kMode == 2) {
        const uint2 a = *reinterpret_cast<const uint2 *>(base + at);
        const uint2 b = *reinterpret_cast<const uint2 *>(base + at + 8);
        return u4{a.x, a.y, b.x, b.y};
    }
    if (kMode == 1) {
        const uint32_t *w = reinterpret_cast<const uint32_t *>(base + at);
        return u4{w[0], w[1], w[2], w[3]};
    }
    const uint32_t *w = reinterpret_cast<const uint32_t *>(base + (at & ~3));
    const uint32_t w0 = w[0], w1 = w[1], w2 = w[2], w3 = w[3], w4 = w[4];
    const uint32_t sh = (uint32_t)(at & 3);
    return u4{__builtin_amdgcn_alignbyte(w1, w0, sh), __builtin_amdgcn_alignbyte(w2, w1, sh),
              __builtin_amdgcn_alignbyte(w3, w2, sh), __builtin_amdgcn_alignbyte(w4, w3, sh)};
}

// Padded input rows [r0, r1) hold the windows of output positions [p0, p1].
__host__ __device__ inline void group_rows(const PGeom &g, int p0, int p1, int &r0, int &r1)
{
    const int HvWv = g.Hv * g.Wv;
    const int b0 = p0 / HvWv, y0 = (p0 - b0 * HvWv) / g.Wv;
    const int b1 = p1 / HvWv, y1 = (p1 - b1 * HvWv) / g.Wv;
    r0 = b0 * g.Hp + y0 * g.by * g.stride;
    r1 = b1 * g.Hp + y1 * g.by * g.stride + g.Khv;
}

// ------------------------------------------------------------------ packing

// Blocks [0, nb_in): one padded input row (b, py) each, transposed through
// LDS from channel rows to channels-last, times clamped to T (a pooled input
// row is pooled there from the staged window rows); the last of them fills
// the readable slack.  A pooled input whose rows are too wide to stage runs a
// grid-stride pass over the Xp bytes instead, each pooling its window from
// the unpooled map.  Blocks [nb_in, nb_in + 32*NT): one map o each
// (maps past Co are zero), written as B fragments: lane l holds map o (l % 32)
// and taps 8*(l/32)..+7 of a slice.
template <int NP, bool kHalfW>
__global__ __launch_bounds__(256) void k_pack_pt(const uint8_t *__restrict__ in,
                                                 const void *__restrict__ wv, PGeom g, int nb_in,
                                                 uint8_t *__restrict__ xp, h8 *__restrict__ bp,
                                                 spk::PoolIn pool)
{
    extern __shared__ __align__(16) uint8_t sm[];
    const uint8_t never = (uint8_t)g.T;
    if ((int)blockIdx.x < nb_in && pool.src && pool.stage < 0) {
        // pooled input too wide to stage: each thread writes Xp bytes
        // (b, py, px, c), the pooling window read from the unpooled map; the
        // Xp body is below 2^30 bytes
        const uint32_t body = (uint32_t)g.B * g.Hp * g.rowb, total = body + (uint32_t)g.slack;
        for (uint32_t e = blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (uint32_t)nb_in * blockDim.x) {
            uint32_t v = never;
            if (e < body) {
                const uint32_t rowi = e / (uint32_t)g.rowb, within = e - rowi * (uint32_t)g.rowb;
                const int b = (int)(rowi / (uint32_t)g.Hp), py = (int)(rowi - (uint32_t)b * g.Hp);
                const int px = (int)(within / (uint32_t)g.Cp), c = (int)within - px * g.Cp;
                const int iy = py - g.pad, ix = px - g.pad;
                if ((unsigned)iy < (unsigned)g.Hi && (unsigned)ix < (unsigned)g.Wi && c < g.Ci) {
                    const long long plane = (long long)b * g.Ci + c;
                    const uint32_t t = spk::pool_cell(pool, plane, iy, ix);
                    if (pool.pooled) pool.pooled[(plane * g.Hi + iy) * g.Wi + ix] = (uint8_t)t;
                    v = min(t, (uint32_t)never);
                }
            }
            xp[e] = (uint8_t)v;
        }
        return;
    }
    if ((int)blockIdx.x < nb_in) {
        const int b = blockIdx.x / g.Hp, py = blockIdx.x - b * g.Hp;
        const int iy = py - g.pad;
        uint8_t *row = xp + ((size_t)b * g.Hp + py) * g.rowb;
        // rows of a multiple of 16 bytes start 16-byte aligned: 16-byte fills and stores
        const bool wide = (g.rowb & 15) == 0;
        const uint4 never16 = make_uint4(0x01010101u * never, 0x01010101u * never, 0x01010101u * never,
                                         0x01010101u * never);
        if ((unsigned)iy < (unsigned)g.Hi) {
            if (wide) {
                for (int e = threadIdx.x; e < g.rowb / 16; e += blockDim.x) reinterpret_cast<uint4 *>(sm)[e] = never16;
            } else {
                for (int e = threadIdx.x; e < g.rowb; e += blockDim.x) sm[e] = never;
            }
            __syncthreads();
            auto put = [&](int c, int x, uint8_t v) { sm[(x + g.pad) * g.Cp + c] = v < never ? v : never; };
            if (pool.src) {
                // the input row is pooled here (and kept when asked for)
                spk::pool_row(pool, (long long)b * g.Ci, g.Ci, g.Hi, g.Wi, iy,
                              reinterpret_cast<uint32_t *>(sm + pool.stage), put);
            } else {
                const uint8_t *src = in + (size_t)b * g.Ci * g.Hi * g.Wi + (size_t)iy * g.Wi;
                const size_t plane = (size_t)g.Hi * g.Wi;
                if ((g.Wi & 3) == 0 && (plane & 3) == 0 && (((uintptr_t)src) & 3) == 0 && (g.Ci & 3) == 0 &&
                    (g.Cp & 3) == 0) {
                    // 4 channels x 4 pixels per thread: four dword loads (one per channel),
                    // times clamped to T byte-wise, a byte transpose to four dwords of 4
                    // channels each, written to LDS as dwords
                    const int wq = g.Wi >> 2, cq = g.Ci >> 2, n16 = cq * wq;
                    const uint32_t t4 = 0x01010101u * never;
                    for (int e = threadIdx.x; e < n16; e += blockDim.x) {
                        const int x4 = e % wq, c4 = e / wq;
                        uint32_t d[4];
#pragma unroll
                        for (int k = 0; k < 4; k++)
                            d[k] = *reinterpret_cast<const uint32_t *>(src + (4 * c4 + k) * plane + 4 * x4);
#pragma unroll
                        for (int k = 0; k < 4; k++) {
                            // bytes above T (T <= 32) become T: a byte is above T when its
                            // top bit is set or its low 7 bits plus 127 - T carry into it
                            const uint32_t gt =
                                (((d[k] & 0x7f7f7f7fu) + 0x01010101u * (uint32_t)(127 - (int)never)) | d[k]) &
                                0x80808080u;
                            const uint32_t full = (gt >> 7) * 0xFFu;
                            d[k] = (d[k] & ~full) | (t4 & full);
                        }
                        const uint32_t t0 = __builtin_amdgcn_perm(d[1], d[0], 0x05010400u);
                        const uint32_t t1 = __builtin_amdgcn_perm(d[3], d[2], 0x05010400u);
                        const uint32_t t2 = __builtin_amdgcn_perm(d[1], d[0], 0x07030602u);
                        const uint32_t t3 = __builtin_amdgcn_perm(d[3], d[2], 0x07030602u);
                        const uint32_t o[4] = {__builtin_amdgcn_perm(t1, t0, 0x05040100u),
                                               __builtin_amdgcn_perm(t1, t0, 0x07060302u),
                                               __builtin_amdgcn_perm(t3, t2, 0x05040100u),
                                               __builtin_amdgcn_perm(t3, t2, 0x07060302u)};
#pragma unroll
                        for (int q = 0; q < 4; q++)
                            *reinterpret_cast<uint32_t *>(sm + (4 * x4 + q + g.pad) * g.Cp + 4 * c4) = o[q];
                    }
                } else if ((g.Wi & 3) == 0 && (plane & 3) == 0 && (((uintptr_t)src) & 3) == 0) {
                    // the row of every channel as dwords, all of a thread's loads in flight first
                    const int wq = g.Wi >> 2, n4 = g.Ci * wq;
                    for (int e0 = threadIdx.x; e0 < n4; e0 += 8 * (int)blockDim.x) {
                        uint32_t v[8];
#pragma unroll
                        for (int u = 0; u < 8; u++) {
                            const int e = min(e0 + u * (int)blockDim.x, n4 - 1);
                            const int c = e / wq, x4 = e - c * wq;
                            v[u] = *reinterpret_cast<const uint32_t *>(src + c * plane + 4 * x4);
                        }
#pragma unroll
                        for (int u = 0; u < 8; u++) {
                            const int e = e0 + u * (int)blockDim.x;
                            if (e >= n4) break;
                            const int c = e / wq, x4 = e - c * wq;
#pragma unroll
                            for (int q = 0; q < 4; q++) put(c, 4 * x4 + q, (uint8_t)(v[u] >> (8 * q)));
                        }
                    }
                } else {
                    const int n = g.Ci * g.Wi;
                    for (int e = threadIdx.x; e < n; e += blockDim.x) {
                        const int c = e / g.Wi, x = e - c * g.Wi;
                        put(c, x, src[(size_t)c * plane + x]);
                    }
                }
            }
            __syncthreads();
            if (wide) {
                for (int e = threadIdx.x; e < g.rowb / 16; e += blockDim.x)
                    reinterpret_cast<uint4 *>(row)[e] = reinterpret_cast<const uint4 *>(sm)[e];
            } else {
                for (int e = threadIdx.x; e < g.rowb; e += blockDim.x) row[e] = sm[e];
            }
        } else if (wide) {
            for (int e = threadIdx.x; e < g.rowb / 16; e += blockDim.x) reinterpret_cast<uint4 *>(row)[e] = never16;
        } else {
            for (int e = threadIdx.x; e < g.rowb; e += blockDim.x) row[e] = never;
        }
        if ((int)blockIdx.x == nb_in - 1)
            for (int e = threadIdx.x; e < g.slack; e += blockDim.x) row[g.rowb + e] = never;
        return;
    }
    // virtual map ov = (jy*bx + jx)*Co + o: real map o of block position (jy, jx)
    const int ov = blockIdx.x - nb_in;
    const int jb = ov / g.Co, o = ov - jb * g.Co;
    const int jy = jb / g.bx, jx = jb - jy * g.bx;
    const int taps = g.Ci * g.Kh * g.Kw;
    float *wl = reinterpret_cast<float *>(sm);
    const bool real = ov < g.Cv;
    for (int e = threadIdx.x; e < taps; e += blockDim.x) {
        float w = 0.0f;
        if (real) {
            const size_t at = (size_t)o * taps + e;
            w = kHalfW ? (float)reinterpret_cast<const _Float16 *>(wv)[at]
                       : reinterpret_cast<const float *>(wv)[at];
        }
        wl[e] = w;
    }
    __syncthreads();
    const int nt = ov / 32, col = ov & 31;
    for (int f = threadIdx.x; f < g.SKp * 2; f += blockDim.x) {
        const int s = f >> 1, half = f & 1;
        const int kyv = s / g.Q16, jq = s - kyv * g.Q16;
        const int ky = kyv - jy * g.stride;
        h8 hi, lo;
        // addresses first (padding taps read word 0), then the reads together:
        // no branch around a read
        int at[8];
        bool live[8];
#pragma unroll
        for (int e = 0; e < 8; e++) {
            const int j = jq * 16 + half * 8 + e;
            const int kxv = j / g.Cp, c = j - kxv * g.Cp;
            const int kx = kxv - jx * g.stride;
            live[e] = s < g.SK && j < g.run && c < g.Ci && (unsigned)ky < (unsigned)g.Kh &&
                      (unsigned)kx < (unsigned)g.Kw;
            at[e] = live[e] ? (c * g.Kh + ky) * g.Kw + kx : 0;
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
        const size_t ts = (size_t)nt * g.SKp + s;
        const int lane = col + 32 * half;
        bp[(ts * NP) * 64 + lane] = hi;
        if (NP == 2) bp[(ts * NP + 1) * 64 + lane] = lo;
    }
}

// -------------------------------------------------------------------- firing

struct Tab {
    int xoff;   // Xp offset of the block's window origin
    int obase;  // output offset of its first position for map 0: b*Co*Ho*Wo + y0*Wo + x0
    int yx;     // y0 << 16 | x0, its first position
};

// Per-group position table (threads 0..kG-1; slots past the group repeat its last).
__device__ __forceinline__ void fill_table(const PGeom &g, int gs, int cnt, Tab *tab)
{
    const int i = threadIdx.x;
    if (i < kG) {
        const int p = gs + min(i, cnt - 1);
        const int HvWv = g.Hv * g.Wv;
        const int b = p / HvWv, rem = p - b * HvWv;
        const int yb = rem / g.Wv, xb = rem - yb * g.Wv;
        const int y0 = yb * g.by, x0 = xb * g.bx;
        Tab t;
        t.xoff = (b * g.Hp + y0 * g.stride) * g.rowb + x0 * g.stride * g.Cp;
        t.obase = b * g.Co * g.Ho * g.Wo + y0 * g.Wo + x0;
        t.yx = (y0 << 16) | x0;
        tab[i] = t;
    }
}

// The Xp bytes [a0, a1 + 32) (a0 16-aligned) as 16-byte words, PF per
// thread of a block of NTH (word threadIdx.x + NTH*i); words past the end of
// Xp read its last.
template <int NTH = kThreads>
struct Staged {
    static constexpr int PF = (kRange / 16 + NTH - 1) / NTH;
    uint4 w[PF];
};

__device__ __forceinline__ int range_words(int a0, int a1) { return (a1 - a0 + 32 + 15) / 16; }

template <int NTH = kThreads>
__device__ __forceinline__ Staged<NTH> load_range(const uint8_t *xp, size_t xp_words, int a0, int a1)
{
    Staged<NTH> st;
    const size_t w0 = (size_t)a0 / 16;
    const int nw = range_words(a0, a1);
#pragma unroll
    for (int i = 0; i < Staged<NTH>::PF; i++) {
        const int k = (int)threadIdx.x + NTH * i;
        if (NTH * i < nw) {  // words past the range are neither loaded nor stored
            size_t w = w0 + (size_t)min(k, nw - 1);
            w = w < xp_words ? w : xp_words - 1;
            st.w[i] = reinterpret_cast<const uint4 *>(xp)[w];
        }
    }
    return st;
}

// Staged words to LDS as halves 1024 + t, plus a flag per word: does any of
// its 16 times fire within the window (clamped times: any byte below T)?
// Each wave also records in cnt how many of its words are flagged, for
// group_sparse.
template <int NTH>
__device__ __forceinline__ void store_range(const Staged<NTH> &st, uint8_t *hal, uint8_t *flags, int *cnt,
                                            uint32_t never4, int nw, int hw)
{
    int flagged = 0, words = 0;
#pragma unroll
    for (int i = 0; i < Staged<NTH>::PF; i++) {
        const int k = (int)threadIdx.x + NTH * i;
        if (NTH * i >= nw) break;
        const uint4 v = st.w[i];
        const u4 lo = {__builtin_amdgcn_perm(0x64646464u, v.x, kSelLo), __builtin_amdgcn_perm(0x64646464u, v.x, kSelHi),
                       __builtin_amdgcn_perm(0x64646464u, v.y, kSelLo), __builtin_amdgcn_perm(0x64646464u, v.y, kSelHi)};
        const u4 hi = {__builtin_amdgcn_perm(0x64646464u, v.z, kSelLo), __builtin_amdgcn_perm(0x64646464u, v.z, kSelHi),
                       __builtin_amdgcn_perm(0x64646464u, v.w, kSelLo), __builtin_amdgcn_perm(0x64646464u, v.w, kSelHi)};
        if (k < hw) {
            reinterpret_cast<u4 *>(hal)[2 * k] = lo;
            reinterpret_cast<u4 *>(hal)[2 * k + 1] = hi;
        }
        const bool f = ((v.x ^ never4) | (v.y ^ never4) | (v.z ^ never4) | (v.w ^ never4)) != 0u;
        if (k < kRange / 16) flags[k] = f ? 1 : 0;  // (larger blocks have threads past the flag bytes)
        flagged += __builtin_popcountll(__builtin_amdgcn_ballot_w64(f && k < nw));
        words += __builtin_popcountll(__builtin_amdgcn_ballot_w64(k < nw));
    }
    if ((threadIdx.x & 63) == 0) {
        cnt[2 * (threadIdx.x >> 6)] = flagged;
        cnt[2 * (threadIdx.x >> 6) + 1] = words;
    }
}

// Whether the staged group is sparse enough to test slices in, the same for
// every wave of the block (from the counts store_range left; call after the
// barrier that follows it).  A tile's slice can be skipped only when none of
// the tile's words under it fires, so with a fraction u of the words
// unflagged about u^pt of the slices are skipped, pt being the words a slice
// of the tile covers (one per position when window runs are 16-byte aligned,
// two otherwise); testing pays when that is above min_skip (below it the
// tests cost more than the skipped products save: 40 % for k_fire_pt, 15 %
// for k_fire_lb, where a skipped slice saves two products).  One decision for
// the block keeps its waves equally loaded between barriers.
template <int NW = kThreads / 64>
__device__ __forceinline__ bool group_sparse(const int *cnt, int pt, float min_skip)
{
    int flagged = 0, words = 0;
#pragma unroll
    for (int w = 0; w < NW; w++) {
        flagged += cnt[2 * w];
        words += cnt[2 * w + 1];
    }
    const float u = words > 0 ? (float)(words - flagged) / (float)words : 0.0f;
    float skip = u;
    for (int i = 1; i < pt; i++) skip *= u;
    return skip > min_skip;
}

// Staged results of positions [gs, min(gs + 64, p_end)) to the outputs,
// consecutive threads on consecutive positions of one map.  Unblocked
// layouts: a thread takes four consecutive positions of two maps, each
// written with one 16-byte and one 4-byte store where the four are
// contiguous in the output.  Blocked layouts: a thread takes one position of
// eight maps, all its staged values read before the stores.
__device__ __forceinline__ void write_out(const PGeom &g, int nt, int gs, int p_end, const Tab *tab,
                                          const float *stv, const uint8_t *stt,
                                          uint8_t *__restrict__ out_t, float *__restrict__ out_v)
{
    constexpr int kPer = 32 * kG / kThreads;  // maps per thread
    constexpr int kMapStep = kThreads / kG;
    const int HoWo = g.Ho * g.Wo;
    const int cnt = min(p_end, gs + kG) - gs;
    const bool blocked = g.by * g.bx > 1;
    // (output bases aligned for the word stores: 16 bytes for V, 4 for t)
    const bool aligned = ((reinterpret_cast<uintptr_t>(out_v) & 15) | (reinterpret_cast<uintptr_t>(out_t) & 3)) == 0;
    if (!blocked && (HoWo & 3) == 0) {
        // four consecutive positions of a map per thread, stored as one
        // 16-byte V word and one 4-byte time word when they are contiguous
        // and aligned in the output
        constexpr int kQ = kG / 4, kMaps = kThreads / kQ;
        const int p4 = 4 * (threadIdx.x % kQ), oc0 = threadIdx.x / kQ;
        if (p4 >= cnt) return;
        const Tab t0 = tab[p4];
        const int n3 = tab[min(p4 + 3, kG - 1)].obase;
        const bool vec = p4 + 3 < cnt && n3 == t0.obase + 3 && (t0.obase & 3) == 0 && aligned;
#pragma unroll
        for (int j = 0; j < 32 / kMaps; j++) {
            const int oc = oc0 + kMaps * j, ov = nt * 32 + oc;
            if (ov >= g.Cv) continue;
            const float *sv = stv + oc * kStageStride + p4;
            const uint8_t *st = stt + oc * kStageStride + p4;
            if (vec) {
                const float4 v4 = make_float4(sv[0], sv[1], sv[2], sv[3]);
                const uint32_t tw = (uint32_t)st[0] | ((uint32_t)st[1] << 8) | ((uint32_t)st[2] << 16) |
                                    ((uint32_t)st[3] << 24);
                const int n = t0.obase + ov * HoWo;
                *reinterpret_cast<float4 *>(out_v + n) = v4;
                *reinterpret_cast<uint32_t *>(out_t + n) = tw;
            } else {
                for (int i = 0; i < 4 && p4 + i < cnt; i++) {
                    const int n = tab[p4 + i].obase + ov * HoWo;
                    out_v[n] = sv[i];
                    out_t[n] = st[i];
                }
            }
        }
        return;
    }
    const int pi = threadIdx.x & (kG - 1), oc0 = threadIdx.x / kG;
    if (pi >= cnt) return;
    const Tab tb = tab[pi];
    float v[kPer];
    uint8_t t[kPer];
#pragma unroll
    for (int j = 0; j < kPer; j++) {
        const int oc = oc0 + kMapStep * j;
        v[j] = stv[oc * kStageStride + pi];
        t[j] = stt[oc * kStageStride + pi];
    }
#pragma unroll
    for (int j = 0; j < kPer; j++) {
        const int ov = nt * 32 + oc0 + kMapStep * j;
        if (ov >= g.Cv) continue;
        int n;
        if (blocked) {  // virtual map (jy*bx + jx)*Co + o
            const int jb = ov / g.Co, o = ov - jb * g.Co;
            const int jy = jb / g.bx, jx = jb - jy * g.bx;
            if ((tb.yx >> 16) + jy >= g.Ho || (tb.yx & 0xffff) + jx >= g.Wo) continue;
            n = tb.obase + o * HoWo + jy * g.Wo + jx;
        } else {
            n = tb.obase + ov * HoWo;
        }
        out_v[n] = v[j];
        out_t[n] = t[j];
    }
}

// Rows of a tile: output element e of a lane in wave half hh is row
// 8*(e/4) + 4*hh + e%4.  The A fragment of row r is given the position slot
// and step below.  TP = 16 and 8: each lane's elements are whole runs of
// steps in order (TP = 16, slot hh, element e = step e; TP = 8, slot hh for
// e < 8 and 2 + hh for e >= 8, step e % 8), so no lane needs the other half's
// results.  TP = 32: step r, the two halves' elements interleaved.
__device__ __forceinline__ void row_slot_step(int r, int lgTP, int &pl, int &tt)
{
    const int hi = r >> 3, half = (r >> 2) & 1, lo = r & 3;
    if (lgTP == 3) {
        pl = 2 * (hi >> 1) + half;
        tt = ((hi & 1) << 2) | lo;
    } else if (lgTP == 4) {
        pl = half;
        tt = (hi << 2) | lo;
    } else {
        pl = 0;
        tt = r;
    }
}

// Merge the two wave halves of one position slot (ft: step or NEVER; last:
// the potential at step T-1, meaningful in the upper half only).  Each swap
// leaves both halves' values in every lane; min and sum do not depend on
// their order.
__device__ __forceinline__ void merge_halves(uint32_t ft, float fv, float last, int hh, uint32_t &tf,
                                             float &vk)
{
    const auto t2 = __builtin_amdgcn_permlane32_swap(ft, ft, false, false);
    const uint32_t fb = __builtin_bit_cast(uint32_t, fv);
    const auto v2 = __builtin_amdgcn_permlane32_swap(fb, fb, false, false);
    const uint32_t lb = __builtin_bit_cast(uint32_t, hh ? last : 0.0f);
    const auto l2 = __builtin_amdgcn_permlane32_swap(lb, lb, false, false);
    const uint32_t t0 = t2[0], t1 = t2[1];
    const float f0 = __builtin_bit_cast(float, (uint32_t)v2[0]);
    const float f1 = __builtin_bit_cast(float, (uint32_t)v2[1]);
    const float vl = __builtin_bit_cast(float, (uint32_t)l2[0]) + __builtin_bit_cast(float, (uint32_t)l2[1]);
    tf = min(t0, t1);
    const float fsel = t0 < t1 ? f0 : f1;
    vk = tf < (uint32_t)spk::kNever ? fsel : vl;
}

// First element in [e0, e0 + n) above theta (as an offset) and its value;
// n when there is none.
__device__ __forceinline__ void first_above(const f16v &acc, int e0, int n, float theta, int &fe, float &fv)
{
    fe = n;
    fv = 0.0f;
#pragma unroll
    for (int e = 15; e >= 0; e--) {
        if (e < e0 || e >= e0 + n) continue;
        const bool c = acc[e] > theta;
        fe = c ? e - e0 : fe;
        fv = c ? acc[e] : fv;
    }
}

// Epilogue of a tile with TP steps per position (rows past T - 1 repeat step
// T - 1, so the last element of a run is the potential at T - 1): the spike
// time (or NEVER) and key potential of each position slot this lane holds,
// for its map lane % 32.  TP = 8: slots hh and 2 + hh (st/sv[0], [1]); TP =
// 16: slot hh; TP = 32: the one slot, the two wave halves merged, in every
// lane.
template <int TP>
__device__ __forceinline__ void tile_epilogue(const f16v &acc, float theta, int hh, uint32_t *st, float *sv)
{
    if constexpr (TP == 8 || TP == 16) {
#pragma unroll
        for (int k = 0; k < 16 / TP; k++) {
            int fe;
            float fv;
            first_above(acc, k * TP, TP, theta, fe, fv);
            st[k] = fe < TP ? (uint32_t)fe : (uint32_t)spk::kNever;
            sv[k] = fe < TP ? fv : acc[k * TP + TP - 1];
        }
    } else {
        // the first element above theta and its step (row 8*(e/4) + 4*hh +
        // e%4), then the minimum over the two halves through lane swaps
        int fe;
        float fv;
        first_above(acc, 0, 16, theta, fe, fv);
        const uint32_t ft = fe < 16 ? (uint32_t)(((fe >> 2) << 3) + 4 * hh + (fe & 3)) : (uint32_t)spk::kNever;
        const float last = acc[15];  // row 31: step T - 1, in the upper half
        merge_halves(ft, fv, last, hh, st[0], sv[0]);
    }
}

// Position slots of the tile a lane stores (see tile_epilogue): count and
// slot of entry k.
__device__ __forceinline__ int slots_held(int lgTP, int hh)
{
    return lgTP == 3 ? 2 : (lgTP == 4 ? 1 : (hh == 0 ? 1 : 0));
}
__device__ __forceinline__ int slot_of(int lgTP, int hh, int k) { return lgTP == 3 ? 2 * k + hh : (lgTP == 4 ? hh : 0); }

// SK: slices of the instance (all in registers), NP: 2 = hi/lo products of a
// float master, 1 = half weights; kMode: alignment of the window runs; QC:
// slices per kernel row when the instance is made for it (SK = Kh * QC), else
// 0.  With QC known, a slice's offset is one register per kernel row plus a
// constant, which the LDS reads take as their immediate offset.  TPC: steps
// per position in a tile when the instance is made for it, else 0.
template <int SK, int NP, int kMode, int QC, int TPC>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
void k_fire_pt(const uint8_t *__restrict__ xp, size_t xp_words, const h8 *__restrict__ bp, PGeom g,
               float theta, int nranges,
               uint8_t *__restrict__ out_t, float *__restrict__ out_v)
{
    extern __shared__ __align__(16) uint8_t lds[];
    const uint8_t *hal = lds + kHalOff;
    const uint8_t *flag = lds + kFlagOff;
    auto stv = [&](int i) { return reinterpret_cast<float *>(lds + kStvOff) + i * 32 * kStageStride; };
    auto stt = [&](int i) { return lds + kSttOff + i * 32 * kStageStride; };
    Tab *tabs = reinterpret_cast<Tab *>(lds + kTabOff);

    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // block -> (column tile, range); the NT blocks of a range share an XCD
    const int xcd = blockIdx.x & 7, q = blockIdx.x >> 3;
    const int nt = q % g.NT;
    const int range = xcd + 8 * (q / g.NT);
    if (range >= nranges) return;
    const int p_begin = (int)((long long)range * g.P / nranges);
    const int p_end = (int)((long long)(range + 1) * g.P / nranges);
    if (p_begin >= p_end) return;

    h8 bw[SK][NP];
#pragma unroll
    for (int s = 0; s < SK; s++)
#pragma unroll
        for (int k = 0; k < NP; k++) bw[s][k] = bp[((size_t)(nt * SK + s) * NP + k) * 64 + lane];

    // slice offsets from the window origin, in bytes of staged halves
    // (slices past the layer's read the origin; their B is zero)
    int off2[SK];
#pragma unroll
    for (int s = 0; s < SK; s++) {
        if constexpr (QC > 0) {
            off2[s] = 2 * (s / QC) * g.rowb + 32 * (s % QC);
        } else {
            const int ky = s / g.Q16, jq = s - ky * g.Q16;
            off2[s] = s < g.SK ? 2 * (ky * g.rowb + jq * 16) : 0;
        }
    }
    // this lane's slice for the fire flags of a tile (lanes past SK: none)
    const int my_off = lane < g.SK ? (lane / g.Q16) * g.rowb + (lane % g.Q16) * 16 : -1;

    // row (p, t) of this lane: slot p = r / TP, step t = r % TP (capped at T - 1)
    const int r = lane & 31, hh = lane >> 5;
    const int lgTP = TPC == 8 ? 3 : (TPC == 16 ? 4 : (TPC == 32 ? 5 : g.lgTP));
    int pl, tt;
    row_slot_step(r, lgTP, pl, tt);
    const uint32_t cbv = 0x6401u + (uint32_t)min(tt, g.T - 1);
    const h2 cc = as_h2(cbv | (cbv << 16));
    const int PT = 32 >> lgTP;  // positions per tile
    const uint32_t never4 = 0x01010101u * (uint32_t)g.T;
    // words a slice of the tile covers (see store_range)
    const int skip_pow = PT * ((g.Cp & 15) == 0 ? 1 : 2);

    {
        int r0, r1;
        group_rows(g, p_begin, min(p_end, p_begin + kG) - 1, r0, r1);
        const int a0 = (r0 * g.rowb) & ~15, a1 = r1 * g.rowb;
        store_range(load_range(xp, xp_words, a0, a1), lds + kHalOff, lds + kFlagOff,
                    reinterpret_cast<int *>(lds + kCntOff), never4, range_words(a0, a1), g.hw);
        fill_table(g, p_begin, min(p_end, p_begin + kG) - p_begin, tabs);
    }

    // Group it: computed from the staged input and table[it % 3] into
    // stage[it % 2]; its results are written out during group it + 1 (or
    // after the loop).  The next group's input is loaded into registers
    // during this one and stored once every wave is done with this one.
    int it = 0;
    for (int gs = p_begin; gs < p_end; gs += kG, it++) {
        const int cnt = min(p_end, gs + kG) - gs;
        const int cur = it & 1;
        const Tab *tab = tabs + (it % 3) * kG;
        int r0, r1;
        group_rows(g, gs, gs + cnt - 1, r0, r1);
        const int a0 = (r0 * g.rowb) & ~15;
        __syncthreads();  // this group's input and table are in LDS; group it-1 is staged
        const int gn = gs + kG;
        const bool more = gn < p_end;
        Staged<> nxt;
        int nxt_words = 0;
        if (more) {
            int n0, n1;
            group_rows(g, gn, min(p_end, gn + kG) - 1, n0, n1);
            const int b0 = (n0 * g.rowb) & ~15, b1 = n1 * g.rowb;
            nxt = load_range(xp, xp_words, b0, b1);
            nxt_words = range_words(b0, b1);
            fill_table(g, gn, min(p_end, gn + kG) - gn, tabs + ((it + 1) % 3) * kG);
        }
        if (it > 0)
            write_out(g, nt, gs - kG, p_end, tabs + ((it + 2) % 3) * kG, stv(cur ^ 1), stt(cur ^ 1), out_t, out_v);
        const bool sparse = group_sparse(reinterpret_cast<const int *>(lds + kCntOff), skip_pow, 0.4f);
        // tiles of the group go round the waves
        const int wp0 = gs + wv * PT, wp1 = gs + cnt, wstep = 4 * PT;
        int xo_next = tab[min(wp0 - gs + pl, cnt - 1)].xoff;
        for (int tp0 = wp0; tp0 < wp1; tp0 += wstep) {
            // this lane's window origin (taps from the staged range start)
            const int org2 = 2 * (xo_next - a0 + 8 * hh);
            auto rd = [&](int s) -> u4 { return lds_read16<kMode>(hal, org2 + off2[s]); };
            f16v acc;
#pragma unroll
            for (int e = 0; e < 16; e++) acc[e] = 0.0f;
            auto step = [&](int s, u4 x) {
                const h8 a = frag_upto(x, cc);
#pragma unroll
                for (int k = 0; k < NP; k++) acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bw[s][k], acc, 0, 0, 0);
            };
            // slices to compute: all, or in a sparse group those where an input
            // of some position of the tile fires (a slice's 16 bytes lie in at
            // most two flagged words)
            uint64_t live = ~0ull;
            if (sparse) {
                live = 0ull;
                for (int j = 0; j < PT; j++) {
                    const int xo = tab[min(tp0 - gs + j, cnt - 1)].xoff - a0;
                    bool f = false;
                    if (my_off >= 0) {
                        const int at = xo + my_off;
                        f = (flag[at >> 4] | flag[(at + 15) >> 4]) != 0;
                    }
                    live |= __builtin_amdgcn_ballot_w64(f);
                }
            }
            // reads run three slices ahead of the products; the dense form
            // has no branch between slices
            constexpr int kAhead = 3;
            u4 win[kAhead];
#pragma unroll
            for (int s = 0; s < kAhead && s < SK; s++) win[s] = rd(s);
            // the products at a raised wave priority (see k_fire_lb)
            __builtin_amdgcn_s_setprio(2);
            if (!sparse) {
#pragma unroll
                for (int s = 0; s < SK; s++) {
                    const u4 x = win[s % kAhead];
                    if (s + kAhead < SK) win[s % kAhead] = rd(s + kAhead);
                    step(s, x);
                    if constexpr (QC > 0 && kMode >= 1) {
                        // keep kAhead reads in flight: per slice, the LDS reads of
                        // one window piece, then the fragment's four VALU ops,
                        // then the products
                        constexpr int kReads = kMode == 1 ? 2 : 1;  // paired b32 reads merge
                        if (s + kAhead < SK) __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
                        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
                        __builtin_amdgcn_sched_group_barrier(0x008, NP, 0);
                    }
                }
            } else {
#pragma unroll
                for (int s = 0; s < SK; s++) {
                    const u4 x = win[s % kAhead];
                    if (s + kAhead < SK) win[s % kAhead] = rd(s + kAhead);
                    // (the bit test on a 32-bit half is one scalar instruction)
                    const uint32_t lw = s < 32 ? (uint32_t)live : (uint32_t)(live >> 32);
                    if (__builtin_expect((lw >> (s & 31)) & 1u, 1)) step(s, x);
                }
            }
            __builtin_amdgcn_s_setprio(0);
            // the next tile's window origin, read while this one finishes
            if (tp0 + wstep < wp1) xo_next = tab[min(tp0 + wstep - gs + pl, cnt - 1)].xoff;
            uint32_t st[2] = {0u, 0u};
            float sv[2] = {0.0f, 0.0f};
            if (lgTP == 3) tile_epilogue<8>(acc, theta, hh, st, sv);
            else if (lgTP == 4) tile_epilogue<16>(acc, theta, hh, st, sv);
            else tile_epilogue<32>(acc, theta, hh, st, sv);
            const int o = lane & 31, ns = slots_held(lgTP, hh);
#pragma unroll
            for (int k = 0; k < 2; k++) {
                const int pi = tp0 - gs + slot_of(lgTP, hh, k);
                if (k < ns && pi < cnt) {
                    stv(cur)[o * kStageStride + pi] = sv[k];
                    stt(cur)[o * kStageStride + pi] = (uint8_t)st[k];
                }
            }
        }
        if (more) {
            __syncthreads();  // every wave is done with this group's input
            store_range(nxt, lds + kHalOff, lds + kFlagOff, reinterpret_cast<int *>(lds + kCntOff), never4,
                        nxt_words, g.hw);
        }
    }
    __syncthreads();  // the last group is staged
    write_out(g, nt, p_begin + (it - 1) * kG, p_end, tabs + ((it - 1) % 3) * kG, stv((it - 1) & 1),
              stt((it - 1) & 1), out_t, out_v);
}

// Layers whose B fragments do not fit a wave's registers: each wave computes
// kRT tiles at once and streams the B fragments of one slice at a time from
// the workspace (L2), kD slices ahead, so every fragment read serves kRT
// products.  Input staging, the epilogue and the write-out are those of
// k_fire_pt; there is no slice skipping.
constexpr int kRT = 4, kD = 4;

template <int NP, int kMode>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
void k_fire_deep(const uint8_t *__restrict__ xp, size_t xp_words, const h8 *__restrict__ bp, PGeom g,
                 float theta, int nranges, uint8_t *__restrict__ out_t, float *__restrict__ out_v)
{
    extern __shared__ __align__(16) uint8_t lds[];
    const uint8_t *hal = lds + kHalOff;
    auto stv = [&](int i) { return reinterpret_cast<float *>(lds + kStvOff) + i * 32 * kStageStride; };
    auto stt = [&](int i) { return lds + kSttOff + i * 32 * kStageStride; };
    Tab *tabs = reinterpret_cast<Tab *>(lds + kTabOff);

    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int xcd = blockIdx.x & 7, q = blockIdx.x >> 3;
    const int nt = q % g.NT;
    const int range = xcd + 8 * (q / g.NT);
    if (range >= nranges) return;
    const int p_begin = (int)((long long)range * g.P / nranges);
    const int p_end = (int)((long long)(range + 1) * g.P / nranges);
    if (p_begin >= p_end) return;
    // B fragment (slice s, part k) of this lane: bcol[(s * NP + k) * 64]
    const h8 *bcol = bp + (size_t)nt * g.SKp * NP * 64 + lane;

    const int r = lane & 31, hh = lane >> 5;
    int pl, tt;
    row_slot_step(r, g.lgTP, pl, tt);
    const uint32_t cbv = 0x6401u + (uint32_t)min(tt, g.T - 1);
    const h2 cc = as_h2(cbv | (cbv << 16));
    const int PT = 32 >> g.lgTP;
    const uint32_t never4 = 0x01010101u * (uint32_t)g.T;

    {
        int r0, r1;
        group_rows(g, p_begin, min(p_end, p_begin + kG) - 1, r0, r1);
        const int a0 = (r0 * g.rowb) & ~15, a1 = r1 * g.rowb;
        store_range(load_range(xp, xp_words, a0, a1), lds + kHalOff, lds + kFlagOff,
                    reinterpret_cast<int *>(lds + kCntOff), never4, range_words(a0, a1), g.hw);
        fill_table(g, p_begin, min(p_end, p_begin + kG) - p_begin, tabs);
    }

    int it = 0;
    for (int gs = p_begin; gs < p_end; gs += kG, it++) {
        const int cnt = min(p_end, gs + kG) - gs;
        const int cur = it & 1;
        const Tab *tab = tabs + (it % 3) * kG;
        int r0, r1;
        group_rows(g, gs, gs + cnt - 1, r0, r1);
        const int a0 = (r0 * g.rowb) & ~15;
        __syncthreads();  // this group's input and table are in LDS; group it-1 is staged
        const int gn = gs + kG;
        const bool more = gn < p_end;
        Staged<> nxt;
        int nxt_words = 0;
        if (more) {
            int n0, n1;
            group_rows(g, gn, min(p_end, gn + kG) - 1, n0, n1);
            const int b0 = (n0 * g.rowb) & ~15, b1 = n1 * g.rowb;
            nxt = load_range(xp, xp_words, b0, b1);
            nxt_words = range_words(b0, b1);
            fill_table(g, gn, min(p_end, gn + kG) - gn, tabs + ((it + 1) % 3) * kG);
        }
        if (it > 0)
            write_out(g, nt, gs - kG, p_end, tabs + ((it + 2) % 3) * kG, stv(cur ^ 1), stt(cur ^ 1), out_t, out_v);

        // tiles of the group: tile i covers positions gs + i*PT ..; wave w
        // takes tiles w, w + 4, ..., kRT of them at a time
        const int ntiles = (cnt + PT - 1) / PT;
        for (int t0 = wv; t0 < ntiles; t0 += 4 * kRT) {
            int org2[kRT];
#pragma unroll
            for (int j = 0; j < kRT; j++) {
                const int slot = min((t0 + 4 * j) * PT + pl, cnt - 1);
                org2[j] = 2 * (tab[slot].xoff - a0 + 8 * hh);
            }
            f16v acc[kRT];
#pragma unroll
            for (int j = 0; j < kRT; j++)
#pragma unroll
                for (int e = 0; e < 16; e++) acc[j][e] = 0.0f;
            h8 ring[kD][NP];
#pragma unroll
            for (int d = 0; d < kD; d++)
#pragma unroll
                for (int k = 0; k < NP; k++) ring[d][k] = bcol[(size_t)(d * NP + k) * 64];
            int ky = 0, jq = 0;
            for (int s0 = 0; s0 < g.SKp; s0 += kD) {
#pragma unroll
                for (int d = 0; d < kD; d++) {
                    const int sl = s0 + d;
                    h8 bq[NP];
#pragma unroll
                    for (int k = 0; k < NP; k++) bq[k] = ring[d][k];
                    const int sn = sl + kD;  // this ring slot's next slice
                    if (sn < g.SKp)
#pragma unroll
                        for (int k = 0; k < NP; k++) ring[d][k] = bcol[(size_t)(sn * NP + k) * 64];
                    const int off = sl < g.SK ? 2 * (ky * g.rowb + jq * 16) : 0;
#pragma unroll
                    for (int j = 0; j < kRT; j++) {
                        const h8 a = frag_upto(lds_read16<kMode>(hal, org2[j] + off), cc);
#pragma unroll
                        for (int k = 0; k < NP; k++)
                            acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bq[k], acc[j], 0, 0, 0);
                    }
                    if (++jq == g.Q16) {
                        jq = 0;
                        ky++;
                    }
                }
            }
            const int o = lane & 31;
#pragma unroll
            for (int j = 0; j < kRT; j++) {
                const int ti = t0 + 4 * j;
                if (ti >= ntiles) continue;
                uint32_t st[2] = {0u, 0u};
                float sv[2] = {0.0f, 0.0f};
                if (g.lgTP == 3) tile_epilogue<8>(acc[j], theta, hh, st, sv);
                else if (g.lgTP == 4) tile_epilogue<16>(acc[j], theta, hh, st, sv);
                else tile_epilogue<32>(acc[j], theta, hh, st, sv);
                const int ns = slots_held(g.lgTP, hh);
#pragma unroll
                for (int k = 0; k < 2; k++) {
                    const int pi = ti * PT + slot_of(g.lgTP, hh, k);
                    if (k < ns && pi < cnt) {
                        stv(cur)[o * kStageStride + pi] = sv[k];
                        stt(cur)[o * kStageStride + pi] = (uint8_t)st[k];
                    }
                }
            }
        }
        if (more) {
            __syncthreads();  // every wave is done with this group's input
            store_range(nxt, lds + kHalOff, lds + kFlagOff, reinterpret_cast<int *>(lds + kCntOff), never4,
                        nxt_words, g.hw);
        }
    }
    __syncthreads();  // the last group is staged
    write_out(g, nt, p_begin + (it - 1) * kG, p_end, tabs + ((it - 1) % 3) * kG, stv((it - 1) & 1),
              stt((it - 1) & 1), out_t, out_v);
}

// ------------------------------------------------------------ LDS-fed firing
//
// k_fire_lb: the firing kernel with the B fragments of two column tiles (64
// maps) in LDS instead of registers.  One block of NW waves fills a CU (the
// fragments take SK*NP*2 KB of its LDS); each A fragment serves the products
// of both column tiles, and with the fragments out of the registers three or
// four waves share a SIMD, so one wave's epilogue, staging and waits overlap
// the others' products.  Positions, groups, staging, slice skipping and the
// epilogue are those of k_fire_pt; a block owns two column tiles of a range.
constexpr int kNTB = 2;         // column tiles per block
constexpr int kMB = 32 * kNTB;  // maps per block

template <int SK, int NP>
struct LbLayout {
    static constexpr size_t stv = (size_t)SK * NP * kNTB * 64 * sizeof(h8);  // B fragments [s][k][c][lane] first
    static constexpr size_t stt = stv + 2 * kMB * kStageStride * sizeof(float);
    static constexpr size_t tab = (stt + 2 * kMB * kStageStride + 15) / 16 * 16;
    static constexpr size_t cnt = tab + kTabBytes;
    static constexpr size_t flag = cnt + 2 * 16 * sizeof(int);
    static constexpr size_t hal = (flag + kRange / 16 + 15) / 16 * 16;
};

// Staged results of positions [gs, min(gs + 64, p_end)) of the block's NM
// maps (first output map m0) to the outputs: four consecutive positions of a
// map per thread, as in write_out.
template <int NTH, int NM = kMB>
__device__ __forceinline__ void write_out_lb(const PGeom &g, int m0, int gs, int p_end, const Tab *tab,
                                             const float *stv, const uint8_t *stt,
                                             uint8_t *__restrict__ out_t, float *__restrict__ out_v)
{
    constexpr int kQ = kG / 4;
    const int HoWo = g.Ho * g.Wo;
    const int cnt = min(p_end, gs + kG) - gs;
    const bool aligned = ((reinterpret_cast<uintptr_t>(out_v) & 15) | (reinterpret_cast<uintptr_t>(out_t) & 3)) == 0;
    for (int idx = threadIdx.x; idx < kQ * NM; idx += NTH) {
        const int p4 = 4 * (idx % kQ), oc = idx / kQ, ov = m0 + oc;
        if (p4 >= cnt || ov >= g.Cv) continue;
        const Tab t0 = tab[p4];
        const int n3 = tab[min(p4 + 3, kG - 1)].obase;
        const float *sv = stv + oc * kStageStride + p4;
        const uint8_t *st = stt + oc * kStageStride + p4;
        if (p4 + 3 < cnt && n3 == t0.obase + 3 && (t0.obase & 3) == 0 && (HoWo & 3) == 0 && aligned) {
            const int n = t0.obase + ov * HoWo;
            *reinterpret_cast<float4 *>(out_v + n) = make_float4(sv[0], sv[1], sv[2], sv[3]);
            *reinterpret_cast<uint32_t *>(out_t + n) =
                (uint32_t)st[0] | ((uint32_t)st[1] << 8) | ((uint32_t)st[2] << 16) | ((uint32_t)st[3] << 24);
        } else {
            for (int i = 0; i < 4 && p4 + i < cnt; i++) {
                const int n = tab[p4 + i].obase + ov * HoWo;
                out_v[n] = sv[i];
                out_t[n] = st[i];
            }
        }
    }
}

// SK (= the layer's packed slices), NP, kMode, QC and TPC as in k_fire_pt
// (QC and TPC fixed: instances are made per layout); NW waves per block.
template <int SK, int NP, int kMode, int QC, int TPC, int NW>
__global__ __launch_bounds__(64 * NW) void k_fire_lb(const uint8_t *__restrict__ xp, size_t xp_words,
                                                     const h8 *__restrict__ bp, PGeom g, float theta,
                                                     int nranges, uint8_t *__restrict__ out_t,
                                                     float *__restrict__ out_v)
{
    constexpr int NTH = 64 * NW;
    typedef LbLayout<SK, NP> L;
    extern __shared__ __align__(16) uint8_t lds[];
    h8 *bl = reinterpret_cast<h8 *>(lds);
    const uint8_t *hal = lds + L::hal;
    const uint8_t *flag = lds + L::flag;
    int *cntw = reinterpret_cast<int *>(lds + L::cnt);
    auto stv = [&](int i) { return reinterpret_cast<float *>(lds + L::stv) + i * kMB * kStageStride; };
    auto stt = [&](int i) { return lds + L::stt + i * kMB * kStageStride; };
    Tab *tabs = reinterpret_cast<Tab *>(lds + L::tab);

    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // block -> (column pair, range); the column pairs of a range share an XCD
    const int ncb = (g.NT + kNTB - 1) / kNTB;
    const int xcd = blockIdx.x & 7, q = blockIdx.x >> 3;
    const int cb = q % ncb;
    const int range = xcd + 8 * (q / ncb);
    if (range >= nranges) return;
    const int p_begin = (int)((long long)range * g.P / nranges);
    const int p_end = (int)((long long)(range + 1) * g.P / nranges);
    if (p_begin >= p_end) return;

    // the B fragments of column tiles 2cb and 2cb + 1 (zero past the last)
    for (int i = threadIdx.x; i < SK * NP * kNTB * 64; i += NTH) {
        const int ln = i & 63, c = (i >> 6) % kNTB, sk = i / (64 * kNTB);
        const int nt = cb * kNTB + c;
        h8 v = (h8)((_Float16)0.0f);
        if (nt < g.NT) v = bp[((size_t)nt * g.SKp * NP + sk) * 64 + ln];
        bl[i] = v;
    }

    int off2[SK];
#pragma unroll
    for (int s = 0; s < SK; s++) off2[s] = 2 * (s / QC) * g.rowb + 32 * (s % QC);
    const int my_off = lane < g.SK ? (lane / g.Q16) * g.rowb + (lane % g.Q16) * 16 : -1;

    const int r = lane & 31, hh = lane >> 5;
    constexpr int lgTP = TPC == 8 ? 3 : (TPC == 16 ? 4 : 5);
    int pl, tt;
    row_slot_step(r, lgTP, pl, tt);
    const uint32_t cbv = 0x6401u + (uint32_t)min(tt, g.T - 1);
    const h2 cc = as_h2(cbv | (cbv << 16));
    constexpr int PT = 32 >> lgTP;
    const uint32_t never4 = 0x01010101u * (uint32_t)g.T;
    const int skip_pow = PT * ((g.Cp & 15) == 0 ? 1 : 2);

    {
        int r0, r1;
        group_rows(g, p_begin, min(p_end, p_begin + kG) - 1, r0, r1);
        const int a0 = (r0 * g.rowb) & ~15, a1 = r1 * g.rowb;
        store_range(load_range<NTH>(xp, xp_words, a0, a1), lds + L::hal, lds + L::flag, cntw, never4,
                    range_words(a0, a1), g.hw);
        fill_table(g, p_begin, min(p_end, p_begin + kG) - p_begin, tabs);
    }

    int it = 0;
    for (int gs = p_begin; gs < p_end; gs += kG, it++) {
        const int cnt = min(p_end, gs + kG) - gs;
        const int cur = it & 1;
        const Tab *tab = tabs + (it % 3) * kG;
        int r0, r1;
        group_rows(g, gs, gs + cnt - 1, r0, r1);
        const int a0 = (r0 * g.rowb) & ~15;
        __syncthreads();  // this group's input and table are in LDS; group it-1 is staged
        const int gn = gs + kG;
        const bool more = gn < p_end;
        Staged<NTH> nxt;
        int nxt_words = 0;
        if (more) {
            int n0, n1;
            group_rows(g, gn, min(p_end, gn + kG) - 1, n0, n1);
            const int b0 = (n0 * g.rowb) & ~15, b1 = n1 * g.rowb;
            nxt = load_range<NTH>(xp, xp_words, b0, b1);
            nxt_words = range_words(b0, b1);
            fill_table(g, gn, min(p_end, gn + kG) - gn, tabs + ((it + 1) % 3) * kG);
        }
        if (it > 0)
            write_out_lb<NTH>(g, cb * kMB, gs - kG, p_end, tabs + ((it + 2) % 3) * kG, stv(cur ^ 1),
                              stt(cur ^ 1), out_t, out_v);
        const bool sparse = group_sparse<NW>(cntw, skip_pow, 0.15f);
        // tiles of the group go round the waves
        const int wp0 = gs + wv * PT, wp1 = gs + cnt, wstep = NW * PT;
        int xo_next = tab[min(wp0 - gs + pl, cnt - 1)].xoff;
        for (int tp0 = wp0; tp0 < wp1; tp0 += wstep) {
            const int org2 = 2 * (xo_next - a0 + 8 * hh);
            auto rdw = [&](int s) -> u4 { return lds_read16<kMode>(hal, org2 + off2[s]); };
            auto rdb = [&](int s, int k, int c) -> h8 { return bl[((s * NP + k) * kNTB + c) * 64 + lane]; };
            f16v acc[kNTB];
#pragma unroll
            for (int c = 0; c < kNTB; c++)
#pragma unroll
                for (int e = 0; e < 16; e++) acc[c][e] = 0.0f;
            uint64_t live = ~0ull;
            if (sparse) {
                live = 0ull;
                for (int j = 0; j < PT; j++) {
                    const int xo = tab[min(tp0 - gs + j, cnt - 1)].xoff - a0;
                    bool f = false;
                    if (my_off >= 0) {
                        const int at = xo + my_off;
                        f = (flag[at >> 4] | flag[(at + 15) >> 4]) != 0;
                    }
                    live |= __builtin_amdgcn_ballot_w64(f);
                }
            }
            // window reads two slices ahead; the B fragments are read where
            // they are used (in a sparse tile, only for its live slices)
            constexpr int kAhead = 2;
            u4 win[kAhead];
#pragma unroll
            for (int s = 0; s < kAhead && s < SK; s++) win[s] = rdw(s);
            auto slice = [&](int s, bool run) {
                const u4 x = win[s % kAhead];
                h8 b[NP][kNTB];
#pragma unroll
                for (int k = 0; k < NP; k++)
#pragma unroll
                    for (int c = 0; c < kNTB; c++) b[k][c] = rdb(s, k, c);
                if (s + kAhead < SK) win[s % kAhead] = rdw(s + kAhead);
                if (run) {
                    const h8 a = frag_upto(x, cc);
#pragma unroll
                    for (int k = 0; k < NP; k++)
#pragma unroll
                        for (int c = 0; c < kNTB; c++)
                            acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b[k][c], acc[c], 0, 0, 0);
                }
            };
            // the products run at a raised wave priority, so that a wave in
            // its slice loop issues ahead of the waves in their epilogue or
            // staging on the same SIMD
            __builtin_amdgcn_s_setprio(2);
            if (!sparse) {
#pragma unroll
                for (int s = 0; s < SK; s++) {
                    slice(s, true);
                    if constexpr (kMode >= 1) {
                        // per slice: the window and B reads, the fragment's four
                        // VALU ops, then the products
                        constexpr int kReads = (kMode == 1 ? 2 : 1) + NP * kNTB;
                        __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
                        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
                        __builtin_amdgcn_sched_group_barrier(0x008, NP * kNTB, 0);
                    }
                }
            } else {
#pragma unroll
                for (int s = 0; s < SK; s++) {
                    const uint32_t lw = s < 32 ? (uint32_t)live : (uint32_t)(live >> 32);
                    slice(s, __builtin_expect((lw >> (s & 31)) & 1u, 1));
                }
            }
            __builtin_amdgcn_s_setprio(0);
            if (tp0 + wstep < wp1) xo_next = tab[min(tp0 + wstep - gs + pl, cnt - 1)].xoff;
            const int o = lane & 31, ns = slots_held(lgTP, hh);
#pragma unroll
            for (int c = 0; c < kNTB; c++) {
                uint32_t st[2] = {0u, 0u};
                float sv[2] = {0.0f, 0.0f};
                tile_epilogue<TPC>(acc[c], theta, hh, st, sv);
#pragma unroll
                for (int k = 0; k < 2; k++) {
                    const int pi = tp0 - gs + slot_of(lgTP, hh, k);
                    if (k < ns && pi < cnt) {
                        stv(cur)[(c * 32 + o) * kStageStride + pi] = sv[k];
                        stt(cur)[(c * 32 + o) * kStageStride + pi] = (uint8_t)st[k];
                    }
                }
            }
        }
        if (more) {
            __syncthreads();  // every wave is done with this group's input
            store_range(nxt, lds + L::hal, lds + L::flag, cntw, never4, nxt_words, g.hw);
        }
    }
    __syncthreads();  // the last group is staged
    write_out_lb<NTH>(g, cb * kMB, p_begin + (it - 1) * kG, p_end, tabs + ((it - 1) % 3) * kG,
                      stv((it - 1) & 1), stt((it - 1) & 1), out_t, out_v);
}

// k_fire_lbk: the LDS-fed firing kernel for layers whose B fragments do not
// fit LDS whole (k_fire_deep's layers): one column tile per block, its
// fragments staged KC slices (one kernel row) at a time.  A wave keeps the
// accumulators of its TPW tiles of the group across the chunks; the next
// chunk's fragments are loaded into registers while the current one's
// products run.  Staging, slice skipping, the epilogue and the write-out are
// those of k_fire_lb.
template <int KC, int NP>
struct LbkLayout {
    static constexpr size_t stv = (size_t)KC * NP * 64 * sizeof(h8);  // B chunk [s][k][lane] first
    static constexpr size_t stt = stv + 2 * 32 * kStageStride * sizeof(float);
    static constexpr size_t tab = (stt + 2 * 32 * kStageStride + 15) / 16 * 16;
    static constexpr size_t cnt = tab + kTabBytes;
    static constexpr size_t flag = cnt + 2 * 16 * sizeof(int);
    static constexpr size_t hal = (flag + kRange / 16 + 15) / 16 * 16;
};

template <int SKT, int NP, int kMode, int QC, int TPC, int NW, int KC>
__global__ __launch_bounds__(64 * NW) void k_fire_lbk(const uint8_t *__restrict__ xp, size_t xp_words,
                                                      const h8 *__restrict__ bp, PGeom g, float theta,
                                                      int nranges, uint8_t *__restrict__ out_t,
                                                      float *__restrict__ out_v)
{
    static_assert(SKT % KC == 0 && SKT <= 64, "whole chunks, slices within the live mask");
    constexpr int NTH = 64 * NW;
    constexpr int NCH = SKT / KC;
    constexpr int lgTP = TPC == 8 ? 3 : (TPC == 16 ? 4 : 5);
    constexpr int PT = 32 >> lgTP;
    constexpr int TPW = (kG / PT + NW - 1) / NW;          // tiles of a group per wave
    constexpr int CW = KC * NP * 64;                      // fragments of a chunk
    constexpr int BPF = (CW + NTH - 1) / NTH;             // of them per thread
    typedef LbkLayout<KC, NP> L;
    extern __shared__ __align__(16) uint8_t lds[];
    h8 *bl = reinterpret_cast<h8 *>(lds);
    const uint8_t *hal = lds + L::hal;
    const uint8_t *flag = lds + L::flag;
    int *cntw = reinterpret_cast<int *>(lds + L::cnt);
    auto stv = [&](int i) { return reinterpret_cast<float *>(lds + L::stv) + i * 32 * kStageStride; };
    auto stt = [&](int i) { return lds + L::stt + i * 32 * kStageStride; };
    Tab *tabs = reinterpret_cast<Tab *>(lds + L::tab);

    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // block -> (column tile, range); the column tiles of a range share an XCD
    const int xcd = blockIdx.x & 7, q = blockIdx.x >> 3;
    const int nt = q % g.NT;
    const int range = xcd + 8 * (q / g.NT);
    if (range >= nranges) return;
    const int p_begin = (int)((long long)range * g.P / nranges);
    const int p_end = (int)((long long)(range + 1) * g.P / nranges);
    if (p_begin >= p_end) return;

    // chunk c's fragments of this thread into registers (slices past the
    // layer's are zero in the packed operand)
    const h8 *bcol = bp + (size_t)nt * g.SKp * NP * 64;
    h8 bpre[BPF];
    auto fetch = [&](int c) {
#pragma unroll
        for (int i = 0; i < BPF; i++) {
            const int e = (int)threadIdx.x + NTH * i;
            if (e < CW) bpre[i] = bcol[(size_t)c * CW + e];
        }
    };
    auto put = [&]() {
#pragma unroll
        for (int i = 0; i < BPF; i++) {
            const int e = (int)threadIdx.x + NTH * i;
            if (e < CW) bl[e] = bpre[i];
        }
    };
    fetch(0);

    const int my_off = lane < g.SK ? (lane / g.Q16) * g.rowb + (lane % g.Q16) * 16 : -1;
    const int r = lane & 31, hh = lane >> 5;
    int pl, tt;
    row_slot_step(r, lgTP, pl, tt);
    const uint32_t cbv = 0x6401u + (uint32_t)min(tt, g.T - 1);
    const h2 cc = as_h2(cbv | (cbv << 16));
    const uint32_t never4 = 0x01010101u * (uint32_t)g.T;
    const int skip_pow = PT * ((g.Cp & 15) == 0 ? 1 : 2);

    {
        int r0, r1;
        group_rows(g, p_begin, min(p_end, p_begin + kG) - 1, r0, r1);
        const int a0 = (r0 * g.rowb) & ~15, a1 = r1 * g.rowb;
        store_range(load_range<NTH>(xp, xp_words, a0, a1), lds + L::hal, lds + L::flag, cntw, never4,
                    range_words(a0, a1), g.hw);
        fill_table(g, p_begin, min(p_end, p_begin + kG) - p_begin, tabs);
    }

    int it = 0;
    for (int gs = p_begin; gs < p_end; gs += kG, it++) {
        const int cnt = min(p_end, gs + kG) - gs;
        const int cur = it & 1;
        const Tab *tab = tabs + (it % 3) * kG;
        int r0, r1;
        group_rows(g, gs, gs + cnt - 1, r0, r1);
        const int a0 = (r0 * g.rowb) & ~15;
        __syncthreads();  // this group's input and table are in LDS; group it-1 is staged
        const int gn = gs + kG;
        const bool more = gn < p_end;
        Staged<NTH> nxt;
        int nxt_words = 0;
        if (more) {
            int n0, n1;
            group_rows(g, gn, min(p_end, gn + kG) - 1, n0, n1);
            const int b0 = (n0 * g.rowb) & ~15, b1 = n1 * g.rowb;
            nxt = load_range<NTH>(xp, xp_words, b0, b1);
            nxt_words = range_words(b0, b1);
            fill_table(g, gn, min(p_end, gn + kG) - gn, tabs + ((it + 1) % 3) * kG);
        }
        if (it > 0)
            write_out_lb<NTH, 32>(g, nt * 32, gs - kG, p_end, tabs + ((it + 2) % 3) * kG, stv(cur ^ 1),
                                  stt(cur ^ 1), out_t, out_v);
        const bool sparse = group_sparse<NW>(cntw, skip_pow, 0.15f);
        // this wave's tiles of the group: wv, wv + NW, ...
        const int ntiles = (cnt + PT - 1) / PT;
        int org2[TPW];
        uint64_t live[TPW];
        f16v acc[TPW];
#pragma unroll
        for (int j = 0; j < TPW; j++) {
            const int ti = wv + NW * j;
            org2[j] = 2 * (tab[min(ti * PT + pl, cnt - 1)].xoff - a0 + 8 * hh);
            live[j] = ti < ntiles ? ~0ull : 0ull;
            if (sparse && ti < ntiles) {
                uint64_t m = 0ull;
                for (int k = 0; k < PT; k++) {
                    const int xo = tab[min(ti * PT + k, cnt - 1)].xoff - a0;
                    bool f = false;
                    if (my_off >= 0) {
                        const int at = xo + my_off;
                        f = (flag[at >> 4] | flag[(at + 15) >> 4]) != 0;
                    }
                    m |= __builtin_amdgcn_ballot_w64(f);
                }
                live[j] = m;
            }
#pragma unroll
            for (int e = 0; e < 16; e++) acc[j][e] = 0.0f;
        }
#pragma unroll
        for (int ch = 0; ch < NCH; ch++) {
            if (ch > 0) __syncthreads();  // every wave is done with chunk ch - 1
            put();
            __syncthreads();  // chunk ch is in LDS
            fetch(ch + 1 < NCH ? ch + 1 : 0);  // the next chunk (the next group starts again at 0)
            __builtin_amdgcn_s_setprio(2);
#pragma unroll
            for (int j = 0; j < TPW; j++) {
                if (!(live[j] >> (ch * KC) & ((KC < 64 ? (1ull << KC) : 0ull) - 1ull))) continue;  // no live slice here
                constexpr int kAhead = 2;
                auto rdw = [&](int sl) -> u4 {
                    return lds_read16<kMode>(hal, org2[j] + 2 * ((ch * KC + sl) / QC) * g.rowb +
                                                      32 * ((ch * KC + sl) % QC));
                };
                u4 win[kAhead];
#pragma unroll
                for (int sl = 0; sl < kAhead && sl < KC; sl++) win[sl] = rdw(sl);
                const uint64_t lw = live[j] >> (ch * KC);
#pragma unroll
                for (int sl = 0; sl < KC; sl++) {
                    const u4 x = win[sl % kAhead];
                    if (sl + kAhead < KC) win[sl % kAhead] = rdw(sl + kAhead);
                    const uint32_t lb = sl < 32 ? (uint32_t)lw : (uint32_t)(lw >> 32);
                    if ((lb >> (sl & 31)) & 1u) {
                        h8 b[NP];
#pragma unroll
                        for (int k = 0; k < NP; k++) b[k] = bl[(sl * NP + k) * 64 + lane];
                        const h8 a = frag_upto(x, cc);
#pragma unroll
                        for (int k = 0; k < NP; k++)
                            acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b[k], acc[j], 0, 0, 0);
                    }
                }
            }
            __builtin_amdgcn_s_setprio(0);
        }
        const int o = lane & 31, ns = slots_held(lgTP, hh);
#pragma unroll
        for (int j = 0; j < TPW; j++) {
            const int ti = wv + NW * j;
            if (ti >= ntiles) continue;
            uint32_t st[2] = {0u, 0u};
            float sv[2] = {0.0f, 0.0f};
            tile_epilogue<TPC>(acc[j], theta, hh, st, sv);
#pragma unroll
            for (int k = 0; k < 2; k++) {
                const int pi = ti * PT + slot_of(lgTP, hh, k);
                if (k < ns && pi < cnt) {
                    stv(cur)[o * kStageStride + pi] = sv[k];
                    stt(cur)[o * kStageStride + pi] = (uint8_t)st[k];
                }
            }
        }
        if (more) {
            __syncthreads();  // every wave is done with this group's input
            store_range(nxt, lds + L::hal, lds + L::flag, cntw, never4, nxt_words, g.hw);
        }
    }
    __syncthreads();  // the last group is staged
    write_out_lb<NTH, 32>(g, nt * 32, p_begin + (it - 1) * kG, p_end, tabs + ((it - 1) % 3) * kG,
                          stv((it - 1) & 1), stt((it - 1) & 1), out_t, out_v);
}

// Kernel instances: slice counts rounded up to these (the extra slices have
// zero weights).  Float masters (hi/lo) keep 4*2*SK registers of B fragments,
// halves 4*SK: both up to 144.
constexpr int kSK2[] = {2, 4, 6, 8, 10, 12, 14, 16, 18};
constexpr int kSK1[] = {4, 8, 12, 16, 20, 24, 28, 32, 36};

int instance_sk(int SK, bool half_w)
{
    const int *t = half_w ? kSK1 : kSK2;
    for (int i = 0; i < 9; i++)
        if (SK <= t[i]) return t[i];
    return 0;
}

// Slices packed for a layer: a register-resident instance's count, or (deep
// layers) the slices rounded up to the prefetch depth.
int packed_sk(int SK, bool half_w)
{
    const int i = instance_sk(SK, half_w);
    return i ? i : (SK + kD - 1) / kD * kD;
}

template <int NP, int kMode>
void launch_deep(dim3 grid, size_t lds, hipStream_t s, const uint8_t *xp, size_t xw, const h8 *bp,
                 const PGeom &g, float theta, int nranges, uint8_t *ot, float *ov)
{
    hipLaunchKernelGGL((k_fire_deep<NP, kMode>), grid, dim3(kThreads), lds, s, xp, xw, bp, g, theta,
                       nranges, ot, ov);
}

typedef void (*PtLaunch)(dim3, size_t, hipStream_t, const uint8_t *, size_t, const h8 *, const PGeom &,
                         float, int, uint8_t *, float *);

template <int SK, int NP, int kMode, int QC = 0, int TPC = 0>
void launch_pt(dim3 grid, size_t lds, hipStream_t s, const uint8_t *xp, size_t xw, const h8 *bp,
               const PGeom &g, float theta, int nranges, uint8_t *ot, float *ov)
{
    hipLaunchKernelGGL((k_fire_pt<SK, NP, kMode, QC, TPC>), grid, dim3(kThreads), lds, s, xp, xw, bp, g,
                       theta, nranges, ot, ov);
}

// Instances made for one slice layout and tile shape: (SK, QC, NP, kMode, TP)
// of a layer whose Khv * Q16 equals the instance's slices.  3x3 over 32
// padded channels with float masters, 5x5 over 6 channels, the 6 x 8 window
// of a 2 x 4 block of 5x5 positions over 6 channels (four maps), 3x3 over 64
// channels with half weights; 16 or 32 steps per position.
struct PtExact {
    int SK, QC, NP, mode, TP;
    PtLaunch fn;
};
const PtExact kExact[] = {
    {18, 6, 2, 3, 16, &launch_pt<18, 2, 3, 6, 16>},
    {10, 2, 2, 1, 16, &launch_pt<10, 2, 1, 2, 16>},
    {10, 2, 2, 1, 32, &launch_pt<10, 2, 1, 2, 32>},
    {18, 3, 2, 1, 32, &launch_pt<18, 2, 1, 3, 32>},
    {36, 12, 1, 3, 32, &launch_pt<36, 1, 3, 12, 32>},
};

#define SPK_PT(S, N) {&launch_pt<S, N, 0>, &launch_pt<S, N, 1>, &launch_pt<S, N, 2>, &launch_pt<S, N, 3>}
const PtLaunch kLaunch2[9][4] = {SPK_PT(2, 2),  SPK_PT(4, 2),  SPK_PT(6, 2),  SPK_PT(8, 2), SPK_PT(10, 2),
                                 SPK_PT(12, 2), SPK_PT(14, 2), SPK_PT(16, 2), SPK_PT(18, 2)};
const PtLaunch kLaunch1[9][4] = {SPK_PT(4, 1),  SPK_PT(8, 1),  SPK_PT(12, 1), SPK_PT(16, 1), SPK_PT(20, 1),
                                 SPK_PT(24, 1), SPK_PT(28, 1), SPK_PT(32, 1), SPK_PT(36, 1)};
#undef SPK_PT
const PtLaunch kDeep[2][4] = {{&launch_deep<1, 0>, &launch_deep<1, 1>, &launch_deep<1, 2>, &launch_deep<1, 3>},
                              {&launch_deep<2, 0>, &launch_deep<2, 1>, &launch_deep<2, 2>, &launch_deep<2, 3>}};

template <int SK, int NP, int kMode, int QC, int TPC, int NW>
void launch_lb(dim3 grid, size_t lds, hipStream_t s, const uint8_t *xp, size_t xw, const h8 *bp,
               const PGeom &g, float theta, int nranges, uint8_t *ot, float *ov)
{
    auto kern = k_fire_lb<SK, NP, kMode, QC, TPC, NW>;
    static const bool attr = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize,
                                                 160 * 1024) == hipSuccess;
    (void)attr;
    hipLaunchKernelGGL(kern, grid, dim3(64 * NW), lds, s, xp, xw, bp, g, theta, nranges, ot, ov);
}

// Layouts the LDS-fed kernel is made for (as kExact), with the LDS it needs
// before the staged input: 3x3 over 64 channels with half weights and 32
// steps per position; 5x5 over 6 channels with float masters and 16.  (3x3
// over 32 padded channels with float masters, the three-layer net's conv2,
// ran slower in it: 56 against 54 us.)
struct LbExact {
    int SK, QC, NP, mode, TP;
    size_t hal;
    PtLaunch fn;
};
const LbExact kLbExact[] = {
    {36, 12, 1, 3, 32, LbLayout<36, 1>::hal, &launch_lb<36, 1, 3, 12, 32, 16>},
    {10, 2, 2, 1, 16, LbLayout<10, 2>::hal, &launch_lb<10, 2, 1, 2, 16, 12>},
};

template <int SKT, int NP, int kMode, int QC, int TPC, int NW, int KC>
void launch_lbk(dim3 grid, size_t lds, hipStream_t s, const uint8_t *xp, size_t xw, const h8 *bp,
                const PGeom &g, float theta, int nranges, uint8_t *ot, float *ov)
{
    auto kern = k_fire_lbk<SKT, NP, kMode, QC, TPC, NW, KC>;
    static const bool attr = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize,
                                                 160 * 1024) == hipSuccess;
    (void)attr;
    hipLaunchKernelGGL(kern, grid, dim3(64 * NW), lds, s, xp, xw, bp, g, theta, nranges, ot, ov);
}

// Layouts of the chunked LDS-fed kernel: 3x3 over 100 channels with float
// masters and 16 steps per position (the example network's conv2), a kernel
// row of 19 slices per chunk.
const LbExact kLbkExact[] = {
    {57, 19, 2, 2, 16, LbkLayout<19, 2>::hal, &launch_lbk<57, 2, 2, 19, 16, 16, 19>},
};

// Largest staged row range over the groups of every range (exact, per geometry).
int max_rows(const PGeom &g, int nranges)
{
    typedef std::tuple<int, int, int, int, int, int, int, int, int, int, int> Key;
    static std::mutex mu;
    static std::map<Key, int> memo;
    const Key key{g.B, g.Hi, g.Wi, g.Kh, g.stride, g.pad, g.Ho, g.Wo, nranges, g.by, g.bx};
    {
        std::lock_guard<std::mutex> lock(mu);
        auto it = memo.find(key);
        if (it != memo.end()) return it->second;
    }
    int best = 0;
    for (int rg = 0; rg < nranges; rg++) {
        const int pb = (int)((long long)rg * g.P / nranges), pe = (int)((long long)(rg + 1) * g.P / nranges);
        for (int gs = pb; gs < pe; gs += kG) {
            int r0, r1;
            group_rows(g, gs, std::min(pe, gs + kG) - 1, r0, r1);
            best = std::max(best, r1 - r0);
        }
    }
    std::lock_guard<std::mutex> lock(mu);
    if (memo.size() > 4096) memo.clear();
    memo[key] = best;
    return best;
}

int cu_count()
{
    static int n = 0;
    if (n == 0) {
        int dev = 0, v = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
            n = v;
        else
            n = 256;
    }
    return n;
}

int n_ranges(const PGeom &g)
{
    const int target = 2 * cu_count();
    int nr = std::max(1, target / g.NT);
    nr = std::min(nr, std::max(1, g.P / 16));
    return nr;
}

size_t fire_lds(const PGeom &g) { return kHalOff + 32 * (size_t)g.hw; }

// Ranges of the LDS-fed kernel: one block per CU, ncb column pairs per range.
int n_ranges_lb(const PGeom &g, int ncb)
{
    int nr = std::max(1, cu_count() / ncb);
    nr = std::min(nr, std::max(1, g.P / 16));
    return nr;
}

}  // namespace

namespace spk {

bool conv_pt_supported(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride,
                       int pad, int Ho, int Wo, bool half_w, bool readout, bool potentials)
{
    if (readout || potentials || T < 1 || T > 32 || B < 1 || Ci < 1 || Co < 1 || Ho < 1 || Wo < 1)
        return false;
    const long long Hp = Hi + 2ll * pad, Wp = Wi + 2ll * pad;
    if ((long long)B * Co * Ho * Wo >= (1ll << 31)) return false;
    if (Wp * (Ci + 8) > 48 * 1024 || (long long)Ci * Kh * Kw * 4 > 64 * 1024) return false;
    if (B * Hp * Wp * (Ci + 8) + 64 * Wp * (Ci + 8) >= (1ll << 30)) return false;
    const PGeom g = make_pgeom(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo, half_w);
    if (g.SK > 4096) return false;
    // a group's rows, with the 16-byte alignment in front and 32 bytes of over-read
    const long long rows = max_rows(g, n_ranges(g));
    return rows * g.rowb + 64 <= kRange;
}

size_t conv_pt_workspace(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride,
                         int pad, int Ho, int Wo)
{
    // the geometry (block shape) may differ between float and half weights
    size_t need = 0;
    for (int hw = 0; hw < 2; hw++) {
        PGeom g = make_pgeom(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo, hw != 0);
        g.SKp = std::max(packed_sk(g.SK, false), packed_sk(g.SK, true));
        need = std::max(need, xp_bytes(g) + bp_bytes(g, 2));
    }
    return need;
}

spk_status conv_fire_pt(const uint8_t *in, int B, int T, int Ci, int Hi, int Wi, const void *w,
                        bool half_w, int Co, int Kh, int Kw, int stride, int pad, int Ho, int Wo,
                        float theta, uint8_t *out_t, float *out_v, void *ws, hipStream_t s,
                        const PoolIn *pool)
{
    PGeom g = make_pgeom(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo, half_w);
    g.SKp = packed_sk(g.SK, half_w);
    uint8_t *xp = reinterpret_cast<uint8_t *>(ws);
    h8 *bp = reinterpret_cast<h8 *>(reinterpret_cast<char *>(ws) + xp_bytes(g));
    // a pooled input row stages its window rows past the row buffer when
    // they fit; otherwise its cells are pooled one by one
    PoolIn pl = pool ? *pool : PoolIn{};
    pl.stage = -1;
    const size_t stage_at = align_up((size_t)g.rowb, 16);
    if (pool && stage_at + pool_stage_bytes(pl, g.Ci) <= 64 * 1024) pl.stage = (int)stage_at;
    // input blocks: one per padded row, or 1024 Xp bytes each (cells pooled one by one)
    const int nb_in = pool && pl.stage < 0 ? ceil_div((long long)g.B * g.Hp * g.rowb + g.slack, 1024)
                                           : g.B * g.Hp;
    const size_t wlds = (size_t)g.Ci * g.Kh * g.Kw * sizeof(float);
    const size_t plds = std::max(wlds, !pool ? (size_t)g.rowb
                                       : pl.stage >= 0 ? stage_at + pool_stage_bytes(pl, g.Ci) : (size_t)0);
    const dim3 pgrid(nb_in + g.NT * 32);
    if (half_w)
        hipLaunchKernelGGL((k_pack_pt<1, true>), pgrid, dim3(256), plds, s, in, w, g, nb_in, xp, bp, pl);
    else
        hipLaunchKernelGGL((k_pack_pt<2, false>), pgrid, dim3(256), plds, s, in, w, g, nb_in, xp, bp, pl);
    SPK_LAUNCHED("spk_conv_fire");

    const int nranges = n_ranges(g);
    // LDS halves for the largest group's range (the words a group stages)
    g.hw = (int)((max_rows(g, nranges) * (long long)g.rowb + 64 + 47) / 16);
    const int per_xcd = (nranges + 7) / 8;
    const dim3 grid(8 * g.NT * per_xcd);
    const size_t xw = ((size_t)g.B * g.Hp * g.rowb + g.slack) / 16;
    // the LDS-fed kernel for the layouts it is made for, when a group's rows
    // fit its staging and everything fits a CU's LDS
    if (g.by * g.bx == 1 && g.NT >= 2 && g.SKp == g.SK) {
        for (const LbExact &e : kLbExact) {
            if (e.SK != g.SK || e.QC != g.Q16 || e.NP != (half_w ? 1 : 2) || e.mode != read_mode(g.Cp) ||
                e.TP != g.TP)
                continue;
            const int ncb = (g.NT + kNTB - 1) / kNTB;
            const int nr = n_ranges_lb(g, ncb);
            const long long rows = max_rows(g, nr);
            if (rows * g.rowb + 64 > kRange) break;
            PGeom gl = g;
            gl.hw = (int)((rows * g.rowb + 64 + 47) / 16);
            const size_t lds = e.hal + 32 * (size_t)gl.hw;
            if (lds > 160 * 1024) break;
            const size_t xw = ((size_t)g.B * g.Hp * g.rowb + g.slack) / 16;
            e.fn(dim3(8 * ncb * ((nr + 7) / 8)), lds, s, xp, xw, bp, gl, theta, nr, out_t, out_v);
            return check_launch("spk_conv_fire");
        }
    }
    // the chunked LDS-fed kernel for the deep layouts it is made for
    if (g.by * g.bx == 1 && !instance_sk(g.SK, half_w)) {
        for (const LbExact &e : kLbkExact) {
            if (e.SK != g.SK || e.QC != g.Q16 || e.NP != (half_w ? 1 : 2) || e.mode != read_mode(g.Cp) ||
                e.TP != g.TP)
                continue;
            const int nr = n_ranges_lb(g, g.NT);
            const long long rows = max_rows(g, nr);
            if (rows * g.rowb + 64 > kRange) break;
            PGeom gl = g;
            gl.hw = (int)((rows * g.rowb + 64 + 47) / 16);
            const size_t lds = e.hal + 32 * (size_t)gl.hw;
            if (lds > 160 * 1024) break;
            const size_t xw = ((size_t)g.B * g.Hp * g.rowb + g.slack) / 16;
            e.fn(dim3(8 * g.NT * ((nr + 7) / 8)), lds, s, xp, xw, bp, gl, theta, nr, out_t, out_v);
            return check_launch("spk_conv_fire");
        }
    }
    PtLaunch launch;
    if (instance_sk(g.SK, half_w)) {
        int idx = 0;
        while ((half_w ? kSK1 : kSK2)[idx] != g.SKp) idx++;
        launch = (half_w ? kLaunch1 : kLaunch2)[idx][read_mode(g.Cp)];
        for (const PtExact &e : kExact)
            if (e.SK == g.SK && g.SKp == g.SK && e.QC == g.Q16 && e.NP == (half_w ? 1 : 2) &&
                e.mode == read_mode(g.Cp) && e.TP == g.TP)
                launch = e.fn;
    } else {
        launch = kDeep[half_w ? 0 : 1][read_mode(g.Cp)];
    }
    launch(grid, fire_lds(g), s, xp, xw, bp, g, theta, nranges, out_t, out_v);
    return check_launch("spk_conv_fire");
}

}  // namespace spk
