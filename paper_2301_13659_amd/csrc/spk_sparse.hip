// Sparse interface (Spyker §II-B): spike lists, their conversions to and from
// time maps, and the spiking convolution driven by a spike list.
//
// A spike list holds, per sample b, the flat indices (c*H + y)*W + x of the
// neurons that fire, grouped by step in ascending order and ascending index
// within a step: spikes[b*cap + j] is the j-th spike of sample b and
// offsets[b*(T + 1) + t] counts its spikes before step t (the entry at T is
// the sample's total).  Spikes past cap are counted but not stored.
//
// The convolution (Eq. 2 with the firing rule of §II-D.3 and §II-E) costs
// what the spikes cost: the list is scattered into a padded channels-last
// time buffer, and a wave per output position compacts the spikes of its
// window into a short list and adds their weights to the potentials of every
// map in step order, testing theta after each step that brought a spike.  A
// lane owns one or two maps; their weights sit in LDS as a tap-major table,
// so an arrival costs one LDS read and one add per map.
#include <hip/hip_fp16.h>

#include <algorithm>
#include <type_traits>

#include "spk_internal.h"

namespace {

// ------------------------------------------------------------ conversions

constexpr int kCvWaves = 16;  // waves of a conversion block
constexpr int kCvThreads = 64 * kCvWaves;

// Neurons [lo, hi) of sample b owned by one wave of the conversion grid: the
// sample is cut into nb chunks, each chunk into kCvWaves runs of whole
// 64-neuron groups.
__device__ __forceinline__ void wave_span(int64_t n, int nb, int chunk, int wave, int64_t &lo,
                                          int64_t &hi)
{
    const int64_t per = (n + nb - 1) / nb;
    const int64_t c0 = min(n, (int64_t)chunk * per), c1 = min(n, c0 + per);
    int64_t wper = (c1 - c0 + kCvWaves - 1) / kCvWaves;
    wper = (wper + 63) / 64 * 64;
    lo = min(c1, c0 + (int64_t)wave * wper);
    hi = min(c1, lo + wper);
}

// Spikes per (sample, chunk, wave, step).
__global__ __launch_bounds__(kCvThreads) void k_list_count(const uint8_t *__restrict__ times,
                                                           int64_t n, int T, int nb,
                                                           int32_t *__restrict__ cnt)
{
    extern __shared__ int32_t sc[];  // kCvWaves x T
    const int b = blockIdx.y, chunk = blockIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int32_t *mine = sc + wave * T;
    for (int t = lane; t < T; t += 64) mine[t] = 0;
    __syncthreads();
    int64_t lo, hi;
    wave_span(n, nb, chunk, wave, lo, hi);
    const uint8_t *tb = times + (size_t)b * n;
    for (int64_t i = lo + lane; i < hi; i += 64) {
        const uint32_t t = tb[i];
        if (t < (uint32_t)T) atomicAdd(&mine[t], 1);
    }
    __syncthreads();
    int32_t *dst = cnt + (((size_t)b * nb + chunk) * kCvWaves + wave) * T;
    for (int t = lane; t < T; t += 64) dst[t] = mine[t];
}

// Per sample: offsets of the steps, and each (chunk, wave)'s first slot of
// each step, in place of its count.  Units q = chunk*kCvWaves + wave are
// visited in neuron order, so a step's spikes come out in index order.
__global__ __launch_bounds__(256) void k_list_scan(int32_t *__restrict__ cnt, int T, int nq,
                                                   int32_t *__restrict__ offsets)
{
    extern __shared__ int32_t ss[];  // nq x T counts, then T step totals
    const int b = blockIdx.x;
    int32_t *c = cnt + (size_t)b * nq * T;
    int32_t *tot = ss + (size_t)nq * T;
    for (int i = threadIdx.x; i < nq * T; i += blockDim.x) ss[i] = c[i];
    __syncthreads();
    for (int t = threadIdx.x; t < T; t += blockDim.x) {
        int32_t run = 0;
        for (int q = 0; q < nq; q++) {
            const int32_t v = ss[q * T + t];
            ss[q * T + t] = run;
            run += v;
        }
        tot[t] = run;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int32_t run = 0;
        for (int t = 0; t < T; t++) {
            const int32_t v = tot[t];
            tot[t] = run;
            offsets[(size_t)b * (T + 1) + t] = run;
            run += v;
        }
        offsets[(size_t)b * (T + 1) + T] = run;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < nq * T; i += blockDim.x) c[i] = ss[i] + tot[i % T];
}

// The spikes, each at its step's slot plus its rank among the earlier
// neurons of the same step: across groups by a running count per (wave,
// step), within a group of 64 by lane, from ballots over the bits of t.
__global__ __launch_bounds__(kCvThreads) void k_list_scatter(const uint8_t *__restrict__ times,
                                                             int64_t n, int T, int tbits, int nb,
                                                             const int32_t *__restrict__ base,
                                                             int cap, uint32_t *__restrict__ spikes)
{
    extern __shared__ int32_t sr[];  // kCvWaves x T running slots
    const int b = blockIdx.y, chunk = blockIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int32_t *run = sr + wave * T;
    const int32_t *src = base + (((size_t)b * nb + chunk) * kCvWaves + wave) * T;
    for (int t = lane; t < T; t += 64) run[t] = src[t];
    __syncthreads();
    int64_t lo, hi;
    wave_span(n, nb, chunk, wave, lo, hi);
    const uint8_t *tb = times + (size_t)b * n;
    uint32_t *sb = spikes + (size_t)b * cap;
    for (int64_t g0 = lo; g0 < hi; g0 += 64) {
        const int64_t i = g0 + lane;
        const uint32_t t = i < hi ? tb[i] : 255u;
        const bool act = t < (uint32_t)T;
        uint64_t same = __ballot(act);
        if (!same) continue;
        for (int k = 0; k < tbits; k++) {
            const bool bit = (t >> k) & 1u;
            const uint64_t m = __ballot(bit);
            same &= bit ? m : ~m;
        }
        if (act) {
            const int rank = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(same >> 32),
                                                            __builtin_amdgcn_mbcnt_lo((uint32_t)same, 0u));
            const int32_t slot = run[t] + rank;
            if (slot < cap) sb[slot] = (uint32_t)i;
            if (rank == 0) run[t] += __popcll(same);
        }
    }
}

__global__ void k_fill_u8(uint8_t *__restrict__ p, size_t n, uint8_t v)
{
    const size_t n16 = n / 16;
    const uint32_t w = 0x01010101u * v;
    const uint4 q = make_uint4(w, w, w, w);
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t j = i; j < n16; j += stride) reinterpret_cast<uint4 *>(p)[j] = q;
    for (size_t j = n16 * 16 + i; j < n; j += stride) p[j] = v;
}

// Step of the j-th stored spike: the last t with offsets[t] <= j.
__device__ __forceinline__ int step_of(const int32_t *ob, int T, int32_t j)
{
    int lo = 0, hi = T - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (ob[mid] <= j) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// Threads of sample blockIdx.y stride over its stored spikes; each writes its
// step at its neuron of
// the B x C x H x W time map (dst_pad < 0) or of the padded channels-last
// buffer [b][y + pad][x + pad][c] (dst_pad >= 0).
__global__ void k_list_place(const uint32_t *__restrict__ spikes, const int32_t *__restrict__ offsets,
                             int cap, int B, int T, int C, int H, int W, int dst_pad,
                             uint8_t *__restrict__ dst)
{
    const int b = blockIdx.y;
    const int32_t *ob = offsets + (size_t)b * (T + 1);
    const int32_t total = min(ob[T], cap);
    const int64_t n = (int64_t)C * H * W;
    for (int32_t j = blockIdx.x * blockDim.x + threadIdx.x; j < total; j += gridDim.x * blockDim.x) {
        const uint32_t idx = spikes[(size_t)b * cap + j];
        if ((int64_t)idx >= n) continue;
        const uint8_t t = (uint8_t)step_of(ob, T, j);
        if (dst_pad < 0) {
            dst[(size_t)b * n + idx] = t;
            continue;
        }
        const int c = (int)(idx / (uint32_t)(H * W));
        const int r = (int)(idx - (uint32_t)c * H * W);
        const int y = r / W, x = r - y * W;
        const int Hp = H + 2 * dst_pad, Wp = W + 2 * dst_pad;
        dst[(((size_t)b * Hp + y + dst_pad) * Wp + x + dst_pad) * C + c] = t;
    }
}

// ------------------------------------------------------------ event conv

constexpr int kEvMaxWaves = 16;
constexpr int kEvMaxChunks = 4;  // list capacity per wave <= 64 * this
constexpr int kEvSlack = 64;

struct EGeom {
    int B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, Ho, Wo;
    int Hp, Wp;
    int rowb;   // Wp * Ci: bytes of one padded input row
    int run;    // Kw * Ci: taps of one kernel row
    int nch;    // ceil(run / 64)
    int taps;   // Kh * run
    int CH;     // maps per block (a chunk of Co), 32, 64 or 128
    int NCH;    // ceil(Co / CH)
    int P, HoWo;
    int nruns;  // ceil(P / 4): runs of four positions
    int cap;    // list entries per wave
    int vec;    // outputs aligned for 4-position vector stores
    int tbits;  // bits of T - 1 (radix passes of the step sort)
    int wchunk; // bytes of one chunk's weight table (multiple of 16)
};

// Weight table of chunk ch: [tap][CH] with tap = ky*run + kx*Ci + c, zero
// for maps past Co, and one zero row at tap = taps.
template <typename WT, bool kHalfIn>
__global__ void k_ev_pack_w(const void *__restrict__ wv, EGeom g, uint8_t *__restrict__ wt)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t per = (int64_t)(g.taps + 1) * g.CH;  // + a zero row
    if (i >= per * g.NCH) return;
    const int ch = (int)(i / per);
    const int r = (int)(i - (int64_t)ch * per);
    const int tap = r / g.CH, cc = r - tap * g.CH;
    const int o = ch * g.CH + cc;
    const int ky = tap / g.run, j = tap - ky * g.run;
    const int kx = j / g.Ci, c = j - kx * g.Ci;
    WT v = (WT)0.0f;
    if (o < g.Co && tap < g.taps) {
        const size_t at = (((size_t)o * g.Ci + c) * g.Kh + ky) * g.Kw + kx;
        if (kHalfIn) v = (WT)reinterpret_cast<const _Float16 *>(wv)[at];
        else v = (WT)reinterpret_cast<const float *>(wv)[at];
    }
    reinterpret_cast<WT *>(wt + (size_t)ch * g.wchunk)[r] = v;
}

// The weights of one table row for this lane's maps, as floats.
template <typename WT, int MPL>
__device__ __forceinline__ void load_row(const WT *row, float (&w)[MPL])
{
    if constexpr (MPL == 2) {
        if constexpr (sizeof(WT) == 2) {
            typedef _Float16 hh2 __attribute__((ext_vector_type(2)));
            const hh2 v = *reinterpret_cast<const hh2 *>(row);
            w[0] = (float)v[0];
            w[1] = (float)v[1];
        } else {
            const float2 v = *reinterpret_cast<const float2 *>(row);
            w[0] = v.x;
            w[1] = v.y;
        }
    } else {
        w[0] = (float)row[0];
    }
}

template <typename WT, int MPL>
__device__ __forceinline__ void add_row(float (&V)[MPL], const WT *row)
{
    float w[MPL];
    load_row<WT, MPL>(row, w);
#pragma unroll
    for (int q = 0; q < MPL; q++) V[q] += w[q];
}

// Raw table words of one row (two halves or one float per map) and their
// accumulation: a half is widened inside a fused multiply-add by 1, which
// rounds once, exactly as the float addition of the widened half.
template <typename WT, int MPL>
struct RowBits {
    typedef typename std::conditional<sizeof(WT) == 2, uint32_t,
                                      typename std::conditional<MPL == 2, float2, float>::type>::type type;
};

template <typename WT, int MPL>
__device__ __forceinline__ typename RowBits<WT, MPL>::type load_bits(const uint8_t *p)
{
    if constexpr (sizeof(WT) == 2) {
        if constexpr (MPL == 2) return *reinterpret_cast<const uint32_t *>(p);
        else return (uint32_t)*reinterpret_cast<const uint16_t *>(p);
    } else {
        return *reinterpret_cast<const typename RowBits<WT, MPL>::type *>(p);
    }
}

template <typename WT, int MPL>
__device__ __forceinline__ void acc_bits(float (&V)[MPL], typename RowBits<WT, MPL>::type b)
{
    if constexpr (sizeof(WT) == 2) {
        typedef _Float16 hh2 __attribute__((ext_vector_type(2)));
        const hh2 h = __builtin_bit_cast(hh2, b);
        V[0] = __builtin_fmaf((float)h[0], 1.0f, V[0]);
        if constexpr (MPL == 2) V[1] = __builtin_fmaf((float)h[1], 1.0f, V[1]);
    } else if constexpr (MPL == 2) {
        V[0] += b.x;
        V[1] += b.y;
    } else {
        V[0] += b;
    }
}

template <int MPL>
__device__ __forceinline__ void fire_check(const float (&V)[MPL], float theta, uint32_t t,
                                           uint32_t (&tf)[MPL], float (&vk)[MPL])
{
#pragma unroll
    for (int q = 0; q < MPL; q++) {
        const bool f = tf[q] == (uint32_t)spk::kNever && V[q] > theta;
        tf[q] = f ? t : tf[q];
        vk[q] = f ? V[q] : vk[q];
    }
}

template <int MPL>
__device__ __forceinline__ bool all_fired(const uint32_t (&tf)[MPL])
{
    bool open = false;
#pragma unroll
    for (int q = 0; q < MPL; q++) open |= tf[q] == (uint32_t)spk::kNever;
    return !__ballot(open);
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t m)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

constexpr int kEvLoads = 16;  // window loads of a position kept in flight

// Load i of a window covers taps [64 * (i % nch), +64) of kernel row
// i / nch.  off: this lane's byte offset from the window origin (0 where the
// lane has no tap, so every load stays inside the window); rowo: the byte
// offset of the lane's tap row in the weight table, -1 where it has none.
template <typename WT>
__device__ __forceinline__ void window_tables(const EGeom &g, int lane, int (&off)[kEvLoads],
                                              int (&rowo)[kEvLoads])
{
#pragma unroll
    for (int i = 0; i < kEvLoads; i++) {
        const int ky = i / g.nch, j = i - ky * g.nch;
        const int k = j * 64 + lane;
        const bool ok = i < g.Kh * g.nch && k < g.run;
        off[i] = ok ? ky * g.rowb + k : 0;
        rowo[i] = ok ? (ky * g.run + k) * g.CH * (int)sizeof(WT) : -1;
    }
}

__device__ __forceinline__ void window_load(const uint8_t *org, const int (&off)[kEvLoads], int nload,
                                            uint32_t (&buf)[kEvLoads])
{
#pragma unroll
    for (int i = 0; i < kEvLoads; i++)
        if (i < nload) buf[i] = org[off[i]];
}

// One output position for this wave's maps.  The spikes of the window are
// compacted into the wave's list as (row << 8 | t), row being the byte
// offset of the spike's tap in the weight table, in tap order.
//  - n <= 64: the list, one entry per lane, is sorted by t with a stable
//    radix sort (ballots and a lane permute per bit); lanes past n hold an
//    entry of the zero row at step 255.  It is walked in order, four table
//    reads in flight, and theta is tested after the last spike of each step.
//  - n <= cap: the steps are walked one by one, each adding its spikes in
//    tap order from up to four 64-entry chunks.
//  - otherwise the window is rescanned once per step.
// Within a step the weights are added in tap order on every path.
template <typename WT, int MPL>
__device__ __forceinline__ void ev_position(const uint8_t *__restrict__ org, bool pf,
                                            const uint32_t (&buf)[kEvLoads],
                                            const int (&rowo)[kEvLoads], const uint8_t *swb,
                                            uint32_t *list, const EGeom &g, int lane, int colb,
                                            float theta, bool test, uint32_t (&tf)[MPL],
                                            float (&vk)[MPL])
{
    float V[MPL];
#pragma unroll
    for (int q = 0; q < MPL; q++) {
        V[q] = 0.0f;
        tf[q] = spk::kNever;
        vk[q] = 0.0f;
    }
    const int rowbytes = g.CH * (int)sizeof(WT);
    int n = 0;
    if (pf) {
        const int nload = g.Kh * g.nch;
#pragma unroll
        for (int i = 0; i < kEvLoads; i++) {
            if (i < nload) {
                const uint32_t t = buf[i];
                const bool act = t < (uint32_t)g.T && rowo[i] >= 0;
                const uint64_t m = __ballot(act);
                int slot = n + (int)lanes_below(m);
                slot = act && slot < g.cap ? slot : g.cap;  // the spare slot
                list[slot] = ((uint32_t)rowo[i] << 8) | t;
                n += __popcll(m);
            }
        }
    } else {
        for (int ky = 0; ky < g.Kh; ky++) {
            const uint8_t *row = org + (size_t)ky * g.rowb;
            for (int j = 0; j < g.nch; j++) {
                const int k = j * 64 + lane;
                const uint32_t t = k < g.run ? (uint32_t)row[k] : 255u;
                const bool act = t < (uint32_t)g.T;
                const uint64_t m = __ballot(act);
                int slot = n + (int)lanes_below(m);
                slot = act && slot < g.cap ? slot : g.cap;
                list[slot] = ((uint32_t)((ky * g.run + k) * rowbytes) << 8) | t;
                n += __popcll(m);
            }
        }
    }
    if (n <= 64) {
        const uint32_t dummy = ((uint32_t)(g.taps * rowbytes) << 8) | 0xFFu;
        uint32_t e = lane < n ? list[lane] : dummy;
        for (int k = 0; k < g.tbits; k++) {
            const bool one = (e >> k) & 1u;
            const uint64_t m0 = __ballot(!one);
            const int dest = one ? __popcll(m0) + (int)lanes_below(~m0) : (int)lanes_below(m0);
            e = (uint32_t)__builtin_amdgcn_ds_permute(dest << 2, (int)e);
        }
        // entries that end a step: the next one has another t
        uint32_t en1 = (uint32_t)__builtin_amdgcn_ds_bpermute(((lane + 1) & 63) << 2, (int)e);
        en1 = lane == 63 ? dummy : en1;
        const uint64_t ends = __ballot((e & 0xFFu) != (en1 & 0xFFu) && (e & 0xFFu) != 0xFFu);
        if (test && theta < 0.0f) {
            const uint32_t t0 = (uint32_t)__builtin_amdgcn_readlane((int)e, 0) & 0xFFu;
            if (t0 != 0) fire_check<MPL>(V, theta, 0u, tf, vk);
        }
        for (int i = 0; i < n; i += 4) {
            uint32_t en[4];
            typename RowBits<WT, MPL>::type w[4];
#pragma unroll
            for (int k = 0; k < 4; k++) {
                en[k] = (uint32_t)__builtin_amdgcn_readlane((int)e, i + k);
                w[k] = load_bits<WT, MPL>(swb + (en[k] >> 8) + colb);
            }
            bool tested = false;
#pragma unroll
            for (int k = 0; k < 4; k++) {
                acc_bits<WT, MPL>(V, w[k]);
                if (test && ((ends >> (i + k)) & 1u)) {
                    fire_check<MPL>(V, theta, en[k] & 0xFFu, tf, vk);
                    tested = true;
                }
            }
            if (tested && all_fired<MPL>(tf)) break;
        }
    } else if (n <= g.cap) {
        const int nc = (n + 63) >> 6;
        uint32_t e[kEvMaxChunks];
#pragma unroll
        for (int c = 0; c < kEvMaxChunks; c++)
            e[c] = (c < nc && c * 64 + lane < n) ? list[c * 64 + lane] : 0xFFFFFFFFu;
        int left = n;
        for (int t = 0; t < g.T && (left > 0 || t == 0); t++) {
            bool any = false;
#pragma unroll
            for (int c = 0; c < kEvMaxChunks; c++) {
                if (c < nc) {
                    uint64_t m = __ballot((e[c] & 0xFFu) == (uint32_t)t);
                    while (m) {
                        const int i = __builtin_ctzll(m);
                        m &= m - 1;
                        const uint32_t ent = (uint32_t)__builtin_amdgcn_readlane((int)e[c], i);
                        add_row<WT, MPL>(V, reinterpret_cast<const WT *>(swb + (ent >> 8) + colb));
                        any = true;
                        left--;
                    }
                }
            }
            if (test && (any || t == 0)) {
                fire_check<MPL>(V, theta, (uint32_t)t, tf, vk);
                if (all_fired<MPL>(tf)) break;
            }
        }
    } else {
        for (int t = 0; t < g.T; t++) {
            bool any = false;
            for (int ky = 0; ky < g.Kh; ky++) {
                const uint8_t *row = org + (size_t)ky * g.rowb;
                for (int j = 0; j < g.nch; j++) {
                    const int k = j * 64 + lane;
                    const uint32_t tt = k < g.run ? (uint32_t)row[k] : 255u;
                    uint64_t m = __ballot(tt == (uint32_t)t);
                    while (m) {
                        const int i = __builtin_ctzll(m);
                        m &= m - 1;
                        const uint32_t ro = (uint32_t)((ky * g.run + j * 64 + i) * rowbytes);
                        add_row<WT, MPL>(V, reinterpret_cast<const WT *>(swb + ro + colb));
                        any = true;
                    }
                }
            }
            if (test && (any || t == 0)) fire_check<MPL>(V, theta, (uint32_t)t, tf, vk);
        }
    }
#pragma unroll
    for (int q = 0; q < MPL; q++) vk[q] = tf[q] == (uint32_t)spk::kNever ? V[q] : vk[q];
}

// Output position p as (sample, row, column), advanced one position at a time.
struct PosIt {
    int b, y, x;
    __device__ void set(const EGeom &g, int p)
    {
        b = p / g.HoWo;
        const int rem = p - b * g.HoWo;
        y = rem / g.Wo;
        x = rem - y * g.Wo;
    }
    __device__ void next(const EGeom &g)
    {
        if (++x == g.Wo) {
            x = 0;
            if (++y == g.Ho) {
                y = 0;
                b++;
            }
        }
    }
    __device__ const uint8_t *origin(const uint8_t *xp, const EGeom &g) const
    {
        return xp + ((size_t)(b * g.Hp + y * g.stride) * g.Wp + x * g.stride) * g.Ci;
    }
};

// Block -> (map chunk, range of position runs); the chunks of a range sit
// on one XCD.  Each wave takes every nwaves-th run of four consecutive
// positions, loads each position's window while the previous one is being
// processed, and writes a map's four results with one store each for the
// times and the potentials.
template <typename WT, int MPL>
__global__ __launch_bounds__(64 * kEvMaxWaves) void k_fire_ev(const uint8_t *__restrict__ xp,
                                                             const uint8_t *__restrict__ wt,
                                                             EGeom g, float theta, int nranges,
                                                             uint8_t *__restrict__ out_t,
                                                             float *__restrict__ out_v)
{
    extern __shared__ __align__(16) uint8_t lds[];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nwaves = blockDim.x >> 6;
    const int xcd = blockIdx.x & 7, q = blockIdx.x >> 3;
    const int ch = q % g.NCH;
    const int range = xcd + 8 * (q / g.NCH);
    if (range >= nranges) return;
    {
        const uint4 *src = reinterpret_cast<const uint4 *>(wt + (size_t)ch * g.wchunk);
        uint4 *dst = reinterpret_cast<uint4 *>(lds);
        for (int i = threadIdx.x; i < g.wchunk / 16; i += blockDim.x) dst[i] = src[i];
    }
    __syncthreads();
    uint32_t *list = reinterpret_cast<uint32_t *>(lds + g.wchunk) + (size_t)wave * (g.cap + 1);
    const int colb = min(lane * MPL, g.CH - MPL) * (int)sizeof(WT);
    const bool test = !(__builtin_isinf(theta) && theta > 0.0f);
    const int r_begin = (int)((long long)range * g.nruns / nranges);
    const int r_end = (int)((long long)(range + 1) * g.nruns / nranges);
    int off[kEvLoads], rowo[kEvLoads];
    window_tables<WT>(g, lane, off, rowo);
    const int nload = g.Kh * g.nch;
    const bool pf = nload <= kEvLoads;
    uint32_t cur[kEvLoads], nxt[kEvLoads];
    int r = r_begin + wave;
    PosIt pos, pn;
    if (r < r_end) {
        pos.set(g, 4 * r);
        if (pf) window_load(pos.origin(xp, g), off, nload, cur);
    }
    for (; r < r_end; r += nwaves) {
        const int p0 = 4 * r;
        const int cnt = min(4, g.P - p0);
        uint32_t tpack[MPL];
        float v4[MPL][4];
#pragma unroll
        for (int mq = 0; mq < MPL; mq++) {
            tpack[mq] = 0u;
#pragma unroll
            for (int k = 0; k < 4; k++) v4[mq][k] = 0.0f;
        }
#pragma unroll 1
        for (int k = 0; k < cnt; k++) {
            // the next position of this wave: the following one, or the
            // first of its next run
            const bool last = k == cnt - 1;
            const bool more = !last || r + nwaves < r_end;
            if (more) {
                pn = pos;
                if (!last) pn.next(g);
                else pn.set(g, 4 * (r + nwaves));
                if (pf) window_load(pn.origin(xp, g), off, nload, nxt);
            }
            uint32_t tf[MPL];
            float vk[MPL];
            ev_position<WT, MPL>(pos.origin(xp, g), pf, cur, rowo, lds, list, g, lane, colb, theta,
                                 test, tf, vk);
#pragma unroll
            for (int mq = 0; mq < MPL; mq++) {
                tpack[mq] |= tf[mq] << (8 * k);
#pragma unroll
                for (int kk = 0; kk < 4; kk++) v4[mq][kk] = kk == k ? vk[mq] : v4[mq][kk];
            }
            if (more) {
                pos = pn;
#pragma unroll
                for (int i = 0; i < kEvLoads; i++) cur[i] = nxt[i];
            }
        }
        const int b0 = p0 / g.HoWo, rem0 = p0 - b0 * g.HoWo;
#pragma unroll
        for (int mq = 0; mq < MPL; mq++) {
            const int cc = lane * MPL + mq;
            const int o = ch * g.CH + cc;
            if (cc >= g.CH || o >= g.Co) continue;
            if (g.vec && cnt == 4) {
                const size_t at = ((size_t)b0 * g.Co + o) * g.HoWo + rem0;
                *reinterpret_cast<uint32_t *>(out_t + at) = tpack[mq];
                *reinterpret_cast<float4 *>(out_v + at) =
                    make_float4(v4[mq][0], v4[mq][1], v4[mq][2], v4[mq][3]);
            } else {
                for (int k = 0; k < cnt; k++) {
                    const int p = p0 + k;
                    const int b = p / g.HoWo, rem = p - b * g.HoWo;
                    const size_t at = ((size_t)b * g.Co + o) * g.HoWo + rem;
                    out_t[at] = (uint8_t)(tpack[mq] >> (8 * k));
                    out_v[at] = k == 0 ? v4[mq][0] : k == 1 ? v4[mq][1] : k == 2 ? v4[mq][2] : v4[mq][3];
                }
            }
        }
    }
}

int device_attr(hipDeviceAttribute_t a, int dflt)
{
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess && hipDeviceGetAttribute(&v, a, dev) == hipSuccess && v > 0)
        return v;
    return dflt;
}

int ev_cus() { static const int n = device_attr(hipDeviceAttributeMultiprocessorCount, 256); return n; }
int ev_lds_block()
{
    static const int n = device_attr(hipDeviceAttributeMaxSharedMemoryPerBlock, 65536);
    return n;
}
int ev_lds_cu()
{
    static const int n = device_attr(hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, 65536);
    return n;
}

// Geometry, block shape and LDS of a sparse conv; false if its weight table
// does not leave room for a list of 64 spikes per wave.
bool ev_plan(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw, int stride, int pad,
             bool half_w, EGeom &g, int &waves, size_t &lds)
{
    g = EGeom{};
    g.B = B; g.T = T; g.Ci = Ci; g.Hi = Hi; g.Wi = Wi; g.Co = Co; g.Kh = Kh; g.Kw = Kw;
    g.stride = stride; g.pad = pad;
    g.Ho = (Hi + 2 * pad - Kh) / stride + 1;
    g.Wo = (Wi + 2 * pad - Kw) / stride + 1;
    g.Hp = Hi + 2 * pad;
    g.Wp = Wi + 2 * pad;
    g.rowb = g.Wp * Ci;
    g.run = Kw * Ci;
    g.nch = (g.run + 63) / 64;
    g.taps = Kh * g.run;
    g.HoWo = g.Ho * g.Wo;
    g.P = B * g.HoWo;
    g.nruns = (g.P + 3) / 4;
    g.tbits = 0;
    while ((1 << g.tbits) < T) g.tbits++;
    const int wb = half_w ? 2 : 4;
    const int lds_max = ev_lds_block();
    for (int CH : {128, 64, 32}) {
        if (CH > 32 && Co <= CH / 2) continue;  // a smaller chunk holds every map
        g.CH = CH;
        g.NCH = (Co + CH - 1) / CH;
        g.wchunk = (int)spk::align_up((size_t)(g.taps + 1) * CH * wb, 16);
        for (int wv : {kEvMaxWaves, 8}) {
            long long room = (long long)lds_max - g.wchunk;
            int cap = room > 0 ? (int)std::min<long long>(64 * kEvMaxChunks, (room / (wv * 4) - 1) / 64 * 64) : 0;
            if (cap >= 64) {
                g.cap = cap;
                waves = wv;
                lds = (size_t)g.wchunk + (size_t)wv * (cap + 1) * 4;
                return true;
            }
        }
    }
    return false;
}

size_t ev_xp_bytes(const EGeom &g)
{
    return spk::align_up((size_t)g.B * g.Hp * g.rowb + kEvSlack, 256);
}

template <typename WT, int MPL>
void launch_ev(dim3 grid, dim3 block, size_t lds, hipStream_t s, const uint8_t *xp,
               const uint8_t *wt, const EGeom &g, float theta, int nranges, uint8_t *ot, float *ov)
{
    hipLaunchKernelGGL((k_fire_ev<WT, MPL>), grid, block, lds, s, xp, wt, g, theta, nranges, ot, ov);
}

}  // namespace

// ------------------------------------------------------------------ ABI

extern "C" size_t spk_times_to_spikes_workspace_size(int B, int C, int H, int W, int T)
{
    if (B < 1 || C < 1 || H < 1 || W < 1 || T < 1 || T > SPK_MAX_T) return 0;
    const int64_t n = (int64_t)C * H * W;
    const int nb = (int)std::max<int64_t>(1, std::min<int64_t>((n + 16383) / 16384,
                                                               8192 / ((int64_t)kCvWaves * T)));
    return spk::align_up((size_t)B * nb * kCvWaves * T * sizeof(int32_t), 256);
}

extern "C" spk_status spk_times_to_spikes(const uint8_t *times, int B, int C, int H, int W, int T,
                                          int cap, uint32_t *spikes, int32_t *offsets, void *ws,
                                          size_t ws_bytes, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(times && offsets && (spikes || cap == 0) && ws, SPK_E_ARG,
                "spk_times_to_spikes: NULL pointer");
    SPK_REQUIRE(B > 0 && C > 0 && H > 0 && W > 0 && cap >= 0, SPK_E_ARG,
                "spk_times_to_spikes: sizes must be positive (cap >= 0)");
    SPK_REQUIRE(T >= 1 && T <= SPK_MAX_T, SPK_E_SHAPE, "spk_times_to_spikes: T=%d not in [1, %d]",
                T, SPK_MAX_T);
    const int64_t n = (int64_t)C * H * W;
    SPK_REQUIRE(n < (1ll << 31), SPK_E_SHAPE, "spk_times_to_spikes: C*H*W >= 2^31");
    const size_t need = spk_times_to_spikes_workspace_size(B, C, H, W, T);
    SPK_REQUIRE(ws_bytes >= need, SPK_E_WORKSPACE, "spk_times_to_spikes: workspace %zu < %zu bytes",
                ws_bytes, need);
    SPK_REQUIRE_WS_ALIGNED(ws, "spk_times_to_spikes");
    SPK_REQUIRE(B <= 65535, SPK_E_SHAPE, "spk_times_to_spikes: B=%d > 65535", B);
    const int nb = (int)std::max<int64_t>(1, std::min<int64_t>((n + 16383) / 16384,
                                                               8192 / ((int64_t)kCvWaves * T)));
    const int nq = nb * kCvWaves;
    int tbits = 0;
    while ((1 << tbits) < T) tbits++;
    int32_t *cnt = static_cast<int32_t *>(ws);
    hipStream_t s = spk::stream_of(stream);
    hipLaunchKernelGGL(k_list_count, dim3(nb, B), dim3(kCvThreads), (size_t)kCvWaves * T * 4, s,
                       times, n, T, nb, cnt);
    hipLaunchKernelGGL(k_list_scan, dim3(B), dim3(256), ((size_t)nq * T + T) * 4, s, cnt, T, nq,
                       offsets);
    if (cap > 0)
        hipLaunchKernelGGL(k_list_scatter, dim3(nb, B), dim3(kCvThreads), (size_t)kCvWaves * T * 4,
                           s, times, n, T, tbits, nb, cnt, cap, spikes);
    SPK_LAUNCHED("spk_times_to_spikes");
    return SPK_OK;
}

extern "C" spk_status spk_spikes_to_times(const uint32_t *spikes, const int32_t *offsets, int cap,
                                          int B, int C, int H, int W, int T, uint8_t *times,
                                          spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(offsets && times && (spikes || cap == 0), SPK_E_ARG,
                "spk_spikes_to_times: NULL pointer");
    SPK_REQUIRE(B > 0 && C > 0 && H > 0 && W > 0 && cap >= 0, SPK_E_ARG,
                "spk_spikes_to_times: sizes must be positive (cap >= 0)");
    SPK_REQUIRE(T >= 1 && T <= SPK_MAX_T, SPK_E_SHAPE, "spk_spikes_to_times: T=%d not in [1, %d]",
                T, SPK_MAX_T);
    const int64_t n = (int64_t)C * H * W;
    SPK_REQUIRE(n < (1ll << 31), SPK_E_SHAPE, "spk_spikes_to_times: C*H*W >= 2^31");
    SPK_REQUIRE(B <= 65535, SPK_E_SHAPE, "spk_spikes_to_times: B=%d > 65535", B);
    hipStream_t s = spk::stream_of(stream);
    const size_t total = (size_t)B * n;
    hipLaunchKernelGGL(k_fill_u8, dim3((unsigned)std::min<size_t>(4096, (total / 16 + 255) / 256 + 1)),
                       dim3(256), 0, s, times, total, (uint8_t)spk::kNever);
    if (cap > 0)
        hipLaunchKernelGGL(k_list_place, dim3(std::min(64, (cap + 4095) / 4096), B), dim3(256), 0, s,
                           spikes, offsets, cap, B, T, C, H, W, -1, times);
    SPK_LAUNCHED("spk_spikes_to_times");
    return SPK_OK;
}

extern "C" size_t spk_conv_fire_sparse_workspace_size(int B, int T, int Ci, int Hi, int Wi, int Co,
                                                      int Kh, int Kw, int stride, int pad,
                                                      spk_dtype w_dtype)
{
    if (B < 1 || T < 1 || Ci < 1 || Hi < 1 || Wi < 1 || Co < 1 || Kh < 1 || Kw < 1 || stride < 1 ||
        pad < 0 || Hi + 2 * pad < Kh || Wi + 2 * pad < Kw)
        return 0;
    EGeom g;
    int waves;
    size_t lds;
    if (!ev_plan(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, w_dtype == SPK_F16, g, waves, lds))
        return 0;
    return ev_xp_bytes(g) + spk::align_up((size_t)g.NCH * g.wchunk, 256);
}

extern "C" spk_status spk_conv_fire_sparse(const uint32_t *spikes, const int32_t *offsets, int cap,
                                           int B, int T, int Ci, int Hi, int Wi, const void *w,
                                           spk_dtype w_dtype, int Co, int Kh, int Kw, int stride,
                                           int pad, float theta, uint8_t *out_times,
                                           float *out_vkey, void *ws, size_t ws_bytes,
                                           spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(offsets && w && out_times && out_vkey && ws && (spikes || cap == 0), SPK_E_ARG,
                "spk_conv_fire_sparse: NULL pointer");
    SPK_REQUIRE(B > 0 && Ci > 0 && Hi > 0 && Wi > 0 && Co > 0 && Kh > 0 && Kw > 0 && stride > 0 &&
                    pad >= 0 && cap >= 0,
                SPK_E_ARG, "spk_conv_fire_sparse: sizes must be positive (pad, cap >= 0)");
    SPK_REQUIRE(T >= 1 && T <= SPK_MAX_T, SPK_E_SHAPE, "spk_conv_fire_sparse: T=%d not in [1, %d]",
                T, SPK_MAX_T);
    SPK_REQUIRE(w_dtype == SPK_F32 || w_dtype == SPK_F16, SPK_E_UNSUPPORTED,
                "spk_conv_fire_sparse: unknown weight dtype %d", (int)w_dtype);
    SPK_REQUIRE(!__builtin_isnan(theta), SPK_E_ARG, "spk_conv_fire_sparse: theta is NaN");
    const int Ho = spk_out_extent(Hi, Kh, stride, pad), Wo = spk_out_extent(Wi, Kw, stride, pad);
    SPK_REQUIRE(Ho > 0 && Wo > 0, SPK_E_SHAPE, "spk_conv_fire_sparse: empty output (%d x %d)", Ho,
                Wo);
    SPK_REQUIRE((long long)Ci * Hi * Wi < (1ll << 31) && (long long)B * Co * Ho * Wo < (1ll << 31),
                SPK_E_SHAPE, "spk_conv_fire_sparse: tensor of 2^31 elements or more");
    SPK_REQUIRE((long long)B * (Hi + 2 * pad) * (Wi + 2 * pad) * Ci < (1ll << 40), SPK_E_SHAPE,
                "spk_conv_fire_sparse: padded input too large");
    SPK_REQUIRE(B <= 65535, SPK_E_SHAPE, "spk_conv_fire_sparse: B=%d > 65535", B);
    EGeom g;
    int waves;
    size_t lds;
    const bool half_w = w_dtype == SPK_F16;
    SPK_REQUIRE(ev_plan(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, half_w, g, waves, lds),
                SPK_E_UNSUPPORTED,
                "spk_conv_fire_sparse: weight table of %d taps does not fit LDS", Kh * Kw * Ci);
    SPK_REQUIRE(Kh * Kw * Ci < (1 << 24), SPK_E_SHAPE, "spk_conv_fire_sparse: window too large");
    const size_t need = ev_xp_bytes(g) + spk::align_up((size_t)g.NCH * g.wchunk, 256);
    SPK_REQUIRE(ws_bytes >= need, SPK_E_WORKSPACE, "spk_conv_fire_sparse: workspace %zu < %zu bytes",
                ws_bytes, need);
    SPK_REQUIRE_WS_ALIGNED(ws, "spk_conv_fire_sparse");
    g.vec = (g.HoWo % 4 == 0) && ((uintptr_t)out_times % 4 == 0) && ((uintptr_t)out_vkey % 16 == 0);
    uint8_t *xp = static_cast<uint8_t *>(ws);
    uint8_t *wt = xp + ev_xp_bytes(g);
    hipStream_t s = spk::stream_of(stream);
    // padded channels-last time buffer: all "never" (T), then the stored spikes
    const size_t xb = ev_xp_bytes(g);
    hipLaunchKernelGGL(k_fill_u8, dim3((unsigned)std::min<size_t>(4096, (xb / 16 + 255) / 256 + 1)),
                       dim3(256), 0, s, xp, xb, (uint8_t)T);
    if (cap > 0)
        hipLaunchKernelGGL(k_list_place, dim3(std::min(64, (cap + 4095) / 4096), B), dim3(256), 0, s,
                           spikes, offsets, cap, B, T, Ci, Hi, Wi, pad, xp);
    const int64_t nw = (int64_t)g.NCH * (g.taps + 1) * g.CH;
    if (half_w)
        hipLaunchKernelGGL((k_ev_pack_w<_Float16, true>), dim3((unsigned)((nw + 255) / 256)), dim3(256),
                           0, s, w, g, wt);
    else
        hipLaunchKernelGGL((k_ev_pack_w<float, false>), dim3((unsigned)((nw + 255) / 256)), dim3(256), 0,
                           s, w, g, wt);
    // blocks: as many as fit the CUs (by LDS and threads), split over chunks
    const int per_cu = std::max(1, std::min(2048 / (64 * waves), ev_lds_cu() / (int)lds));
    int nranges = std::max(1, ev_cus() * per_cu / g.NCH);
    nranges = std::min(nranges, g.nruns);
    const int q = g.NCH * ((nranges + 7) / 8);
    const dim3 grid(8 * q), block(64 * waves);
    const bool mpl2 = g.CH == 128;
    if (half_w) {
        if (mpl2) launch_ev<_Float16, 2>(grid, block, lds, s, xp, wt, g, theta, nranges, out_times, out_vkey);
        else launch_ev<_Float16, 1>(grid, block, lds, s, xp, wt, g, theta, nranges, out_times, out_vkey);
    } else {
        if (mpl2) launch_ev<float, 2>(grid, block, lds, s, xp, wt, g, theta, nranges, out_times, out_vkey);
        else launch_ev<float, 1>(grid, block, lds, s, xp, wt, g, theta, nranges, out_times, out_vkey);
    }
    SPK_LAUNCHED("spk_conv_fire_sparse");
    return SPK_OK;
}
