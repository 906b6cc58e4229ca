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

// One thread per (sample, stored spike): writes its step at its neuron of
// the B x C x H x W time map (dst_pad < 0) or of the padded channels-last
// buffer [b][y + pad][x + pad][c] (dst_pad >= 0).
__global__ void k_list_place(const uint32_t *__restrict__ spikes, const int32_t *__restrict__ offsets,
                             int cap, int B, int T, int C, int H, int W, int dst_pad,
                             uint8_t *__restrict__ dst)
{
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= (int64_t)B * cap) return;
    const int b = (int)(g / cap);
    const int32_t j = (int32_t)(g - (int64_t)b * cap);
    const int32_t *ob = offsets + (size_t)b * (T + 1);
    if (j >= ob[T]) return;
    const uint32_t idx = spikes[g];
    const int64_t n = (int64_t)C * H * W;
    if ((int64_t)idx >= n) return;
    const uint8_t t = (uint8_t)step_of(ob, T, j);
    if (dst_pad < 0) {
        dst[(size_t)b * n + idx] = t;
        return;
    }
    const int c = (int)(idx / (uint32_t)(H * W));
    const int r = (int)(idx - (uint32_t)c * H * W);
    const int y = r / W, x = r - y * W;
    const int Hp = H + 2 * dst_pad, Wp = W + 2 * dst_pad;
    dst[(((size_t)b * Hp + y + dst_pad) * Wp + x + dst_pad) * C + c] = t;
}

// ------------------------------------------------------------ event conv

constexpr int kEvMaxWaves = 16;
constexpr int kEvMaxChunks = 16;  // list capacity per wave <= 64 * this
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
    int wchunk; // bytes of one chunk's weight table (multiple of 16)
};

// Weight table of chunk ch: [tap][CH] with tap = ky*run + kx*Ci + c, zero
// for maps past Co.
template <typename WT, bool kHalfIn>
__global__ void k_ev_pack_w(const void *__restrict__ wv, EGeom g, uint8_t *__restrict__ wt)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t per = (int64_t)g.taps * g.CH;
    if (i >= per * g.NCH) return;
    const int ch = (int)(i / per);
    const int r = (int)(i - (int64_t)ch * per);
    const int tap = r / g.CH, cc = r - tap * g.CH;
    const int o = ch * g.CH + cc;
    const int ky = tap / g.run, j = tap - ky * g.run;
    const int kx = j / g.Ci, c = j - kx * g.Ci;
    WT v = (WT)0.0f;
    if (o < g.Co) {
        const size_t at = (((size_t)o * g.Ci + c) * g.Kh + ky) * g.Kw + kx;
        if (kHalfIn) v = (WT)reinterpret_cast<const _Float16 *>(wv)[at];
        else v = (WT)reinterpret_cast<const float *>(wv)[at];
    }
    reinterpret_cast<WT *>(wt + (size_t)ch * g.wchunk)[r] = v;
}

template <typename WT, int MPL>
__device__ __forceinline__ void add_row(float (&V)[MPL], const WT *row)
{
    if constexpr (MPL == 2) {
        if constexpr (sizeof(WT) == 2) {
            typedef _Float16 hh2 __attribute__((ext_vector_type(2)));
            const hh2 w = *reinterpret_cast<const hh2 *>(row);
            V[0] += (float)w[0];
            V[1] += (float)w[1];
        } else {
            const float2 w = *reinterpret_cast<const float2 *>(row);
            V[0] += w.x;
            V[1] += w.y;
        }
    } else {
        V[0] += (float)row[0];
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

// One output position for this wave's maps: compact the spikes of the
// window into the wave's list (tap << 8 | t, in tap order), then walk the
// steps; each step adds the weights of its spikes in tap order and, if it
// brought any (or is step 0), tests theta.  A window with more spikes than
// the list holds is walked by rescanning it once per step.
template <typename WT, int MPL>
__device__ __forceinline__ void ev_position(const uint8_t *__restrict__ xp, const WT *sw,
                                            uint32_t *list, const EGeom &g, int p, int lane,
                                            int col, float theta, bool readout,
                                            uint32_t (&tf)[MPL], float (&vk)[MPL])
{
    const int b = p / g.HoWo, rem = p - b * g.HoWo;
    const int y = rem / g.Wo, x = rem - y * g.Wo;
    const uint8_t *org = xp + ((size_t)(b * g.Hp + y * g.stride) * g.Wp + x * g.stride) * g.Ci;
    float V[MPL];
#pragma unroll
    for (int q = 0; q < MPL; q++) {
        V[q] = 0.0f;
        tf[q] = spk::kNever;
        vk[q] = 0.0f;
    }
    int n = 0;
    for (int ky = 0; ky < g.Kh; ky++) {
        const uint8_t *row = org + (size_t)ky * g.rowb;
        for (int j = 0; j < g.nch; j++) {
            const int k = j * 64 + lane;
            const uint32_t t = k < g.run ? (uint32_t)row[k] : 255u;
            const bool act = t < (uint32_t)g.T;
            const uint64_t m = __ballot(act);
            if (m) {
                const int slot = n + (int)__builtin_amdgcn_mbcnt_hi(
                                         (uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
                if (act && slot < g.cap) list[slot] = ((uint32_t)(ky * g.run + k) << 8) | t;
                n += __popcll(m);
            }
        }
    }
    if (n <= g.cap) {
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
                        add_row<WT, MPL>(V, sw + (size_t)(ent >> 8) * g.CH + col);
                        any = true;
                        left--;
                    }
                }
            }
            if (!readout && (any || t == 0)) {
                fire_check<MPL>(V, theta, (uint32_t)t, tf, vk);
                bool open = false;
#pragma unroll
                for (int q = 0; q < MPL; q++) open |= tf[q] == (uint32_t)spk::kNever;
                if (!__ballot(open)) break;
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
                        add_row<WT, MPL>(V, sw + (size_t)(ky * g.run + j * 64 + i) * g.CH + col);
                        any = true;
                    }
                }
            }
            if (!readout && (any || t == 0)) fire_check<MPL>(V, theta, (uint32_t)t, tf, vk);
        }
    }
#pragma unroll
    for (int q = 0; q < MPL; q++) vk[q] = tf[q] == (uint32_t)spk::kNever ? V[q] : vk[q];
}

// Block -> (map chunk, range of position runs); the chunks of a range sit
// on one XCD.  Each wave takes every nwaves-th run of four consecutive
// positions and writes a map's four results with one store each for the
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
    const WT *sw = reinterpret_cast<const WT *>(lds);
    uint32_t *list = reinterpret_cast<uint32_t *>(lds + g.wchunk) + (size_t)wave * g.cap;
    const int col = min(lane * MPL, g.CH - MPL);
    const bool readout = __builtin_isinf(theta) && theta > 0.0f;
    const int r_begin = (int)((long long)range * g.nruns / nranges);
    const int r_end = (int)((long long)(range + 1) * g.nruns / nranges);
    for (int r = r_begin + wave; r < r_end; r += nwaves) {
        const int p0 = 4 * r;
        uint32_t tf[4][MPL];
        float vk[4][MPL];
#pragma unroll
        for (int k = 0; k < 4; k++) {
            if (p0 + k < g.P)
                ev_position<WT, MPL>(xp, sw, list, g, p0 + k, lane, col, theta, readout, tf[k], vk[k]);
        }
#pragma unroll
        for (int mq = 0; mq < MPL; mq++) {
            const int cc = lane * MPL + mq;
            const int o = ch * g.CH + cc;
            if (cc >= g.CH || o >= g.Co) continue;
            const int b0 = p0 / g.HoWo, rem0 = p0 - b0 * g.HoWo;
            if (g.vec && p0 + 3 < g.P) {
                const size_t at = ((size_t)b0 * g.Co + o) * g.HoWo + rem0;
                *reinterpret_cast<uint32_t *>(out_t + at) =
                    tf[0][mq] | (tf[1][mq] << 8) | (tf[2][mq] << 16) | (tf[3][mq] << 24);
                *reinterpret_cast<float4 *>(out_v + at) =
                    make_float4(vk[0][mq], vk[1][mq], vk[2][mq], vk[3][mq]);
            } else {
#pragma unroll
                for (int k = 0; k < 4; k++) {
                    const int p = p0 + k;
                    if (p >= g.P) break;
                    const int b = p / g.HoWo, rem = p - b * g.HoWo;
                    const size_t at = ((size_t)b * g.Co + o) * g.HoWo + rem;
                    out_t[at] = (uint8_t)tf[k][mq];
                    out_v[at] = vk[k][mq];
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
    const int wb = half_w ? 2 : 4;
    const int lds_max = ev_lds_block();
    for (int CH : {128, 64, 32}) {
        if (CH > 32 && Co <= CH / 2) continue;  // a smaller chunk holds every map
        g.CH = CH;
        g.NCH = (Co + CH - 1) / CH;
        g.wchunk = (int)spk::align_up((size_t)g.taps * CH * wb, 16);
        for (int wv : {kEvMaxWaves, 8}) {
            long long room = (long long)lds_max - g.wchunk;
            int cap = room > 0 ? (int)std::min<long long>(64 * kEvMaxChunks, room / (wv * 4) / 64 * 64) : 0;
            if (cap >= 64) {
                g.cap = cap;
                waves = wv;
                lds = (size_t)g.wchunk + (size_t)wv * cap * 4;
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
    hipStream_t s = spk::stream_of(stream);
    const size_t total = (size_t)B * n;
    hipLaunchKernelGGL(k_fill_u8, dim3((unsigned)std::min<size_t>(4096, (total / 16 + 255) / 256 + 1)),
                       dim3(256), 0, s, times, total, (uint8_t)spk::kNever);
    const int64_t nthreads = (int64_t)B * cap;
    if (nthreads > 0)
        hipLaunchKernelGGL(k_list_place, dim3((unsigned)((nthreads + 255) / 256)), dim3(256), 0, s,
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
    g.vec = (g.HoWo % 4 == 0) && ((uintptr_t)out_times % 4 == 0) && ((uintptr_t)out_vkey % 16 == 0);
    uint8_t *xp = static_cast<uint8_t *>(ws);
    uint8_t *wt = xp + ev_xp_bytes(g);
    hipStream_t s = spk::stream_of(stream);
    // padded channels-last time buffer: all "never" (T), then the stored spikes
    const size_t xb = ev_xp_bytes(g);
    hipLaunchKernelGGL(k_fill_u8, dim3((unsigned)std::min<size_t>(4096, (xb / 16 + 255) / 256 + 1)),
                       dim3(256), 0, s, xp, xb, (uint8_t)T);
    const int64_t nthreads = (int64_t)B * cap;
    if (nthreads > 0)
        hipLaunchKernelGGL(k_list_place, dim3((unsigned)((nthreads + 255) / 256)), dim3(256), 0, s,
                           spikes, offsets, cap, B, T, Ci, Hi, Wi, pad, xp);
    const int64_t nw = (int64_t)g.NCH * g.taps * g.CH;
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
