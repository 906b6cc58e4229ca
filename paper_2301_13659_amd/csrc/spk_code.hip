// spk_latency_code: rank-order latency coding (Spyker §II-D.2, §II-D.3).
//
// Ranking uses one 64-bit key per value: the high word maps the float to an
// unsigned integer whose ascending order is descending value order, the low
// word is the flat index inside the sample.  Keys are unique, so any sort of
// them is the stable "value descending, index ascending" order, and the rank
// of an eligible value is its position among the sorted keys.  Ineligible
// values (<= min_value, NaN) get the all-ones key, sort to the end and are
// written as never firing up front.
//
//  - Samples of up to kSmall values are ranked by one workgroup each: the
//    eligible keys are counted into buckets of their value word, a prefix sum
//    of the counts gives each bucket's first rank and a scan of its members
//    the rest.  Samples with a crowded bucket are sorted instead: every
//    thread sorts 8 keys in registers, then merge levels in LDS merge the
//    runs (no padding to a power of two).
//  - Larger samples: no sort.  Only the keys at the T - 1 ranks where the
//    step changes are needed; they are selected with a histogram of the top
//    key bits and a radix selection inside the buckets that hold them, and
//    every value then counts the boundary keys at or below its own (see
//    below).  The working arrays live in the caller workspace.
#include <cstring>

#include "spk_dog.h"
#include "spk_internal.h"

namespace {

constexpr int kSmall = 8192;    // keys per LDS sort (2 x 64 KB)
constexpr int kThreads = 1024;
constexpr uint64_t kDead = ~0ull;

__device__ __forceinline__ uint32_t order_desc(float v)
{
    if (v == 0.0f) v = 0.0f;  // -0 and +0 are one value
    uint32_t u = __float_as_uint(v);
    uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);  // ascending float order
    return ~asc;
}

__device__ __forceinline__ uint64_t make_key(float v, float min_value, uint32_t i)
{
    return (v > min_value) ? (((uint64_t)order_desc(v) << 32) | i) : kDead;
}

__device__ __forceinline__ int block_sum(int v, int *red)
{
    for (int o = 32; o > 0; o >>= 1) v += __shfl_down(v, o, 64);
    int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    if (lane == 0) red[wid] = v;
    __syncthreads();
    int tot = 0;
    if (threadIdx.x == 0) {
        for (int w = 0; w < (int)(blockDim.x >> 6); w++) tot += red[w];
        red[0] = tot;
    }
    __syncthreads();
    tot = red[0];
    __syncthreads();
    return tot;
}

// Exclusive prefix sum of v over the block in thread order; total gets the sum.
__device__ __forceinline__ int block_exclusive_scan(int v, int *red, int &total)
{
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    int s = v;
    for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(s, o, 64);
        if (lane >= o) s += t;
    }
    if (lane == 63) red[wid] = s;
    __syncthreads();
    int before = 0, tot = 0;
    for (int w = 0; w < (int)(blockDim.x >> 6); w++) {
        const int c = red[w];
        before += w < wid ? c : 0;
        tot += c;
    }
    __syncthreads();
    total = tot;
    return before + s - v;
}

// Sort 8 keys held by one thread (ascending), a fixed compare-exchange network.
__device__ __forceinline__ void cswap(uint64_t &a, uint64_t &b)
{
    const uint64_t lo = a < b ? a : b, hi = a < b ? b : a;
    a = lo;
    b = hi;
}

__device__ __forceinline__ void sort8(uint64_t *k)
{
    // Batcher's odd-even merge sort for 8 elements (19 exchanges)
    cswap(k[0], k[1]); cswap(k[2], k[3]); cswap(k[4], k[5]); cswap(k[6], k[7]);
    cswap(k[0], k[2]); cswap(k[1], k[3]); cswap(k[4], k[6]); cswap(k[5], k[7]);
    cswap(k[1], k[2]); cswap(k[5], k[6]);
    cswap(k[0], k[4]); cswap(k[1], k[5]); cswap(k[2], k[6]); cswap(k[3], k[7]);
    cswap(k[2], k[4]); cswap(k[3], k[5]);
    cswap(k[1], k[2]); cswap(k[3], k[4]); cswap(k[5], k[6]);
}

// Merge runs of `width` sorted keys pairwise (src -> dst, n keys), one key
// per thread at a time: a key's place in the merged run is its place in its
// own run plus the number of keys below it in the other run (keys are unique),
// found by binary search.
__device__ void merge_level_rank(const uint64_t *src, uint64_t *dst, int n, int width)
{
    for (int e = threadIdx.x; e < n; e += blockDim.x) {
        const int lo = (e / (2 * width)) * 2 * width;
        const int na = min(width, n - lo), nb = max(0, min(width, n - lo - width));
        const uint64_t key = src[e];
        const bool in_a = e < lo + na;
        const uint64_t *other = in_a ? src + lo + na : src + lo;
        int l = 0, h = in_a ? nb : na;
        while (l < h) {
            const int mid = (l + h) >> 1;
            if (other[mid] < key) l = mid + 1;
            else h = mid;
        }
        dst[lo + (in_a ? e - lo : e - lo - na) + l] = key;
    }
}

// Sorts the N compacted keys of one sample held in src (dst: a second buffer
// of N keys) and writes each one's step: register sort of 8 per thread, then
// LDS merge levels by rank; rank r of the N sorted keys fires at r*T/N.
__device__ void sort_and_time(uint64_t *src, uint64_t *dst, int N, int T, uint8_t *__restrict__ ts)
{
    const int first = threadIdx.x * 8;
    uint64_t k8[8];
    if (first < N) {
#pragma unroll
        for (int j = 0; j < 8; j++) k8[j] = first + j < N ? src[first + j] : kDead;
        sort8(k8);
#pragma unroll
        for (int j = 0; j < 8; j++)
            if (first + j < N) src[first + j] = k8[j];
    }
    __syncthreads();
    for (int width = 8; width < N; width *= 2) {
        merge_level_rank(src, dst, N, width);
        __syncthreads();
        uint64_t *t = src;
        src = dst;
        dst = t;
    }
    for (int r = threadIdx.x; r < N; r += blockDim.x)
        ts[(uint32_t)src[r]] = (uint8_t)(((long long)r * T) / N);
}

// Whole sample in one workgroup, ranked by bucketing.  A key's rank is the
// number of eligible keys below it: the keys whose value word lies in a lower
// bucket, plus those of its own bucket that are smaller.  Buckets split the
// sample's span of value words [lo, hi] into kBk equal runs of 2^sh words
// (a monotone map), so the first term is a prefix sum of the bucket counts
// and the second a scan of the bucket's members once the keys are scattered
// in bucket order.  When a bucket holds more than kBkMax keys (many equal or
// nearly equal values) the scattered keys are sorted instead.  n <= 8 * blockDim.
constexpr int kBk = 4096;
constexpr int kBkMax = 96;

// The ranks of one sample whose values thread tid holds in xv[j] (flat index
// tid + kThreads * j, for those below n), written to ts.  keys: 2 * n keys of
// dynamic LDS; cnt, red, mm: the kernel's static LDS.
__device__ __forceinline__ void bucket_code(const float (&xv)[8], int n, int T, float min_value,
                                            uint8_t *__restrict__ ts, uint64_t *keys, int *cnt,
                                            int *red, uint32_t *mm)
{
    const int tid = threadIdx.x, lane = tid & 63;
    for (int e = tid; e <= kBk; e += kThreads) cnt[e] = 0;
    if (tid == 0) {
        mm[0] = ~0u;
        mm[1] = 0u;
        mm[2] = 0u;
    }
    uint64_t k8[8];
    uint32_t lo = ~0u, hi = 0u;
#pragma unroll
    for (int j = 0; j < 8; j++) {
        const int i = tid + kThreads * j;
        uint64_t key = kDead;
        if (i < n) {
            key = make_key(xv[j], min_value, (uint32_t)i);
            if (key == kDead) {
                ts[i] = spk::kNever;
            } else {
                lo = min(lo, (uint32_t)(key >> 32));
                hi = max(hi, (uint32_t)(key >> 32));
            }
        }
        k8[j] = key;
    }
    for (int o = 32; o > 0; o >>= 1) {
        lo = min(lo, (uint32_t)__shfl_xor((int)lo, o, 64));
        hi = max(hi, (uint32_t)__shfl_xor((int)hi, o, 64));
    }
    __syncthreads();  // counts and mm initialised
    if (lane == 0) {
        atomicMin(&mm[0], lo);
        atomicMax(&mm[1], hi);
    }
    __syncthreads();
    const uint32_t w0 = mm[0], w1 = mm[1];
    if (w0 > w1) return;  // no eligible value (uniform over the block)
    const uint32_t span = w1 - w0;
    const int sh = (span >> 12) == 0u ? 0 : 32 - __clz((int)span) - 12;  // (span >> sh) < kBk
    int bk[8], slot[8];
#pragma unroll
    for (int j = 0; j < 8; j++) {
        bk[j] = 0;
        slot[j] = 0;
        if (k8[j] != kDead) {
            bk[j] = (int)(((uint32_t)(k8[j] >> 32) - w0) >> sh);
            slot[j] = atomicAdd(&cnt[bk[j]], 1);
        }
    }
    __syncthreads();
    // exclusive prefix sum of the counts (4 consecutive buckets per thread)
    int c4[4], sum = 0, big = 0;
#pragma unroll
    for (int q = 0; q < 4; q++) {
        c4[q] = cnt[4 * tid + q];
        sum += c4[q];
        big = max(big, c4[q]);
    }
    for (int o = 32; o > 0; o >>= 1) big = max(big, __shfl_xor(big, o, 64));
    if (lane == 0) atomicMax(&mm[2], (uint32_t)big);
    int N;
    int at = block_exclusive_scan(sum, red, N);  // has barriers: every count is read
#pragma unroll
    for (int q = 0; q < 4; q++) {
        cnt[4 * tid + q] = at;
        at += c4[q];
    }
    if (tid == 0) cnt[kBk] = N;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 8; j++)
        if (k8[j] != kDead) keys[cnt[bk[j]] + slot[j]] = k8[j];
    __syncthreads();
    if ((int)mm[2] > kBkMax) {  // uniform: sort the scattered keys
        sort_and_time(keys, keys + n, N, T, ts);
        return;
    }
#pragma unroll
    for (int j = 0; j < 8; j++) {
        if (k8[j] == kDead) continue;
        const int s0 = cnt[bk[j]], s1 = cnt[bk[j] + 1];
        int r = s0;
        for (int m = s0; m < s1; m++) r += keys[m] < k8[j] ? 1 : 0;
        ts[tid + kThreads * j] = (uint8_t)(((long long)r * T) / N);
    }
}

__global__ __launch_bounds__(kThreads) void k_code_bucket(const float *__restrict__ x, int n, int T,
                                                          float min_value, uint8_t *__restrict__ times)
{
    extern __shared__ uint64_t keys[];  // two buffers of n keys (the second for the sort)
    __shared__ int cnt[kBk + 1];        // bucket counts, then their first slots
    __shared__ int red[kThreads / 64];
    __shared__ uint32_t mm[3];          // lowest and highest value word, largest bucket
    const int b = blockIdx.x;
    const float *xs = x + (size_t)b * n;
    float xv[8];
#pragma unroll
    for (int j = 0; j < 8; j++) xv[j] = xs[min((int)threadIdx.x + kThreads * j, n - 1)];  // coalesced, all loads first
    bucket_code(xv, n, T, min_value, times + (size_t)b * n, keys, cnt, red, mm);
}

// DoG filtering and rank coding of one sample per block (spk_dog_latency_code;
// the filters fit one coefficient block, p.fidx[f] = f).  The sample's image
// is staged in LDS as the filter kernel stages it (u / 255, 0 in the
// padding), over the rows and columns every filter's window reaches.  Each
// thread computes runs of kDogRun outputs along a row with the window
// arithmetic of spk_dog_filter (so the values, and hence the ranks, are
// those of the two calls in sequence) into an LDS array of the sample's
// values, from which each thread takes its flat indices for the ranking.
// The staged image and the values sit in the region the keys use later.
constexpr int kDogRun = 7;

__host__ __device__ inline int dog_runs(int Wo) { return (Wo + kDogRun - 1) / kDogRun; }

__global__ __launch_bounds__(kThreads) void k_dog_code(const uint8_t *__restrict__ img, int C, int H, int W,
                                                       int F, int Ho, int Wo, spk::dog::DogParams p, int T,
                                                       float min_value, uint8_t *__restrict__ times,
                                                       float *__restrict__ dog_out)
{
    extern __shared__ uint64_t keys[];
    __shared__ int cnt[kBk + 1];
    __shared__ int red[kThreads / 64];
    __shared__ uint32_t mm[3];
    __shared__ float coef[spk::dog::kMaxCoef];
    const int b = blockIdx.x, tid = threadIdx.x;
    const int n = C * F * Ho * Wo, nr = dog_runs(Wo);
    const int Hs = Ho + p.hi - p.lo, Ws = nr * kDogRun + p.hi - p.lo;  // staged rows and columns
    float *stage = reinterpret_cast<float *>(keys);
    float *vals = stage + (size_t)C * Hs * Ws;
    const uint8_t *src = img + (size_t)b * C * H * W;
    for (int i = tid; i < p.cbase[F - 1] + p.ks[F - 1] * p.ks[F - 1]; i += kThreads) coef[i] = p.coef[i];
    for (int i = tid; i < C * Hs * Ws; i += kThreads) {
        const int c = i / (Hs * Ws), r = i - c * Hs * Ws, yy = r / Ws, xx = r - yy * Ws;
        stage[i] = spk::dog::pixel(src + (size_t)c * H * W, H, W, yy + p.lo, xx + p.lo);
    }
    __syncthreads();
    for (int u = tid; u < C * F * Ho * nr; u += kThreads) {
        const int pl = u / (Ho * nr), yq = u - pl * Ho * nr, y = yq / nr, x0 = (yq - y * nr) * kDogRun;
        const int c = pl / F, f = pl - c * F, o = p.off[f] - p.lo;
        float acc[kDogRun];
        spk::dog::window_run_k<kDogRun>(p.ks[f], coef + p.cbase[f],
                                        stage + ((size_t)c * Hs + y + o) * Ws + x0 + o, Ws, acc);
#pragma unroll
        for (int r = 0; r < kDogRun; r++) {
            if (x0 + r < Wo) {
                const int i = (pl * Ho + y) * Wo + x0 + r;
                vals[i] = acc[r];
                if (dog_out) dog_out[(size_t)b * n + i] = acc[r];
            }
        }
    }
    __syncthreads();
    float xv[8];
#pragma unroll
    for (int j = 0; j < 8; j++) xv[j] = vals[min(tid + kThreads * j, n - 1)];
    __syncthreads();  // the staged image and the values are dead: their LDS becomes the keys
    bucket_code(xv, n, T, min_value, times + (size_t)b * n, keys, cnt, red, mm);
}

// ------------------------------------------------------------------------
// Samples of more than kSmall values.  A value's step depends on its rank r
// only through floor(r*T/N): with R_k = ceil(k*N/T), t >= k exactly when
// r >= R_k.  So only the T - 1 keys at ranks R_k (the boundaries between
// steps) are needed, not a sort: t = the number of boundary keys at or below
// the value's key.  The boundaries are found by selection:
//  1. a histogram of the top 16 bits of the keys (the sign, exponent and 7
//     mantissa bits of the value word) per sample;
//  2. its prefix sum gives the bucket holding each R_k and the boundary's
//     rank inside that bucket;
//  3. the keys of those buckets are gathered into lists;
//  4. per boundary, a radix select (8-bit digits over the remaining 48 key
//     bits) finds the key of that rank in its bucket's list;
//  5. every value counts the boundary keys at or below its own.
// Work is a few passes over the values plus the keys of T - 1 buckets,
// whatever the sample size; equal values only make a bucket larger.
constexpr int kHB = 65536;  // histogram buckets (top 16 key bits)
constexpr int kCl = 8;      // values per thread in the streaming passes
constexpr int kClT = 256;   // threads of the streaming passes
constexpr int kMaxB = SPK_MAX_T;  // boundaries per sample (T - 1 <= 253)

struct ClBound {   // one boundary k of one sample
    int bucket;    // -1: R_k >= N, the boundary is past every key
    int local;     // its rank inside the bucket
    int list;      // index of the bucket's list in the sample's table
};

struct ClList {    // one distinct boundary bucket of a sample
    int bucket, offset, size;
};

// 0. clear the histograms and counts (B x kHB + B) and the list fill counters
__global__ void k_cl_zero(int *__restrict__ p, long long n)
{
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

// 1. histogram of the eligible keys' top 16 bits, and the eligible count
__global__ __launch_bounds__(kClT) void k_cl_hist(const float *__restrict__ x, int n, float min_value,
                                                  int *__restrict__ hist, int *__restrict__ count)
{
    __shared__ int red[kClT / 64];
    const int b = blockIdx.y;
    const float *xs = x + (size_t)b * n;
    int *h = hist + (size_t)b * kHB;
    const int base = blockIdx.x * kClT * kCl + threadIdx.x;
    float v[kCl];
#pragma unroll
    for (int j = 0; j < kCl; j++) v[j] = xs[min(base + kClT * j, n - 1)];
    int mine = 0;
#pragma unroll
    for (int j = 0; j < kCl; j++) {
        if (base + kClT * j < n && v[j] > min_value) {
            atomicAdd(&h[order_desc(v[j]) >> 16], 1);
            mine++;
        }
    }
    const int tot = block_sum(mine, red);
    if (threadIdx.x == 0 && tot) atomicAdd(&count[b], tot);
}

// 2. one block per sample: prefix sum of the histogram, the bucket and local
// rank of every boundary, and the table of distinct boundary buckets (with
// their list offsets inside the sample's list area and a membership bitmap).
// The histogram is scanned in chunks of 4 * blockDim buckets, each thread
// reading 4 consecutive counts (one 16-byte load, coalesced over the block).
__global__ __launch_bounds__(kThreads) void k_cl_bounds(const int *__restrict__ hist,
                                                        const int *__restrict__ count, int T,
                                                        ClBound *__restrict__ bnd, ClList *__restrict__ lists,
                                                        int *__restrict__ nlists, uint32_t *__restrict__ bitmap,
                                                        int *__restrict__ fill)
{
    constexpr int kChunk = 4 * kThreads;
    __shared__ int red[kThreads / 64];
    __shared__ int s_bucket[kMaxB], s_local[kMaxB];
    const int b = blockIdx.x;
    const int *h = hist + (size_t)b * kHB;
    const int N = count[b];
    uint32_t *bm = bitmap + (size_t)b * (kHB / 32);
    for (int i = threadIdx.x; i < kHB / 32; i += kThreads) bm[i] = 0u;
    for (int k = threadIdx.x; k < T - 1; k += kThreads) {
        s_bucket[k] = -1;  // R_k >= N: past every key
        s_local[k] = 0;
    }
    int chunk_base = 0;  // keys in the chunks before
    for (int c0 = 0; c0 < kHB; c0 += kChunk) {
        const int4 c4 = reinterpret_cast<const int4 *>(h + c0)[threadIdx.x];
        const int c[4] = {c4.x, c4.y, c4.z, c4.w};
        const int sum = c[0] + c[1] + c[2] + c[3];
        int total;
        const int start = chunk_base + block_exclusive_scan(sum, red, total);  // has barriers
        // each boundary rank R_k in this thread's four buckets
        if (sum > 0) {
            // k with start <= R_k < start + sum, R_k = ceil(k N / T): the
            // first has k > T (start - 1) / N
            const int k0 = max(1, (int)((long long)(start - 1) * T / N));
            for (int k = k0; k < T; k++) {
                const long long R = ((long long)k * N + T - 1) / T;
                if (R >= (long long)start + sum) break;
                if (R < start) continue;
                int at = start;
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    if (R >= at && R < at + c[q]) {
                        s_bucket[k - 1] = c0 + 4 * threadIdx.x + q;
                        s_local[k - 1] = (int)(R - at);
                    }
                    at += c[q];
                }
            }
        }
        chunk_base += total;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        // buckets are nondecreasing in k: consecutive equal ones share a list
        int nl = 0, off = 0, prev = -1;
        for (int k = 0; k < T - 1; k++) {
            const int bk = s_bucket[k];
            ClBound r{bk, s_local[k], -1};
            if (bk >= 0) {
                if (bk != prev) {
                    const int sz = h[bk];
                    lists[(size_t)b * kMaxB + nl] = ClList{bk, off, sz};
                    fill[(size_t)b * kMaxB + nl] = 0;
                    bm[bk >> 5] |= 1u << (bk & 31);
                    off += sz;
                    nl++;
                    prev = bk;
                }
                r.list = nl - 1;
            }
            bnd[(size_t)b * kMaxB + k] = r;
        }
        nlists[b] = nl;
    }
}

// 3. the keys of the boundary buckets into their lists (any order)
__global__ __launch_bounds__(kClT) void k_cl_gather(const float *__restrict__ x, int n, float min_value,
                                                    const ClList *__restrict__ lists,
                                                    const int *__restrict__ nlists,
                                                    const uint32_t *__restrict__ bitmap,
                                                    int *__restrict__ fill, uint64_t *__restrict__ keys)
{
    __shared__ uint32_t bm[kHB / 32];
    __shared__ int s_bk[kMaxB];
    const int b = blockIdx.y;
    const int nl = nlists[b];
    if (nl == 0) return;  // uniform: no boundary (no eligible value)
    for (int i = threadIdx.x; i < kHB / 32; i += kClT) bm[i] = bitmap[(size_t)b * (kHB / 32) + i];
    for (int i = threadIdx.x; i < nl; i += kClT) s_bk[i] = lists[(size_t)b * kMaxB + i].bucket;
    __syncthreads();
    const float *xs = x + (size_t)b * n;
    const int base = blockIdx.x * kClT * kCl + threadIdx.x;
    float v[kCl];
#pragma unroll
    for (int j = 0; j < kCl; j++) v[j] = xs[min(base + kClT * j, n - 1)];
#pragma unroll
    for (int j = 0; j < kCl; j++) {
        const int i = base + kClT * j;
        if (i >= n || !(v[j] > min_value)) continue;
        const uint32_t w = order_desc(v[j]);
        const int bk = (int)(w >> 16);
        if (!((bm[bk >> 5] >> (bk & 31)) & 1u)) continue;
        int lo = 0, hi = nl - 1;  // the list of bucket bk (buckets ascend with the list index)
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (s_bk[mid] < bk) lo = mid + 1;
            else hi = mid;
        }
        const ClList L = lists[(size_t)b * kMaxB + lo];
        const int slot = atomicAdd(&fill[(size_t)b * kMaxB + lo], 1);
        keys[(size_t)b * n + L.offset + slot] = ((uint64_t)w << 32) | (uint32_t)i;
    }
}

// 4. one block per (boundary, sample): the key of rank `local` in its bucket's
// list, by radix selection over the 48 bits below the bucket's (8-bit digits,
// most significant first).  Boundaries past every key get the all-ones key.
__global__ __launch_bounds__(kClT) void k_cl_select(const ClBound *__restrict__ bnd,
                                                    const ClList *__restrict__ lists,
                                                    const uint64_t *__restrict__ keys, int n,
                                                    uint64_t *__restrict__ bkeys)
{
    __shared__ int hist[256];
    __shared__ uint64_t s_prefix;
    __shared__ int s_rank;
    const int k = blockIdx.x, b = blockIdx.y;
    const ClBound r = bnd[(size_t)b * kMaxB + k];
    if (r.bucket < 0) {
        if (threadIdx.x == 0) bkeys[(size_t)b * kMaxB + k] = kDead;
        return;
    }
    const ClList L = lists[(size_t)b * kMaxB + r.list];
    const uint64_t *ks = keys + (size_t)b * n + L.offset;
    uint64_t prefix = (uint64_t)r.bucket << 48;  // decided bits
    int rank = r.local;
    for (int shift = 40; shift >= 0; shift -= 8) {
        const uint64_t mask = ~0ull << (shift + 8);  // bits decided so far
        for (int i = threadIdx.x; i < 256; i += kClT) hist[i] = 0;
        __syncthreads();
        for (int i = threadIdx.x; i < L.size; i += kClT) {
            const uint64_t key = ks[i];
            if ((key & mask) == prefix) atomicAdd(&hist[(int)((key >> shift) & 255u)], 1);
        }
        __syncthreads();
        if (threadIdx.x < 64) {  // one wave: the digit whose run holds the rank
            int c4[4], s = 0;
#pragma unroll
            for (int q = 0; q < 4; q++) {
                c4[q] = hist[threadIdx.x * 4 + q];
                s += c4[q];
            }
            int incl = s;
            for (int o = 1; o < 64; o <<= 1) {
                const int t = __shfl_up(incl, o, 64);
                if ((int)threadIdx.x >= o) incl += t;
            }
            int at = incl - s;
            for (int q = 0; q < 4; q++) {
                if (rank >= at && rank < at + c4[q]) {
                    s_prefix = prefix | ((uint64_t)(threadIdx.x * 4 + q) << shift);
                    s_rank = rank - at;
                }
                at += c4[q];
            }
        }
        __syncthreads();
        prefix = s_prefix;
        rank = s_rank;
        __syncthreads();
    }
    if (threadIdx.x == 0) bkeys[(size_t)b * kMaxB + k] = prefix;
}

// 5. every value's step: the number of boundary keys at or below its key
// (they ascend with k); values at or below min_value never fire.
__global__ __launch_bounds__(kClT) void k_cl_final(const float *__restrict__ x, int n, int T,
                                                   float min_value, const uint64_t *__restrict__ bkeys,
                                                   uint8_t *__restrict__ times)
{
    __shared__ uint64_t bk[kMaxB];
    const int b = blockIdx.y;
    for (int i = threadIdx.x; i < T - 1; i += kClT) bk[i] = bkeys[(size_t)b * kMaxB + i];
    __syncthreads();
    const float *xs = x + (size_t)b * n;
    uint8_t *ts = times + (size_t)b * n;
    const int base = blockIdx.x * kClT * kCl + threadIdx.x;
    float v[kCl];
#pragma unroll
    for (int j = 0; j < kCl; j++) v[j] = xs[min(base + kClT * j, n - 1)];
#pragma unroll
    for (int j = 0; j < kCl; j++) {
        const int i = base + kClT * j;
        if (i >= n) continue;
        uint8_t t = spk::kNever;
        if (v[j] > min_value) {
            const uint64_t key = ((uint64_t)order_desc(v[j]) << 32) | (uint32_t)i;
            int lo = 0, hi = T - 1;  // first boundary above the key
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (bk[mid] <= key) lo = mid + 1;
                else hi = mid;
            }
            t = (uint8_t)lo;
        }
        ts[i] = t;
    }
}

// Linear mode (sort disabled): one workgroup per sample.
__global__ __launch_bounds__(kThreads) void k_code_linear(const float *__restrict__ x, int n, int T,
                                                          float min_value,
                                                          uint8_t *__restrict__ times)
{
#pragma clang fp contract(off)
    __shared__ float red[kThreads / 64];
    const int b = blockIdx.x;
    const float *xs = x + (size_t)b * n;
    uint8_t *ts = times + (size_t)b * n;
    float m = -INFINITY;
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
        float v = xs[i];
        if (v > min_value) m = fmaxf(m, v);
    }
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_down(m, o, 64));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        float mm = red[0];
        for (int w = 1; w < (int)(blockDim.x >> 6); w++) mm = fmaxf(mm, red[w]);
        red[0] = mm;
    }
    __syncthreads();
    const float vmax = red[0];
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
        float v = xs[i];
        uint8_t t = spk::kNever;
        if (v > min_value) {
            float q = v / vmax;
            float s = 1.0f - q;
            float u = s * (float)T;
            int ti = (int)floorf(u);
            ti = min(ti, T - 1);
            ti = max(ti, 0);
            t = (uint8_t)ti;
        }
        ts[i] = t;
    }
}

__global__ void k_code_frames(const uint8_t *__restrict__ times, int T, int n,
                              uint8_t *__restrict__ frames)
{
    const int b = blockIdx.z, t = blockIdx.y;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    frames[((size_t)b * T + t) * n + i] = (uint8_t)(times[(size_t)b * n + i] <= t);
}

// Workspace of the large-sample path: histograms, counts, boundary records,
// list tables, bitmaps, fill counters, boundary keys and the lists (at most
// the sample's values).
struct ClWs {
    size_t hist, count, bnd, lists, nlists, bitmap, fill, bkeys, keys, total;
};

ClWs cl_layout(int B, long long n)
{
    ClWs w{};
    size_t at = 0;
    auto take = [&](size_t bytes) {
        const size_t here = at;
        at += spk::align_up(bytes, 256);
        return here;
    };
    w.hist = take((size_t)B * kHB * sizeof(int));
    w.count = take((size_t)B * sizeof(int));
    w.bnd = take((size_t)B * kMaxB * sizeof(ClBound));
    w.lists = take((size_t)B * kMaxB * sizeof(ClList));
    w.nlists = take((size_t)B * sizeof(int));
    w.bitmap = take((size_t)B * (kHB / 32) * sizeof(uint32_t));
    w.fill = take((size_t)B * kMaxB * sizeof(int));
    w.bkeys = take((size_t)B * kMaxB * sizeof(uint64_t));
    w.keys = take((size_t)B * n * sizeof(uint64_t));
    w.total = at;
    return w;
}

size_t ws_layout(int B, long long n) { return n <= kSmall ? 0 : cl_layout(B, n).total; }

// The fused DoG + coding kernel applies when every filter fits one
// coefficient block, the sample fits the bucketed coder and the staged image
// fits LDS beside the kernel's static arrays; lds: its dynamic LDS bytes.
bool dog_code_fits(int C, int F, int Ho, int Wo, const spk::dog::DogParams &p, size_t &lds)
{
    const long long n = (long long)C * F * Ho * Wo;
    const long long stage = (long long)C * (Ho + p.hi - p.lo) * (dog_runs(Wo) * kDogRun + p.hi - p.lo) * 4;
    lds = (size_t)std::max(2 * n * 8, stage + 4 * n);
    return p.nf == F && n <= kSmall && lds + 20 * 1024 <= 160 * 1024;
}

}  // namespace

extern "C" size_t spk_latency_code_workspace_size(int B, int C, int H, int W)
{
    if (B <= 0 || C <= 0 || H <= 0 || W <= 0) return 0;
    return ws_layout(B, (long long)C * H * W);
}

extern "C" spk_status spk_latency_code(const float *x, int B, int C, int H, int W, int T,
                                       float min_value, int mode, uint8_t *times, uint8_t *frames,
                                       void *ws, size_t ws_bytes, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(x && times, SPK_E_ARG, "spk_latency_code: NULL pointer");
    SPK_REQUIRE(B > 0 && C > 0 && H > 0 && W > 0, SPK_E_ARG,
                "spk_latency_code: B=%d C=%d H=%d W=%d must be positive", B, C, H, W);
    SPK_REQUIRE(mode == SPK_CODE_RANK || mode == SPK_CODE_LINEAR, SPK_E_ARG,
                "spk_latency_code: unknown mode %d", mode);
    SPK_REQUIRE(T >= 1 && T <= SPK_MAX_T, SPK_E_SHAPE, "spk_latency_code: T=%d not in [1, %d]", T,
                SPK_MAX_T);
    const long long nl = (long long)C * H * W;
    SPK_REQUIRE(nl < (1LL << 31) && (long long)B * nl < (1LL << 40), SPK_E_SHAPE,
                "spk_latency_code: sample of %lld values too large", nl);
    SPK_REQUIRE(B <= 65535, SPK_E_SHAPE, "spk_latency_code: B=%d > 65535", B);
    const int n = (int)nl;
    const size_t need = mode == SPK_CODE_RANK ? ws_layout(B, n) : 0;
    SPK_REQUIRE(ws_bytes >= need && (need == 0 || ws), SPK_E_WORKSPACE,
                "spk_latency_code: workspace of %zu bytes needed, %zu given", need, ws_bytes);
    SPK_REQUIRE_WS_ALIGNED(ws, "spk_latency_code");
    hipStream_t s = spk::stream_of(stream);

    if (mode == SPK_CODE_LINEAR) {
        hipLaunchKernelGGL(k_code_linear, dim3(B), dim3(kThreads), 0, s, x, n, T, min_value, times);
        SPK_LAUNCHED("spk_latency_code");
    } else if (n <= kSmall) {
        const size_t lds = 2 * (size_t)n * sizeof(uint64_t);
        if (lds > 64 * 1024)
            (void)hipFuncSetAttribute(reinterpret_cast<const void *>(k_code_bucket),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        hipLaunchKernelGGL(k_code_bucket, dim3(B), dim3(kThreads), lds, s, x, n, T, min_value, times);
        SPK_LAUNCHED("spk_latency_code");
    } else {
        const ClWs L = cl_layout(B, n);
        char *w = (char *)ws;
        int *hist = (int *)(w + L.hist), *count = (int *)(w + L.count);
        ClBound *bnd = (ClBound *)(w + L.bnd);
        ClList *lists = (ClList *)(w + L.lists);
        int *nlists = (int *)(w + L.nlists), *fill = (int *)(w + L.fill);
        uint32_t *bitmap = (uint32_t *)(w + L.bitmap);
        uint64_t *bkeys = (uint64_t *)(w + L.bkeys), *keys = (uint64_t *)(w + L.keys);
        // histograms and counts are adjacent: one clearing pass
        const long long nz = (long long)(L.count - L.hist) / 4 + B;
        hipLaunchKernelGGL(k_cl_zero, dim3(spk::ceil_div(nz, 256)), dim3(256), 0, s, hist, nz);
        SPK_LAUNCHED("spk_latency_code");
        const dim3 sgrid(spk::ceil_div(n, kClT * kCl), B);
        hipLaunchKernelGGL(k_cl_hist, sgrid, dim3(kClT), 0, s, x, n, min_value, hist, count);
        SPK_LAUNCHED("spk_latency_code");
        hipLaunchKernelGGL(k_cl_bounds, dim3(B), dim3(kThreads), 0, s, hist, count, T, bnd, lists, nlists,
                           bitmap, fill);
        SPK_LAUNCHED("spk_latency_code");
        hipLaunchKernelGGL(k_cl_gather, sgrid, dim3(kClT), 0, s, x, n, min_value, lists, nlists, bitmap,
                           fill, keys);
        SPK_LAUNCHED("spk_latency_code");
        if (T > 1) {
            hipLaunchKernelGGL(k_cl_select, dim3(T - 1, B), dim3(kClT), 0, s, bnd, lists, keys, n, bkeys);
            SPK_LAUNCHED("spk_latency_code");
        }
        hipLaunchKernelGGL(k_cl_final, sgrid, dim3(kClT), 0, s, x, n, T, min_value, bkeys, times);
        SPK_LAUNCHED("spk_latency_code");
    }
    if (frames) {
        SPK_REQUIRE(T <= 65535, SPK_E_SHAPE, "spk_latency_code: T too large for frames");
        hipLaunchKernelGGL(k_code_frames, dim3(spk::ceil_div(n, 256), T, B), dim3(256), 0, s, times,
                           T, n, frames);
        SPK_LAUNCHED("spk_latency_code");
    }
    return SPK_OK;
}

extern "C" size_t spk_dog_latency_code_workspace_size(int B, int C, int H, int W,
                                                     const spk_dog_desc *filters, int F, int pad)
{
    int Ho = 0, Wo = 0;
    if (!filters || spk::dog::plan("spk_dog_latency_code_workspace_size", B, C, H, W, filters, F, pad, Ho,
                                   Wo) != SPK_OK)
        return 0;
    spk::dog::DogParams p;
    spk::dog::group(filters, F, pad, 0, p);
    size_t lds = 0;
    if (dog_code_fits(C, F, Ho, Wo, p, lds)) return 0;
    return spk::align_up((size_t)B * C * F * Ho * Wo * sizeof(float), 256) +
           spk_latency_code_workspace_size(B, C * F, Ho, Wo);
}

extern "C" spk_status spk_dog_latency_code(const uint8_t *img, int B, int C, int H, int W,
                                           const spk_dog_desc *filters, int F, int pad, int T,
                                           float min_value, uint8_t *times, float *dog_out, void *ws,
                                           size_t ws_bytes, spk_stream stream)
{
    spk::clear_error();
    SPK_REQUIRE(img && filters && times, SPK_E_ARG, "spk_dog_latency_code: NULL pointer");
    int Ho = 0, Wo = 0;
    const spk_status st = spk::dog::plan("spk_dog_latency_code", B, C, H, W, filters, F, pad, Ho, Wo);
    if (st != SPK_OK) return st;
    SPK_REQUIRE(T >= 1 && T <= SPK_MAX_T, SPK_E_SHAPE, "spk_dog_latency_code: T=%d not in [1, %d]", T,
                SPK_MAX_T);
    SPK_REQUIRE((long long)C * F * Ho * Wo < (1LL << 31), SPK_E_SHAPE,
                "spk_dog_latency_code: sample of %lld values too large", (long long)C * F * Ho * Wo);
    spk::dog::DogParams p;
    spk::dog::group(filters, F, pad, 0, p);
    size_t lds = 0;
    if (dog_code_fits(C, F, Ho, Wo, p, lds)) {
        SPK_REQUIRE(B <= 65535, SPK_E_SHAPE, "spk_dog_latency_code: B=%d > 65535", B);
        if (lds > 64 * 1024)
            (void)hipFuncSetAttribute(reinterpret_cast<const void *>(k_dog_code),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        hipLaunchKernelGGL(k_dog_code, dim3(B), dim3(kThreads), lds, spk::stream_of(stream), img, C, H, W,
                           F, Ho, Wo, p, T, min_value, times, dog_out);
        SPK_LAUNCHED("spk_dog_latency_code");
        return SPK_OK;
    }
    // the two calls in sequence, the filter outputs in dog_out or the workspace
    const size_t xb = spk::align_up((size_t)B * C * F * Ho * Wo * sizeof(float), 256);
    const size_t cw = spk_latency_code_workspace_size(B, C * F, Ho, Wo);
    SPK_REQUIRE(ws && ws_bytes >= xb + cw, SPK_E_WORKSPACE,
                "spk_dog_latency_code: workspace of %zu bytes needed, %zu given", xb + cw, ws_bytes);
    SPK_REQUIRE_WS_ALIGNED(ws, "spk_dog_latency_code");
    float *x = dog_out ? dog_out : static_cast<float *>(ws);
    spk_status s2 = spk_dog_filter(img, B, C, H, W, filters, F, pad, x, stream);
    if (s2 != SPK_OK) return s2;
    return spk_latency_code(x, B, C * F, Ho, Wo, T, min_value, SPK_CODE_RANK, times, nullptr,
                            cw ? static_cast<char *>(ws) + xb : nullptr, cw, stream);
}
