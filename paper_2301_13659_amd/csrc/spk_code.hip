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
//  - Larger samples: workgroups sort kSmall-key chunks in LDS, then merge
//    passes double the sorted runs (merge-path split per thread) until each
//    sample is one run; the ping-pong buffers live in the caller workspace.
#include <cstring>

#include "spk_internal.h"

namespace {

constexpr int kSmall = 8192;    // keys per LDS sort (2 x 64 KB)
constexpr int kThreads = 1024;
constexpr int kMergePerThread = 8;
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

// Merge runs of `width` sorted keys pairwise (src -> dst, n keys); thread t
// produces outputs [8t, 8t + 8) from a merge-path split.
__device__ void merge_level(const uint64_t *src, uint64_t *dst, int n, int width)
{
    const int first = threadIdx.x * 8;
    if (first >= n) return;
    const int lo = (first / (2 * width)) * 2 * width;
    const int na = min(width, n - lo), nb = max(0, min(width, n - lo - width));
    const uint64_t *A = src + lo, *Bv = src + lo + na;
    const int p = first - lo;
    int ilo = max(0, p - nb), ihi = min(p, na);
    while (ilo < ihi) {
        const int i = (ilo + ihi) >> 1;
        if (A[i] < Bv[p - i - 1]) ilo = i + 1;
        else ihi = i;
    }
    int i = ilo, j = p - ilo;
    const int end = min(p + 8, na + nb);
    for (int q = p; q < end; q++) {
        const bool takeA = (j >= nb) || (i < na && A[i] < Bv[j]);
        dst[lo + q] = takeA ? A[i++] : Bv[j++];
    }
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

__global__ __launch_bounds__(kThreads) void k_code_bucket(const float *__restrict__ x, int n, int T,
                                                          float min_value, uint8_t *__restrict__ times)
{
    extern __shared__ uint64_t keys[];  // two buffers of n keys (the second for the sort)
    __shared__ int cnt[kBk + 1];        // bucket counts, then their first slots
    __shared__ int red[kThreads / 64];
    __shared__ uint32_t mm[3];          // lowest and highest value word, largest bucket
    const int b = blockIdx.x;
    const float *xs = x + (size_t)b * n;
    uint8_t *ts = times + (size_t)b * n;
    const int tid = threadIdx.x, lane = tid & 63;

    float xv[8];
#pragma unroll
    for (int j = 0; j < 8; j++) xv[j] = xs[min(tid + kThreads * j, n - 1)];  // coalesced, all loads first
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

// Large samples, step 1: keys, never-firing outputs, eligible counts.
__global__ void k_code_keys(const float *__restrict__ x, int B, int n, float min_value,
                            uint64_t *__restrict__ keys, uint8_t *__restrict__ times,
                            int *__restrict__ count)
{
    __shared__ int red[256 / 64];
    const int b = blockIdx.y;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    int mine = 0;
    if (i < n) {
        uint64_t key = make_key(x[(size_t)b * n + i], min_value, (uint32_t)i);
        keys[(size_t)b * n + i] = key;
        if (key == kDead) times[(size_t)b * n + i] = spk::kNever;
        else mine = 1;
    }
    int tot = block_sum(mine, red);
    if (threadIdx.x == 0 && tot) atomicAdd(&count[b], tot);
}

__global__ void k_zero_int(int *p, int n)
{
    int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

// Large samples, step 2: sort kSmall-key chunks (register sort of 8, then
// merge levels in LDS).
__global__ __launch_bounds__(kThreads) void k_code_chunks(uint64_t *__restrict__ keys, int n)
{
    extern __shared__ uint64_t s[];  // two buffers of kSmall keys
    const int b = blockIdx.y;
    const int base = blockIdx.x * kSmall;
    const int len = min(kSmall, n - base);
    uint64_t *g = keys + (size_t)b * n + base;
    uint64_t k8[8];
    const int first = threadIdx.x * 8;
#pragma unroll
    for (int j = 0; j < 8; j++) k8[j] = (first + j < len) ? g[first + j] : kDead;
    sort8(k8);
    uint64_t *src = s, *dst = s + kSmall;
#pragma unroll
    for (int j = 0; j < 8; j++)
        if (first + j < len) src[first + j] = k8[j];
    __syncthreads();
    for (int width = 8; width < len; width *= 2) {
        merge_level(src, dst, len, width);
        __syncthreads();
        uint64_t *t = src;
        src = dst;
        dst = t;
    }
    for (int i = threadIdx.x; i < len; i += blockDim.x) g[i] = src[i];
}

// Large samples, step 3: merge sorted runs of `width` pairwise, src -> dst.
__global__ void k_code_merge(const uint64_t *__restrict__ src, uint64_t *__restrict__ dst, int n,
                             int width)
{
    const int b = blockIdx.y;
    const long long first = ((long long)blockIdx.x * blockDim.x + threadIdx.x) * kMergePerThread;
    if (first >= n) return;
    const uint64_t *S = src + (size_t)b * n;
    uint64_t *D = dst + (size_t)b * n;
    const int lo = (int)(first / (2LL * width)) * 2 * width;
    const int na = min(width, n - lo);
    const int nb = max(0, min(width, n - lo - width));
    const uint64_t *A = S + lo, *Bv = S + lo + na;
    const int p = (int)first - lo;
    // co-rank: number i of A keys among the first p merged keys
    int ilo = max(0, p - nb), ihi = min(p, na);
    while (ilo < ihi) {
        int i = (ilo + ihi) >> 1;
        if (A[i] < Bv[p - i - 1]) ilo = i + 1;
        else ihi = i;
    }
    int i = ilo, j = p - ilo;
    const int end = min(p + kMergePerThread, na + nb);
    for (int q = p; q < end; q++) {
        bool takeA = (j >= nb) || (i < na && A[i] < Bv[j]);
        D[lo + q] = takeA ? A[i++] : Bv[j++];
    }
}

// Large samples, step 4: rank -> time.
__global__ void k_code_scatter(const uint64_t *__restrict__ keys, int n, int T,
                               const int *__restrict__ count, uint8_t *__restrict__ times)
{
    const int b = blockIdx.y;
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    const int N = count[b];
    if (r >= N) return;
    uint32_t idx = (uint32_t)keys[(size_t)b * n + r];
    times[(size_t)b * n + idx] = (uint8_t)(((long long)r * T) / N);
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

size_t ws_layout(int B, long long n, size_t *off_b, size_t *off_cnt)
{
    if (n <= kSmall) {
        *off_b = *off_cnt = 0;
        return 0;
    }
    size_t keys = spk::align_up((size_t)B * n * sizeof(uint64_t), 256);
    *off_b = keys;
    *off_cnt = 2 * keys;
    return 2 * keys + spk::align_up((size_t)B * sizeof(int), 256);
}

}  // namespace

extern "C" size_t spk_latency_code_workspace_size(int B, int C, int H, int W)
{
    if (B <= 0 || C <= 0 || H <= 0 || W <= 0) return 0;
    size_t a, c;
    return ws_layout(B, (long long)C * H * W, &a, &c);
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
    size_t off_b, off_cnt;
    const size_t need = mode == SPK_CODE_RANK ? ws_layout(B, n, &off_b, &off_cnt) : 0;
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
        uint64_t *ka = (uint64_t *)ws;
        uint64_t *kb = (uint64_t *)((char *)ws + off_b);
        int *cnt = (int *)((char *)ws + off_cnt);
        hipLaunchKernelGGL(k_zero_int, dim3(spk::ceil_div(B, 256)), dim3(256), 0, s, cnt, B);
        SPK_LAUNCHED("spk_latency_code");
        hipLaunchKernelGGL(k_code_keys, dim3(spk::ceil_div(n, 256), B), dim3(256), 0, s, x, B, n,
                           min_value, ka, times, cnt);
        SPK_LAUNCHED("spk_latency_code");
        const size_t clds = 2 * (size_t)kSmall * sizeof(uint64_t);
        (void)hipFuncSetAttribute(reinterpret_cast<const void *>(k_code_chunks),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)clds);
        hipLaunchKernelGGL(k_code_chunks, dim3(spk::ceil_div(n, kSmall), B), dim3(kThreads), clds, s,
                           ka, n);
        SPK_LAUNCHED("spk_latency_code");
        uint64_t *src = ka, *dst = kb;
        for (long long width = kSmall; width < n; width *= 2) {
            dim3 grid(spk::ceil_div(spk::ceil_div(n, kMergePerThread), 256), B);
            hipLaunchKernelGGL(k_code_merge, grid, dim3(256), 0, s, src, dst, n, (int)width);
            SPK_LAUNCHED("spk_latency_code");
            std::swap(src, dst);
        }
        hipLaunchKernelGGL(k_code_scatter, dim3(spk::ceil_div(n, 256), B), dim3(256), 0, s, src, n,
                           T, cnt, times);
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
