/*
 * spk_oracle.c -- TEST INFRASTRUCTURE, not part of the product.
 *
 * A plain, slow, obviously correct CPU implementation of the spiking-conv
 * pipeline of Spyker (arXiv 2301.13659): DoG filtering, rank-order latency
 * coding, convolution with integrate-and-fire, spike-time max-pooling,
 * lateral inhibition with k-winners-take-all, and STDP / R-STDP.  It exists
 * only to check the GPU library against.  Only the tests, the smoke check and
 * the benchmark's CPU-baseline leg may load it.  It shares no code, header,
 * table or helper with the GPU library.
 *
 * Precision: double everywhere the paper leaves it open (potentials, weight
 * updates).  Two places use float on purpose because a float value decides an
 * integer there and both implementations must take that decision in the same
 * precision: the DoG output (its ranks become spike times) and the linear
 * (no-sort) coding formula.
 *
 * Every function is written from the definitions in the paper, in the order
 * the paper states them; no blocking, fusion or reordering.  Readings of
 * passages the paper leaves open are noted where they are taken.
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared (build() in oracle/__init__.py).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_NEVER 255

/* ------------------------------------------------------------------------ */
/* DoG filter bank: §II-C.1 (Difference of Gaussian filter), §II-C.4 Eq. 1. */
/* ------------------------------------------------------------------------ */

/*
 * One DoG kernel of odd size K: the difference of two discrete Gaussians with
 * standard deviations s1 and s2 (§II-C.1: each filter is described by two
 * standard deviations).  Reading: each Gaussian is sampled at integer offsets
 * in [-R, R]^2, R = (K-1)/2, and normalised to unit sum in double; the
 * difference is then rounded once to float.
 */
void or_dog_kernel(int K, double s1, double s2, float *k)
{
    int R = (K - 1) / 2;
    double *g1 = (double *)malloc(sizeof(double) * K * K);
    double *g2 = (double *)malloc(sizeof(double) * K * K);
    double sum1 = 0.0, sum2 = 0.0;
    for (int i = -R; i <= R; i++)
        for (int j = -R; j <= R; j++) {
            double r2 = (double)(i * i + j * j);
            g1[(i + R) * K + (j + R)] = exp(-r2 / (2.0 * s1 * s1));
            g2[(i + R) * K + (j + R)] = exp(-r2 / (2.0 * s2 * s2));
            sum1 += g1[(i + R) * K + (j + R)];
            sum2 += g2[(i + R) * K + (j + R)];
        }
    for (int n = 0; n < K * K; n++)
        k[n] = (float)(g1[n] / sum1 - g2[n] / sum2);
    free(g1);
    free(g2);
}

/*
 * Filter a uint8 image batch (B x C x H x W) with F DoG kernels applied to each
 * channel separately (§II-C.4: C_o = C_i * K_c).  Output channel c*F + f.
 * pad < 0 selects "same" padding per filter ((K_f - 1) / 2, so filters of
 * different sizes give one output size); pad >= 0 applies Eq. 1 with one
 * padding, which requires every filter to have the same K.
 *
 * Arithmetic, all in float with round-to-nearest and no fused multiply-add:
 * pixel x = (float)u / 255; acc = 0; acc = acc + k[i][j] * x over the window
 * in row-major order; pixels outside the image count as 0.
 */
void or_dog_filter(const uint8_t *img, int B, int C, int H, int W,
                   const int *ksize, const double *sigma1, const double *sigma2,
                   int F, int pad, float *out)
{
    int K0 = ksize[0];
    int Ho = pad < 0 ? H : H + 2 * pad - K0 + 1;
    int Wo = pad < 0 ? W : W + 2 * pad - K0 + 1;
    for (int f = 0; f < F; f++) {
        int K = ksize[f];
        int P = pad < 0 ? (K - 1) / 2 : pad;
        float *k = (float *)malloc(sizeof(float) * K * K);
        or_dog_kernel(K, sigma1[f], sigma2[f], k);
        for (int b = 0; b < B; b++)
            for (int c = 0; c < C; c++)
                for (int y = 0; y < Ho; y++)
                    for (int x = 0; x < Wo; x++) {
                        float acc = 0.0f;
                        for (int i = 0; i < K; i++)
                            for (int j = 0; j < K; j++) {
                                int iy = y + i - P, ix = x + j - P;
                                float v = 0.0f;
                                if (iy >= 0 && iy < H && ix >= 0 && ix < W)
                                    v = (float)img[((size_t)(b * C + c) * H + iy) * W + ix] / 255.0f;
                                float prod = k[i * K + j] * v;
                                acc = acc + prod;
                            }
                        out[((size_t)(b * C * F + c * F + f) * Ho + y) * Wo + x] = acc;
                    }
        free(k);
    }
}

/* ------------------------------------------------------------------------ */
/* Rank-order latency coding: §II-D.2 and §II-D.3 (Coding in Spyker).        */
/* ------------------------------------------------------------------------ */

typedef struct {
    float v;
    int64_t i;
} or_vi;

/* value descending, then flat index ascending (the reading of the sort's tie-break) */
static int or_cmp_rank(const void *pa, const void *pb)
{
    const or_vi *a = (const or_vi *)pa, *b = (const or_vi *)pb;
    if (a->v > b->v) return -1;
    if (a->v < b->v) return 1;
    return (a->i < b->i) ? -1 : (a->i > b->i);
}

/*
 * For each sample, every value above min_value spikes once (values at or
 * below it never do: the threshold applied before coding in the paper's
 * transform).  mode 0 (rank): the eligible values of the whole sample
 * (C*H*W jointly) are sorted by intensity, higher first, and the N spikes
 * are spread evenly over T steps: the value of rank r fires at floor(r*T/N).
 * mode 1 (no sort, "linear"): t = min(T-1, floor((1 - v/vmax) * T)) in float,
 * vmax the sample maximum.  Non-spiking neurons get NEVER (255).
 */
void or_latency_code(const float *x, int B, int64_t n_per_sample, int T,
                     float min_value, int mode, uint8_t *times)
{
    or_vi *buf = (or_vi *)malloc(sizeof(or_vi) * (size_t)(n_per_sample > 0 ? n_per_sample : 1));
    for (int b = 0; b < B; b++) {
        const float *xs = x + (size_t)b * n_per_sample;
        uint8_t *ts = times + (size_t)b * n_per_sample;
        int64_t N = 0;
        for (int64_t i = 0; i < n_per_sample; i++) {
            ts[i] = OR_NEVER;
            if (xs[i] > min_value) {
                buf[N].v = xs[i];
                buf[N].i = i;
                N++;
            }
        }
        if (N == 0) continue;
        if (mode == 0) {
            qsort(buf, (size_t)N, sizeof(or_vi), or_cmp_rank);
            for (int64_t r = 0; r < N; r++)
                ts[buf[r].i] = (uint8_t)((r * (int64_t)T) / N);
        } else {
            float vmax = buf[0].v;
            for (int64_t r = 1; r < N; r++)
                if (buf[r].v > vmax) vmax = buf[r].v;
            for (int64_t r = 0; r < N; r++) {
                float q = buf[r].v / vmax;
                float s = 1.0f - q;
                float u = s * (float)T;
                int t = (int)floorf(u);
                if (t > T - 1) t = T - 1;
                if (t < 0) t = 0;
                ts[buf[r].i] = (uint8_t)t;
            }
        }
    }
    free(buf);
}

/* Cumulative frames (§II-D.3): a neuron that fires at t_i is on in every frame t >= t_i. */
void or_times_to_frames(const uint8_t *times, int B, int T, int64_t n_per_sample, uint8_t *frames)
{
    for (int b = 0; b < B; b++)
        for (int t = 0; t < T; t++)
            for (int64_t i = 0; i < n_per_sample; i++)
                frames[((size_t)b * T + t) * n_per_sample + i] =
                    (uint8_t)(times[(size_t)b * n_per_sample + i] <= t);
}

/* Inverse of the above: the first frame in which the neuron is on, else NEVER. */
void or_frames_to_times(const uint8_t *frames, int B, int T, int64_t n_per_sample, uint8_t *times)
{
    for (int b = 0; b < B; b++)
        for (int64_t i = 0; i < n_per_sample; i++) {
            uint8_t t_first = OR_NEVER;
            for (int t = T - 1; t >= 0; t--)
                if (frames[((size_t)b * T + t) * n_per_sample + i]) t_first = (uint8_t)t;
            times[(size_t)b * n_per_sample + i] = t_first;
        }
}

/* ------------------------------------------------------------------------ */
/* Convolution + integrate-and-fire: §II-E.1 (Convolution), Eq. 2.           */
/* ------------------------------------------------------------------------ */

/*
 * Potentials of one output neuron (b, o, y, x) at every step t: the 2-D
 * convolution of frame t of the input (S_t[c, iy, ix] = [time <= t]) with
 * kernel o, with zero padding and stride (Eq. 2), summed in double:
 *   V_t = sum over c, ky, kx of W[o, c, ky, kx] * S_t[c, y*s + ky - p, x*s + kx - p].
 */
void or_conv_neuron(const uint8_t *in_times, int T, int Ci, int Hi, int Wi,
                    const float *w, int Kh, int Kw, int stride, int pad,
                    int b, int o, int y, int x, double *V)
{
    for (int t = 0; t < T; t++) {
        double acc = 0.0;
        for (int c = 0; c < Ci; c++)
            for (int ky = 0; ky < Kh; ky++)
                for (int kx = 0; kx < Kw; kx++) {
                    int iy = y * stride + ky - pad, ix = x * stride + kx - pad;
                    double s = 0.0;
                    if (iy >= 0 && iy < Hi && ix >= 0 && ix < Wi &&
                        in_times[((size_t)(b * Ci + c) * Hi + iy) * Wi + ix] <= t)
                        s = 1.0;
                    acc += (double)w[((size_t)(o * Ci + c) * Kh + ky) * Kw + kx] * s;
                }
        V[t] = acc;
    }
}

/*
 * Integrate-and-fire on one neuron's potentials: it spikes where the
 * potential is higher than the threshold (§II-E.1), once (rank-order coding:
 * a neuron fires at most once, §II-B), so its spike time is the first t with
 * V_t > theta, else NEVER (theta = +inf never fires).  Its key potential is V
 * at that step, or V at the last step if it never fires (the potential that
 * breaks ties between equal spike times in winner selection, §II-F.3).
 */
void or_fire_neuron(const double *V, int T, double theta, uint8_t *t_f, double *vkey)
{
    *t_f = OR_NEVER;
    *vkey = V[T - 1];
    for (int t = 0; t < T; t++)
        if (V[t] > theta) {
            *t_f = (uint8_t)t;
            *vkey = V[t];
            return;
        }
}

/*
 * The whole layer: every (b, o, y, x) of B x Co x Ho x Wo, with Ho and Wo from
 * Eq. 2.  potentials (nullable) receives B x T x Co x Ho x Wo (the BTCHW
 * order of §II-A).
 */
void or_conv_fire(const uint8_t *in_times, int B, int T, int Ci, int Hi, int Wi,
                  const float *w, int Co, int Kh, int Kw, int stride, int pad, double theta,
                  uint8_t *out_times, float *out_vkey, float *potentials)
{
    int Ho = (Hi + 2 * pad - Kh) / stride + 1;
    int Wo = (Wi + 2 * pad - Kw) / stride + 1;
    double *V = (double *)malloc(sizeof(double) * T);
    for (int b = 0; b < B; b++)
        for (int o = 0; o < Co; o++)
            for (int y = 0; y < Ho; y++)
                for (int x = 0; x < Wo; x++) {
                    or_conv_neuron(in_times, T, Ci, Hi, Wi, w, Kh, Kw, stride, pad, b, o, y, x, V);
                    uint8_t tf;
                    double vk;
                    or_fire_neuron(V, T, theta, &tf, &vk);
                    size_t n = ((size_t)(b * Co + o) * Ho + y) * Wo + x;
                    out_times[n] = tf;
                    out_vkey[n] = (float)vk;
                    if (potentials)
                        for (int t = 0; t < T; t++)
                            potentials[(((size_t)b * T + t) * Co + o) * Ho * Wo + (size_t)y * Wo + x] =
                                (float)V[t];
                }
    free(V);
}

/* ------------------------------------------------------------------------ */
/* Pooling: §II-E.3, Eq. 3.                                                  */
/* ------------------------------------------------------------------------ */

/*
 * Max-pooling under rank-order coding keeps the neuron of the window that
 * fires earliest: out = min over the window of the input times.  Window
 * positions in the padding count as never firing.
 */
void or_pool(const uint8_t *in_times, int B, int C, int Hi, int Wi, int Kh, int Kw,
             int stride, int pad, uint8_t *out_times)
{
    int Ho = (Hi + 2 * pad - Kh) / stride + 1;
    int Wo = (Wi + 2 * pad - Kw) / stride + 1;
    for (int b = 0; b < B; b++)
        for (int c = 0; c < C; c++)
            for (int y = 0; y < Ho; y++)
                for (int x = 0; x < Wo; x++) {
                    uint8_t m = OR_NEVER;
                    for (int ky = 0; ky < Kh; ky++)
                        for (int kx = 0; kx < Kw; kx++) {
                            int iy = y * stride + ky - pad, ix = x * stride + kx - pad;
                            if (iy >= 0 && iy < Hi && ix >= 0 && ix < Wi) {
                                uint8_t v = in_times[((size_t)(b * C + c) * Hi + iy) * Wi + ix];
                                if (v < m) m = v;
                            }
                        }
                    out_times[((size_t)(b * C + c) * Ho + y) * Wo + x] = m;
                }
}

/* ------------------------------------------------------------------------ */
/* Lateral inhibition and k-WTA: §II-F.3.                                    */
/* ------------------------------------------------------------------------ */

/* (t, -v, index) order: earlier spike first, then higher potential, then lower index */
static int or_better(int ta, float va, int64_t ia, int tb, float vb, int64_t ib)
{
    if (ta != tb) return ta < tb;
    if (va != vb) return va > vb;
    return ia < ib;
}

/*
 * Pointwise lateral inhibition: at each location (b, y, x) only the neuron of
 * the map that fires first survives (ties: higher potential, then lower
 * channel); every other fired neuron there is set to NEVER.  In place.
 */
void or_inhibit(uint8_t *times, const float *vkey, int B, int C, int H, int W)
{
    for (int b = 0; b < B; b++)
        for (int y = 0; y < H; y++)
            for (int x = 0; x < W; x++) {
                int best = -1;
                for (int c = 0; c < C; c++) {
                    size_t n = ((size_t)(b * C + c) * H + y) * W + x;
                    if (times[n] == OR_NEVER) continue;
                    if (best < 0) { best = c; continue; }
                    size_t m = ((size_t)(b * C + best) * H + y) * W + x;
                    if (or_better(times[n], vkey[n], c, times[m], vkey[m], best)) best = c;
                }
                for (int c = 0; c < C; c++) {
                    size_t n = ((size_t)(b * C + c) * H + y) * W + x;
                    if (c != best) times[n] = OR_NEVER;
                }
            }
}

typedef struct {
    int32_t c, y, x, t;
    float v;
} or_winner;

/*
 * k-winners-take-all for convolution (the paper's convwta(array, radius,
 * count)).  Per sample, up to k rounds: the best remaining candidate wins
 * (earliest spike, then higher potential, then lower flat index (c*H+y)*W+x);
 * its whole map and every neuron of any map within Chebyshev distance
 * `radius` of its location stop being candidates.  Candidates are the fired
 * neurons; in readout mode (no threshold) every neuron is a candidate and
 * the rank is potential only (higher first, then lower index) with t = T-1.
 * Unused slots get c = -1.  Returns nothing; n_winners[b] is the count.
 */
void or_kwta(const uint8_t *times, const float *vkey, int B, int C, int H, int W, int T,
             int k, int radius, int readout, or_winner *winners, int32_t *n_winners)
{
    size_t per = (size_t)C * H * W;
    uint8_t *alive = (uint8_t *)malloc(per ? per : 1);
    for (int b = 0; b < B; b++) {
        const uint8_t *tb = times + b * per;
        const float *vb = vkey + b * per;
        for (size_t n = 0; n < per; n++) alive[n] = readout ? 1 : (tb[n] != OR_NEVER);
        int count = 0;
        for (int round = 0; round < k; round++) {
            int64_t best = -1;
            for (size_t n = 0; n < per; n++) {
                if (!alive[n]) continue;
                if (best < 0) { best = (int64_t)n; continue; }
                int tn = readout ? 0 : tb[n], tm = readout ? 0 : tb[best];
                if (or_better(tn, vb[n], (int64_t)n, tm, vb[best], best)) best = (int64_t)n;
            }
            if (best < 0) break;
            int c = (int)(best / ((int64_t)H * W));
            int y = (int)((best / W) % H);
            int x = (int)(best % W);
            or_winner *wn = &winners[(size_t)b * k + count];
            wn->c = c;
            wn->y = y;
            wn->x = x;
            wn->t = readout ? T - 1 : tb[best];
            wn->v = vb[best];
            count++;
            for (int cc = 0; cc < C; cc++)
                for (int yy = 0; yy < H; yy++)
                    for (int xx = 0; xx < W; xx++) {
                        int near = abs(yy - y) <= radius && abs(xx - x) <= radius;
                        if (cc == c || near) alive[((size_t)cc * H + yy) * W + xx] = 0;
                    }
        }
        n_winners[b] = count;
        for (int s = count; s < k; s++) {
            or_winner *wn = &winners[(size_t)b * k + s];
            wn->c = -1;
            wn->y = wn->x = wn->t = -1;
            wn->v = 0.0f;
        }
    }
    free(alive);
}

/* ------------------------------------------------------------------------ */
/* STDP and R-STDP: §II-F.1 Eq. 4-6, §II-F.2 Eq. 7.                          */
/* ------------------------------------------------------------------------ */

typedef struct {
    float a_causal, a_anticausal, lower, upper;
    int32_t stabilize;
} or_stdp_cfg;

/*
 * Update the weights of the winners' kernels.  For winner (b, o=c, y, x, t_post)
 * with configuration q, each synapse (ci, ky, kx) of kernel o sees the input
 * neuron at (ci, y*s+ky-p, x*s+kx-p) of sample b with spike time t_pre (NEVER
 * in the padding).  A pre spike at or before the post spike potentiates
 * (Eq. 4 first case, taken for the t_pre == t_post overlap), a later or
 * missing one depresses.  With the stabiliser, dW = A * (W - L) * (U - W)
 * (Eq. 4), without it dW = A (Eq. 5), from the weight before the update.
 * The mini-batch rule does not differ from the single-sample rule
 * (§II-F.1): every winner's dW is taken from the pre-update weights and the
 * changes are summed; then W = clamp(W + sum, L, U) (Eq. 6, read as clipping
 * the updated weight) for every weight that received a change.  All in double.
 * winner_cfg (nullable: all 0) maps winner b*k+slot to a configuration.
 * R-STDP (Eq. 7) is this same update with a reward and a punish configuration.
 */
int or_stdp_update(float *w, int Co, int Ci, int Kh, int Kw, int stride, int pad,
                   const uint8_t *in_times, int B, int Hi, int Wi,
                   const or_winner *winners, const int32_t *n_winners, int k,
                   const or_stdp_cfg *cfg, int n_cfg, const int32_t *winner_cfg)
{
    /* One clamp range per call: configurations with different bounds would
     * leave the clamp of a weight touched by both undefined. */
    for (int q = 1; q < n_cfg; q++)
        if (cfg[q].lower != cfg[0].lower || cfg[q].upper != cfg[0].upper) return -1;
    size_t nw = (size_t)Co * Ci * Kh * Kw;
    double *D = (double *)calloc(nw ? nw : 1, sizeof(double));
    uint8_t *touched = (uint8_t *)calloc(nw ? nw : 1, 1);
    double L = cfg[0].lower, U = cfg[0].upper;
    for (int b = 0; b < B; b++)
        for (int s = 0; s < n_winners[b]; s++) {
            const or_winner *wn = &winners[(size_t)b * k + s];
            const or_stdp_cfg *q = &cfg[winner_cfg ? winner_cfg[(size_t)b * k + s] : 0];
            int o = wn->c;
            for (int c = 0; c < Ci; c++)
                for (int ky = 0; ky < Kh; ky++)
                    for (int kx = 0; kx < Kw; kx++) {
                        int iy = wn->y * stride + ky - pad, ix = wn->x * stride + kx - pad;
                        int t_pre = OR_NEVER;
                        if (iy >= 0 && iy < Hi && ix >= 0 && ix < Wi)
                            t_pre = in_times[((size_t)(b * Ci + c) * Hi + iy) * Wi + ix];
                        double A = (t_pre <= wn->t) ? (double)q->a_causal : (double)q->a_anticausal;
                        size_t n = ((size_t)(o * Ci + c) * Kh + ky) * Kw + kx;
                        double W0 = (double)w[n];
                        double dW = q->stabilize ? A * (W0 - L) * (U - W0) : A;
                        D[n] += dW;
                        touched[n] = 1;
                    }
        }
    for (size_t n = 0; n < nw; n++) {
        if (!touched[n]) continue;
        double v = (double)w[n] + D[n];
        if (v > U) v = U;
        if (v < L) v = L;
        w[n] = (float)v;
    }
    free(D);
    free(touched);
    return 0;
}

/*
 * R-STDP configuration choice (§II-F.2): a winner is rewarded (configuration
 * 0) when the class of its map, c / group, equals the sample's label, and
 * punished (configuration 1) otherwise.
 */
void or_rstdp_select(const or_winner *winners, const int32_t *n_winners, int B, int k,
                     const int32_t *labels, int group, int32_t *winner_cfg)
{
    for (int b = 0; b < B; b++)
        for (int s = 0; s < k; s++) {
            const or_winner *wn = &winners[(size_t)b * k + s];
            winner_cfg[(size_t)b * k + s] =
                (s < n_winners[b] && wn->c / group == labels[b]) ? 0 : 1;
        }
}

/* ------------------------------------------------------------------------ */
/* Fully connected layer winners: §II-E.2 (FC layer), §II-F.3 (fcwta).      */
/* ------------------------------------------------------------------------ */

/*
 * k-winners-take-all for a fully connected layer (the paper's
 * fcwta(array, radius, count)).  Neurons of a sample are indexed o in [0, O).
 * Per sample, up to k rounds: the best remaining candidate wins (earliest
 * spike, then higher potential, then lower index); it and every neuron whose
 * index lies within `radius` of its index stop being candidates.  Reading:
 * the radius of fcwta measures distance along the neuron index, the one
 * dimension an FC layer has.  Candidates are the fired neurons; in readout
 * mode every neuron, ranked by potential only, reported with t = T-1.
 * Winners are reported as {c = o, y = 0, x = 0, t, v}; unused slots c = -1.
 */
void or_fc_wta(const uint8_t *times, const float *vkey, int B, int O, int T, int k, int radius,
               int readout, or_winner *winners, int32_t *n_winners)
{
    uint8_t *alive = (uint8_t *)malloc(O > 0 ? (size_t)O : 1);
    for (int b = 0; b < B; b++) {
        const uint8_t *tb = times + (size_t)b * O;
        const float *vb = vkey + (size_t)b * O;
        for (int o = 0; o < O; o++) alive[o] = readout ? 1 : (tb[o] != OR_NEVER);
        int count = 0;
        for (int round = 0; round < k; round++) {
            int best = -1;
            for (int o = 0; o < O; o++) {
                if (!alive[o]) continue;
                if (best < 0) { best = o; continue; }
                int to = readout ? 0 : tb[o], tm = readout ? 0 : tb[best];
                if (or_better(to, vb[o], o, tm, vb[best], best)) best = o;
            }
            if (best < 0) break;
            or_winner *wn = &winners[(size_t)b * k + count];
            wn->c = best;
            wn->y = 0;
            wn->x = 0;
            wn->t = readout ? T - 1 : tb[best];
            wn->v = vb[best];
            count++;
            for (int o = 0; o < O; o++)
                if (abs(o - best) <= radius) alive[o] = 0;
        }
        n_winners[b] = count;
        for (int s = count; s < k; s++) {
            or_winner *wn = &winners[(size_t)b * k + s];
            wn->c = -1;
            wn->y = wn->x = wn->t = -1;
            wn->v = 0.0f;
        }
    }
    free(alive);
}

/* ------------------------------------------------------------------------ */
/* Sparse interface: §II-B (spike indices instead of full buffers).         */
/* ------------------------------------------------------------------------ */

/*
 * A spike list holds, per sample, the flat indices (c*H + y)*W + x of the
 * neurons that fire, grouped by time step in ascending order and ascending
 * index within a step: offsets[b*(T+1) + t] is the number of spikes of sample
 * b before step t (offsets[.. + T] the total), spikes[b*cap + j] its j-th
 * spike.  Spikes past cap are counted but not stored.
 */
void or_times_to_spikes(const uint8_t *times, int B, int64_t n, int T, int cap, uint32_t *spikes,
                        int32_t *offsets)
{
    for (int b = 0; b < B; b++) {
        const uint8_t *tb = times + (size_t)b * n;
        int32_t cnt = 0;
        for (int t = 0; t < T; t++) {
            offsets[(size_t)b * (T + 1) + t] = cnt;
            for (int64_t i = 0; i < n; i++)
                if (tb[i] == t) {
                    if (cnt < cap) spikes[(size_t)b * cap + cnt] = (uint32_t)i;
                    cnt++;
                }
        }
        offsets[(size_t)b * (T + 1) + T] = cnt;
    }
}

/* The time map a spike list describes (its stored spikes only). */
void or_spikes_to_times(const uint32_t *spikes, const int32_t *offsets, int B, int64_t n, int T,
                        int cap, uint8_t *times)
{
    memset(times, OR_NEVER, (size_t)B * n);
    for (int b = 0; b < B; b++)
        for (int t = 0; t < T; t++) {
            const int32_t *ob = offsets + (size_t)b * (T + 1);
            int32_t end = ob[t + 1] < cap ? ob[t + 1] : cap;
            for (int32_t j = ob[t]; j < end; j++) {
                uint32_t i = spikes[(size_t)b * cap + j];
                if ((int64_t)i < n) times[(size_t)b * n + i] = (uint8_t)t;
            }
        }
}

/*
 * Conv + fire driven by a spike list: each stored spike of step t adds its
 * weight to every output neuron whose window holds it (the change of
 * potential at t, Eq. 2 restricted to the new arrivals); the potential is the
 * running sum of those changes over the steps, and the firing rule is that
 * of or_fire_neuron.  Work is proportional to the spikes times their fan-out.
 */
void or_conv_fire_spikes(const uint32_t *spikes, const int32_t *offsets, int cap, int B, int T,
                         int Ci, int Hi, int Wi, const float *w, int Co, int Kh, int Kw, int stride,
                         int pad, double theta, uint8_t *out_times, float *out_vkey)
{
    int Ho = (Hi + 2 * pad - Kh) / stride + 1;
    int Wo = (Wi + 2 * pad - Kw) / stride + 1;
    size_t per_t = (size_t)Co * Ho * Wo;
    double *dV = (double *)malloc(sizeof(double) * T * per_t);
    double *V = (double *)malloc(sizeof(double) * T);
    for (int b = 0; b < B; b++) {
        memset(dV, 0, sizeof(double) * T * per_t);
        const int32_t *ob = offsets + (size_t)b * (T + 1);
        for (int t = 0; t < T; t++) {
            int32_t end = ob[t + 1] < cap ? ob[t + 1] : cap;
            for (int32_t j = ob[t]; j < end; j++) {
                uint32_t i = spikes[(size_t)b * cap + j];
                if ((int64_t)i >= (int64_t)Ci * Hi * Wi) continue;
                int c = (int)(i / (uint32_t)(Hi * Wi));
                int iy = (int)(i / (uint32_t)Wi) % Hi, ix = (int)(i % (uint32_t)Wi);
                for (int ky = 0; ky < Kh; ky++) {
                    int ny = iy + pad - ky;
                    if (ny < 0 || ny % stride) continue;
                    int y = ny / stride;
                    if (y >= Ho) continue;
                    for (int kx = 0; kx < Kw; kx++) {
                        int nx = ix + pad - kx;
                        if (nx < 0 || nx % stride) continue;
                        int x = nx / stride;
                        if (x >= Wo) continue;
                        for (int o = 0; o < Co; o++)
                            dV[t * per_t + ((size_t)o * Ho + y) * Wo + x] +=
                                (double)w[(((size_t)o * Ci + c) * Kh + ky) * Kw + kx];
                    }
                }
            }
        }
        for (size_t q = 0; q < per_t; q++) {
            double acc = 0.0;
            for (int t = 0; t < T; t++) {
                acc += dV[t * per_t + q];
                V[t] = acc;
            }
            uint8_t tf;
            double vk;
            or_fire_neuron(V, T, theta, &tf, &vk);
            out_times[(size_t)b * per_t + q] = tf;
            out_vkey[(size_t)b * per_t + q] = (float)vk;
        }
    }
    free(V);
    free(dV);
}

/* ------------------------------------------------------------------------ */
/* Steps around the hot path in the example network of §IV.                 */
/* ------------------------------------------------------------------------ */

/* Weak filter responses are silenced before coding: x <= threshold -> value. */
void or_threshold(float *x, int64_t n, float threshold, float value)
{
    for (int64_t i = 0; i < n; i++)
        if (!(x[i] > threshold)) x[i] = value;
}

/* Trained weights binarized: below mid -> lower, otherwise upper. */
void or_quantize(float *w, int64_t n, float lower, float mid, float upper)
{
    for (int64_t i = 0; i < n; i++) w[i] = w[i] < mid ? lower : upper;
}

/* A neuron's feature: how many of the T cumulative frames have it on. */
void or_gather(const uint8_t *times, int64_t n, int T, float *out)
{
    for (int64_t i = 0; i < n; i++) {
        int on = 0;
        for (int t = 0; t < T; t++)
            if (times[i] <= t) on++;
        out[i] = (float)on;
    }
}

/* ------------------------------------------------------------------------ */
/* Rate coding (§II-D.1) and the rate-coded network (§II-E.3, §III-D).      */
/* ------------------------------------------------------------------------ */

/*
 * Per sample, the firing probability of a value is its ratio to the
 * sample's largest value (values <= min_value never fire); at each step the
 * neuron fires when that step's uniform draw u (an input, B x T x n) is below
 * it.  Frames are B x T x n, one per step, not cumulative.
 */
void or_rate_code(const float *x, const float *u, int B, int64_t n, int T, float min_value,
                  uint8_t *frames)
{
    for (int b = 0; b < B; b++) {
        const float *xb = x + (size_t)b * n;
        float xmax = 0.0f;
        int any = 0;
        for (int64_t i = 0; i < n; i++)
            if (xb[i] > min_value && (!any || xb[i] > xmax)) {
                xmax = xb[i];
                any = 1;
            }
        for (int t = 0; t < T; t++)
            for (int64_t i = 0; i < n; i++) {
                float p = (any && xb[i] > min_value) ? xb[i] / xmax : 0.0f;
                size_t at = ((size_t)b * T + t) * n + i;
                frames[at] = u[at] < p ? 1 : 0;
            }
    }
}

/*
 * Integrate-and-fire over rate-coded frames: the potential adds each step's
 * input current (Eq. 2 on that step's frame); when it exceeds theta the
 * neuron fires at that step and its potential returns to zero.  out_frames
 * B x T x Co x Ho x Wo, counts B x Co x Ho x Wo (spikes per neuron).
 */
void or_conv_if_rate(const uint8_t *frames, int B, int T, int Ci, int Hi, int Wi, const float *w,
                     int Co, int Kh, int Kw, int stride, int pad, double theta,
                     uint8_t *out_frames, int32_t *counts)
{
    int Ho = (Hi + 2 * pad - Kh) / stride + 1;
    int Wo = (Wi + 2 * pad - Kw) / stride + 1;
    for (int b = 0; b < B; b++)
        for (int o = 0; o < Co; o++)
            for (int y = 0; y < Ho; y++)
                for (int x = 0; x < Wo; x++) {
                    double V = 0.0;
                    int32_t cnt = 0;
                    for (int t = 0; t < T; t++) {
                        const uint8_t *f = frames + ((size_t)b * T + t) * Ci * Hi * Wi;
                        double I = 0.0;
                        for (int c = 0; c < Ci; c++)
                            for (int ky = 0; ky < Kh; ky++)
                                for (int kx = 0; kx < Kw; kx++) {
                                    int iy = y * stride + ky - pad, ix = x * stride + kx - pad;
                                    if (iy < 0 || iy >= Hi || ix < 0 || ix >= Wi) continue;
                                    if (f[((size_t)c * Hi + iy) * Wi + ix])
                                        I += (double)w[(((size_t)o * Ci + c) * Kh + ky) * Kw + kx];
                                }
                        V += I;
                        uint8_t s = 0;
                        if (V > theta) {
                            s = 1;
                            V = 0.0;
                            cnt++;
                        }
                        out_frames[(((size_t)b * T + t) * Co + o) * Ho * Wo + (size_t)y * Wo + x] = s;
                    }
                    counts[((size_t)(b * Co + o) * Ho + y) * Wo + x] = cnt;
                }
}

/*
 * Rate-based max pooling: each window passes on the spike train of its
 * neuron with the most spikes (the first in row-major order among equals);
 * padding holds no neuron, and a window with none gives an empty train.
 */
void or_rate_pool(const uint8_t *in_frames, const int32_t *in_counts, int B, int T, int C, int Hi,
                  int Wi, int Kh, int Kw, int stride, int pad, uint8_t *out_frames,
                  int32_t *out_counts)
{
    int Ho = (Hi + 2 * pad - Kh) / stride + 1;
    int Wo = (Wi + 2 * pad - Kw) / stride + 1;
    for (int b = 0; b < B; b++)
        for (int c = 0; c < C; c++)
            for (int y = 0; y < Ho; y++)
                for (int x = 0; x < Wo; x++) {
                    int by = -1, bx = -1;
                    int32_t best = -1;
                    for (int ky = 0; ky < Kh; ky++)
                        for (int kx = 0; kx < Kw; kx++) {
                            int iy = y * stride + ky - pad, ix = x * stride + kx - pad;
                            if (iy < 0 || iy >= Hi || ix < 0 || ix >= Wi) continue;
                            int32_t v = in_counts[((size_t)(b * C + c) * Hi + iy) * Wi + ix];
                            if (v > best) {
                                best = v;
                                by = iy;
                                bx = ix;
                            }
                        }
                    out_counts[((size_t)(b * C + c) * Ho + y) * Wo + x] = best < 0 ? 0 : best;
                    for (int t = 0; t < T; t++) {
                        uint8_t s = 0;
                        if (by >= 0)
                            s = in_frames[(((size_t)b * T + t) * C + c) * Hi * Wi + (size_t)by * Wi + bx];
                        out_frames[(((size_t)b * T + t) * C + c) * Ho * Wo + (size_t)y * Wo + x] = s;
                    }
                }
}

/* The fire step alone over dense potentials B x T x n (§II-E, §II-D.3): the
 * rule of or_fire_neuron applied to each neuron's potentials. */
void or_fire(const float *V, int B, int T, int64_t n, double theta, uint8_t *out_times, float *out_vkey)
{
    double *v = (double *)malloc(sizeof(double) * T);
    for (int b = 0; b < B; b++)
        for (int64_t i = 0; i < n; i++) {
            for (int t = 0; t < T; t++) v[t] = (double)V[((size_t)b * T + t) * n + i];
            uint8_t tf;
            double vk;
            or_fire_neuron(v, T, theta, &tf, &vk);
            out_times[(size_t)b * n + i] = tf;
            out_vkey[(size_t)b * n + i] = (float)vk;
        }
    free(v);
}
