/*
 * sanitize_driver.c -- TEST INFRASTRUCTURE: runs every function of the
 * oracle (spk_oracle.c, compiled into this program) on small seeded inputs
 * and edge cases, in exactly sized heap buffers, so that a build with
 * -fsanitize=address,undefined reports any out-of-bounds access, use of
 * freed memory, leak or undefined arithmetic.  It checks memory safety only;
 * the values are pinned by the Python tests.  Exit status 0 = every call ran.
 */
#include <stdio.h>

#include "spk_oracle.c"

static uint64_t g_state = 13659;

static uint32_t rnd(void)
{
    g_state = g_state * 6364136223846793005ull + 1442695040888963407ull;
    return (uint32_t)(g_state >> 33);
}

static float rndf(void) { return (float)(rnd() & 0xffffff) / 16777216.0f; }

static void *xmalloc(size_t n)
{
    void *p = malloc(n ? n : 1);
    if (!p) {
        fprintf(stderr, "out of memory\n");
        exit(2);
    }
    return p;
}

/* uint8 time map: fires with probability dens at a uniform step of [0, T). */
static uint8_t *times_map(size_t n, int T, float dens)
{
    uint8_t *t = (uint8_t *)xmalloc(n);
    for (size_t i = 0; i < n; i++) t[i] = rndf() < dens ? (uint8_t)(rnd() % (uint32_t)T) : OR_NEVER;
    return t;
}

static float *floats(size_t n, float lo, float hi)
{
    float *x = (float *)xmalloc(n * sizeof(float));
    for (size_t i = 0; i < n; i++) x[i] = lo + (hi - lo) * rndf();
    return x;
}

static void run_dog(int B, int C, int H, int W, int pad)
{
    int ks[3] = {3, 7, 13};
    double s1[3] = {3.0 / 7, 1.0, 13.0 / 7}, s2[3] = {6.0 / 7, 2.0, 26.0 / 7};
    int F = pad >= 0 ? 1 : 3;
    if (pad >= 0) ks[0] = 7;
    int K = ks[0];
    int Ho = pad < 0 ? H : H + 2 * pad - K + 1, Wo = pad < 0 ? W : W + 2 * pad - K + 1;
    uint8_t *img = (uint8_t *)xmalloc((size_t)B * C * H * W);
    for (size_t i = 0; i < (size_t)B * C * H * W; i++) img[i] = (uint8_t)rnd();
    float *out = (float *)xmalloc(sizeof(float) * B * C * F * Ho * Wo);
    float *k = (float *)xmalloc(sizeof(float) * 13 * 13);
    or_dog_kernel(13, 1.5, 3.0, k);
    or_dog_filter(img, B, C, H, W, ks, s1, s2, F, pad, out);
    free(k);
    free(out);
    free(img);
}

static void run_code(int B, int64_t n, int T, int mode, int flat)
{
    float *x = floats((size_t)B * n, -0.2f, 1.0f);
    if (flat)
        for (int64_t i = 0; i < B * n; i++) x[i] = 0.5f;
    if (n > 3) {
        x[0] = NAN;
        x[1] = INFINITY;
        x[2] = -0.0f;
    }
    uint8_t *t = (uint8_t *)xmalloc((size_t)B * n);
    uint8_t *fr = (uint8_t *)xmalloc((size_t)B * T * n);
    uint8_t *back = (uint8_t *)xmalloc((size_t)B * n);
    or_latency_code(x, B, n, T, 0.01f, mode, t);
    or_times_to_frames(t, B, T, n, fr);
    or_frames_to_times(fr, B, T, n, back);
    free(back);
    free(fr);
    free(t);
    free(x);
}

static void run_conv(int B, int Ci, int Hi, int Wi, int Co, int K, int s, int p, int T, double theta,
                     float dens)
{
    int Ho = (Hi + 2 * p - K) / s + 1, Wo = (Wi + 2 * p - K) / s + 1;
    size_t nin = (size_t)B * Ci * Hi * Wi, nout = (size_t)B * Co * Ho * Wo;
    uint8_t *tin = times_map(nin, T, dens);
    float *w = floats((size_t)Co * Ci * K * K, -0.2f, 1.0f);
    uint8_t *tf = (uint8_t *)xmalloc(nout), *tf2 = (uint8_t *)xmalloc(nout);
    float *vk = (float *)xmalloc(nout * sizeof(float)), *vk2 = (float *)xmalloc(nout * sizeof(float));
    float *V = (float *)xmalloc(nout * T * sizeof(float));
    or_conv_fire(tin, B, T, Ci, Hi, Wi, w, Co, K, K, s, p, theta, tf, vk, V);
    double *Vn = (double *)xmalloc(sizeof(double) * T);
    uint8_t t1;
    double v1;
    or_conv_neuron(tin, T, Ci, Hi, Wi, w, K, K, s, p, B - 1, Co - 1, Ho - 1, Wo - 1, Vn);
    or_fire_neuron(Vn, T, theta, &t1, &v1);
    free(Vn);
    or_fire(V, B, T, (int64_t)Co * Ho * Wo, theta, tf2, vk2);
    /* spike lists, full and truncated, and the event-form conv */
    int64_t n = (int64_t)Ci * Hi * Wi;
    for (int cap_div = 1; cap_div <= 3; cap_div += 2) {
        int cap = (int)(n / cap_div);
        uint32_t *sp = (uint32_t *)xmalloc(sizeof(uint32_t) * (size_t)B * (cap ? cap : 1));
        int32_t *off = (int32_t *)xmalloc(sizeof(int32_t) * (size_t)B * (T + 1));
        uint8_t *back = (uint8_t *)xmalloc(nin);
        or_times_to_spikes(tin, B, n, T, cap, sp, off);
        or_spikes_to_times(sp, off, B, n, T, cap, back);
        or_conv_fire_spikes(sp, off, cap, B, T, Ci, Hi, Wi, w, Co, K, K, s, p, theta, tf2, vk2);
        free(back);
        free(off);
        free(sp);
    }
    /* pooling of the output, inhibition, winners, learning */
    int Hp = (Ho - 2) / 2 + 1, Wp = (Wo - 2) / 2 + 1;
    if (Ho >= 2 && Wo >= 2) {
        uint8_t *pl = (uint8_t *)xmalloc((size_t)B * Co * Hp * Wp);
        or_pool(tf, B, Co, Ho, Wo, 2, 2, 2, 0, pl);
        free(pl);
    }
    uint8_t *pl1 = (uint8_t *)xmalloc(nout);
    or_pool(tf, B, Co, Ho, Wo, 3, 3, 1, 1, pl1);
    free(pl1);
    int k = 5;
    or_winner *win = (or_winner *)xmalloc(sizeof(or_winner) * B * k);
    int32_t *nw = (int32_t *)xmalloc(sizeof(int32_t) * B);
    or_inhibit(tf, vk, B, Co, Ho, Wo);
    or_kwta(tf, vk, B, Co, Ho, Wo, T, k, 1, 0, win, nw);
    or_kwta(tf, vk, B, Co, Ho, Wo, T, k, 0, 1, win, nw);
    int32_t *labels = (int32_t *)xmalloc(sizeof(int32_t) * B), *wc = (int32_t *)xmalloc(sizeof(int32_t) * B * k);
    for (int b = 0; b < B; b++) labels[b] = (int32_t)(rnd() % 3);
    or_rstdp_select(win, nw, B, k, labels, 2, wc);
    or_stdp_cfg cfg[2] = {{0.004f, -0.003f, 0.0f, 1.0f, 1}, {-0.0005f, 0.004f, 0.0f, 1.0f, 0}};
    or_stdp_update(w, Co, Ci, K, K, s, p, tin, B, Hi, Wi, win, nw, k, cfg, 2, wc);
    or_stdp_update(w, Co, Ci, K, K, s, p, tin, B, Hi, Wi, win, nw, k, cfg, 1, NULL);
    or_fc_wta(tf, vk, B, Co * Ho * Wo, T, k, 2, 0, win, nw);
    or_fc_wta(tf, vk, B, Co * Ho * Wo, T, k, 0, 1, win, nw);
    float *feat = (float *)xmalloc(nout * sizeof(float));
    or_gather(tf, (int64_t)nout, T, feat);
    or_threshold(vk, (int64_t)nout, 0.5f, 0.0f);
    or_quantize(w, (int64_t)Co * Ci * K * K, 0.0f, 0.5f, 1.0f);
    free(feat);
    free(wc);
    free(labels);
    free(nw);
    free(win);
    free(V);
    free(vk2);
    free(vk);
    free(tf2);
    free(tf);
    free(w);
    free(tin);
}

static void run_rate(int B, int Ci, int Hi, int Wi, int Co, int K, int p, int T)
{
    int64_t n = (int64_t)Ci * Hi * Wi;
    float *x = floats((size_t)B * n, -0.1f, 1.0f);
    float *u = floats((size_t)B * T * n, 0.0f, 1.0f);
    uint8_t *fr = (uint8_t *)xmalloc((size_t)B * T * n);
    or_rate_code(x, u, B, n, T, 0.01f, fr);
    int Ho = Hi + 2 * p - K + 1, Wo = Wi + 2 * p - K + 1;
    float *w = floats((size_t)Co * Ci * K * K, 0.0f, 1.0f);
    size_t no = (size_t)B * Co * Ho * Wo;
    uint8_t *fo = (uint8_t *)xmalloc(no * T);
    int32_t *cnt = (int32_t *)xmalloc(no * sizeof(int32_t));
    or_conv_if_rate(fr, B, T, Ci, Hi, Wi, w, Co, K, K, 1, p, 1.5, fo, cnt);
    int Hp = (Ho - 2) / 2 + 1, Wp = (Wo - 2) / 2 + 1;
    uint8_t *fp = (uint8_t *)xmalloc((size_t)B * T * Co * Hp * Wp);
    int32_t *cp = (int32_t *)xmalloc(sizeof(int32_t) * B * Co * Hp * Wp);
    or_rate_pool(fo, cnt, B, T, Co, Ho, Wo, 2, 2, 2, 0, fp, cp);
    free(cp);
    free(fp);
    free(cnt);
    free(fo);
    free(w);
    free(fr);
    free(u);
    free(x);
}

int main(void)
{
    run_dog(2, 1, 28, 28, -1);
    run_dog(1, 2, 9, 11, 0);
    run_dog(1, 1, 7, 7, 3);
    run_code(3, 6 * 28 * 28, 15, 0, 0);
    run_code(2, 1000, 254, 0, 1);
    run_code(2, 50, 7, 1, 0);
    run_code(1, 1, 1, 0, 0);
    run_conv(2, 3, 9, 11, 5, 3, 1, 1, 7, 2.0, 0.4f);
    run_conv(2, 4, 13, 10, 6, 4, 2, 1, 5, 1.0, 0.5f);
    run_conv(1, 2, 6, 6, 3, 5, 1, 0, 254, 3.0, 0.3f);
    run_conv(2, 6, 8, 8, 4, 3, 1, 1, 15, INFINITY, 0.6f);
    run_conv(1, 1, 3, 3, 1, 3, 3, 0, 1, -0.5, 1.0f);
    run_conv(2, 5, 7, 7, 3, 3, 1, 1, 9, 2.0, 0.0f);
    run_rate(2, 3, 9, 9, 4, 3, 1, 20);
    run_rate(1, 1, 5, 6, 2, 5, 2, 3);
    printf("oracle sanitizer driver: all calls ran\n");
    return 0;
}
