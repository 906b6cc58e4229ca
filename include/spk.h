/*
 * spk.h -- C ABI of libspk, the MI355X (gfx950) hot path of convolutional
 * spiking networks as described in Spyker (Shirsavar & Dehaqani, arXiv
 * 2301.13659): DoG filtering, rank-order latency coding, spiking convolution
 * with integrate-and-fire, spike-time pooling, lateral inhibition with
 * k-winners-take-all, and STDP / R-STDP.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Array arguments are DEVICE pointers owned by the caller, contiguous,
 *    in NCHW order (B x C x H x W); frame and potential arrays are BTCHW
 *    (batch, time, channel, height, width), the order of the paper's §II-A.
 *    Small descriptor arrays (spk_dog_desc, spk_stdp_config) are HOST pointers.
 *  - Spike activity is held as a uint8 first-spike-time map: entry t in
 *    [0, T) means the neuron fires at step t and, frames being cumulative
 *    (§II-D.3), stays on in every later frame; SPK_NEVER (255) means it never
 *    fires.  Hence T <= SPK_MAX_T (254).
 *  - The library never allocates device memory and never synchronises.  Calls
 *    that need scratch take a caller workspace (ws, ws_bytes) sized by the
 *    matching *_workspace_size query; ws may be NULL when that size is 0.  A
 *    workspace must be 256-byte aligned (hipMalloc's and torch's are);
 *    SPK_E_ARG otherwise.
 *  - Every call enqueues its kernels on `stream` (a hipStream_t; NULL is the
 *    null stream) and returns before they run.  Faults of the kernels surface
 *    at the caller's next synchronisation.
 *  - All arguments are validated on the host before anything is launched.  A
 *    call that returns anything but SPK_OK or SPK_E_HIP has launched nothing
 *    and touched no memory; spk_last_error() (per thread) then describes why.
 *    SPK_E_HIP means a launch failed after earlier kernels of the call may
 *    already have been enqueued.
 *  - Outputs may not alias inputs unless a call says so.
 */
#ifndef SPK_H
#define SPK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPK_NEVER 255
#define SPK_MAX_T 254

typedef enum {
    SPK_OK = 0,
    SPK_E_ARG = 1,          /* NULL pointer, non-positive size, bad enum   */
    SPK_E_SHAPE = 2,        /* derived size <= 0, T out of range, size limit */
    SPK_E_UNSUPPORTED = 3,  /* dtype or parameter combination not supported */
    SPK_E_WORKSPACE = 4,    /* workspace missing or smaller than required  */
    SPK_E_HIP = 5           /* a HIP launch reported an error              */
} spk_status;

typedef enum { SPK_F32 = 0, SPK_F16 = 1 } spk_dtype;
typedef enum { SPK_CODE_RANK = 0, SPK_CODE_LINEAR = 1 } spk_code_mode;

typedef void *spk_stream; /* hipStream_t */

/* One DoG filter: odd kernel size and the two standard deviations (§II-C.1). */
typedef struct {
    int32_t ksize;
    double sigma1, sigma2;
} spk_dog_desc;

/* One k-WTA winner (§II-F.3): map c, location (y, x), spike time t, key potential v. */
typedef struct {
    int32_t c, y, x, t;
    float v;
} spk_winner;

/* One STDP configuration, the paper's STDPConfig(positive, negative, stabilize,
 * lower, upper) of §II-F.1: a_causal applies when the pre spike comes at or
 * before the post spike, a_anticausal otherwise. */
typedef struct {
    float a_causal, a_anticausal, lower, upper;
    int32_t stabilize;
} spk_stdp_config;

/* Library version string ("spk <major>.<minor> gfx950"). */
const char *spk_version(void);

/* Description of the last failure of a call made by this thread ("" if none). */
const char *spk_last_error(void);

/* Output extent of a convolution or pooling window along one axis, Eq. 2 / Eq. 3
 * (§II-E.1, §II-E.3): floor((in + 2*pad - k) / stride) + 1, or -1 when the
 * arguments give no output (k < 1, stride < 1, pad < 0 or in + 2*pad < k). */
int spk_out_extent(int in, int k, int stride, int pad);

/*
 * spk_dog_filter -- DoG feature enhancement, §II-C.1 with the shape rule of
 * §II-C.4 (Eq. 1): every one of the F filters is applied to every input
 * channel separately, giving B x (C*F) x Ho x Wo, output channel c*F + f.
 *   img      uint8 B x C x H x W (device); pixel value u is taken as u / 255.
 *   filters  F descriptors (host); each kernel is the difference of two
 *            unit-sum discrete Gaussians sampled on [-R, R]^2, R = (K-1)/2,
 *            computed in double on the host and rounded to float.
 *   pad      -1: "same" padding per filter, Ho = H, Wo = W (filters may have
 *            different sizes); >= 0: Eq. 1, Ho = H + 2*pad - K + 1, all
 *            filters must then share K.
 *   out      float B x (C*F) x Ho x Wo (device).
 * Each output is accumulated in float, window row-major, without fused
 * multiply-add, so results are reproducible bit for bit.
 * Errors: SPK_E_ARG (NULL, sizes <= 0, even or < 1 ksize, sigma <= 0),
 * SPK_E_SHAPE (ksize > 21, F > 8, or output size <= 0), SPK_E_UNSUPPORTED
 * (pad >= 0 with mixed kernel sizes).
 */
spk_status spk_dog_filter(const uint8_t *img, int B, int C, int H, int W,
                          const spk_dog_desc *filters, int F, int pad,
                          float *out, spk_stream stream);

/*
 * spk_latency_code -- rank-order (latency) coding, §II-D.2 and §II-D.3.
 * Per sample, the values above min_value (the threshold applied before
 * coding) each fire once; the rest never fire.
 *   SPK_CODE_RANK   the eligible values of the whole sample (all C*H*W
 *                   jointly) are sorted, higher first, ties to the lower flat
 *                   index; the N spikes are spread evenly over T steps: rank
 *                   r fires at floor(r*T/N).
 *   SPK_CODE_LINEAR the sort disabled: t = min(T-1, floor((1 - v/vmax)*T)) in
 *                   float, vmax the largest value of the sample.
 *   x       float B x C x H x W (device).
 *   times   uint8 B x C x H x W (device) first-spike times.
 *   frames  nullable uint8 B x T x C x H x W (device) cumulative frames.
 *   ws      workspace of spk_latency_code_workspace_size(B, C, H, W) bytes.
 * Errors: SPK_E_ARG, SPK_E_SHAPE (T < 1 or > SPK_MAX_T, C*H*W >= 2^31),
 * SPK_E_WORKSPACE.
 */
size_t spk_latency_code_workspace_size(int B, int C, int H, int W);
spk_status spk_latency_code(const float *x, int B, int C, int H, int W, int T,
                            float min_value, int mode, uint8_t *times, uint8_t *frames,
                            void *ws, size_t ws_bytes, spk_stream stream);

/*
 * spk_dog_latency_code -- the network's input stage in one call: DoG
 * filtering (§II-C.1, as spk_dog_filter) followed by rank-order coding of the
 * filter outputs (§II-D.2, as spk_latency_code with SPK_CODE_RANK), giving
 * times bit for bit equal to the two calls in sequence.
 *   img, filters, pad   as for spk_dog_filter; Ho, Wo its output extent.
 *   T, min_value        as for spk_latency_code.
 *   times    uint8 B x (C*F) x Ho x Wo (device) first-spike times.
 *   dog_out  nullable float B x (C*F) x Ho x Wo (device): also receives the
 *            filter outputs.
 *   ws       workspace of spk_dog_latency_code_workspace_size bytes (device,
 *            256-byte aligned; may be NULL when that size is 0).
 * When all F kernels fit one coefficient block (sum of K^2 <= 480), a sample
 * has at most 8192 outputs and its image fits LDS, one kernel does both steps
 * (one workgroup per sample) and the workspace size is 0; otherwise the two
 * calls run in sequence, the filter outputs held in dog_out or the workspace.
 * Errors: those of spk_dog_filter and spk_latency_code, SPK_E_WORKSPACE.
 */
size_t spk_dog_latency_code_workspace_size(int B, int C, int H, int W,
                                           const spk_dog_desc *filters, int F, int pad);
spk_status spk_dog_latency_code(const uint8_t *img, int B, int C, int H, int W,
                                const spk_dog_desc *filters, int F, int pad, int T,
                                float min_value, uint8_t *times, float *dog_out, void *ws,
                                size_t ws_bytes, spk_stream stream);

/*
 * spk_conv_fire -- spiking convolution with integrate-and-fire, §II-E.1
 * (Eq. 2 for the output size).  For every output neuron (b, o, y, x) and
 * step t, V_t = sum over c, ky, kx of W[o, c, ky, kx] * S_t[b, c, y*stride +
 * ky - pad, x*stride + kx - pad], where S_t = [in_times <= t] is frame t of
 * the cumulative input and padding is silent.  The neuron fires once, at the
 * first t with V_t > theta (§II-E.1; at most once under rank-order coding,
 * §II-B); theta = +inf never fires (readout).
 *   in_times   uint8 B x Ci x Hi x Wi (device).
 *   w          Co x Ci x Kh x Kw (device): float (SPK_F32 master weights) or
 *              IEEE half bits (SPK_F16 operand).
 *   out_times  uint8 B x Co x Ho x Wo (device): spike time, or SPK_NEVER.
 *   out_vkey   float B x Co x Ho x Wo (device): V at the spike time, or V at
 *              step T-1 for neurons that never fire (the potential that
 *              orders equal spike times in winner selection, §II-F.3).
 *   potentials nullable float B x T x Co x Ho x Wo (device): every V_t
 *              (the paper's dense interface, §II-B).
 *   ws         workspace of spk_conv_fire_workspace_size(..., theta, potentials
 *              != NULL) bytes: a padded channels-last copy of the input and
 *              the weights packed as matrix-core operands (and, for readout
 *              calls, per-split partial sums).  Its contents on entry do not
 *              matter; it holds nothing the caller needs afterwards.
 * Potentials are accumulated in float from products that are exact: binary
 * spikes times half weights, or times the two halves hi + lo of a float
 * weight (hi = half(w), lo = half(w - hi)).
 * Errors: SPK_E_ARG, SPK_E_SHAPE (T out of range, Ho or Wo <= 0),
 * SPK_E_UNSUPPORTED (w_dtype), SPK_E_WORKSPACE.
 */
size_t spk_conv_fire_workspace_size(int B, int T, int Ci, int Hi, int Wi, int Co,
                                    int Kh, int Kw, int stride, int pad, float theta,
                                    int potentials);
spk_status spk_conv_fire(const uint8_t *in_times, int B, int T, int Ci, int Hi, int Wi,
                         const void *w, spk_dtype w_dtype, int Co, int Kh, int Kw,
                         int stride, int pad, float theta,
                         uint8_t *out_times, float *out_vkey, float *potentials,
                         void *ws, size_t ws_bytes, spk_stream stream);

/*
 * spk_pool_conv_fire -- max-pooling (§II-E.3) followed by spk_conv_fire
 * (§II-E.1), the pooling done inside the convolution's own packing pass
 * rather than by a separate spk_pool call.
 *   in_times   uint8 B x Ci x H0 x W0 (device): the previous layer's map.
 *   pool_kh, pool_kw, pool_stride, pool_pad  the pooling window, as spk_pool;
 *              the layer input is B x Ci x Hi x Wi with Hi =
 *              spk_out_extent(H0, pool_kh, pool_stride, pool_pad) (Wi alike).
 *              A 1 x 1 window of stride 1 and no padding is the identity.
 *   pooled_times nullable uint8 B x Ci x Hi x Wi (device): receives the
 *              pooled map, bit-identical to spk_pool's (STDP of this layer
 *              needs it as its input).
 *   packed_w   nullable (device): B fragments of w written by
 *              spk_conv_pack_weights, which readout layers (theta = +inf)
 *              then read instead of packing w on every call.  It must
 *              describe the current w (the call may read either); other
 *              layers ignore it.
 *   w, w_dtype, Co, Kh, Kw, stride, pad, theta, out_times, out_vkey: as
 *              spk_conv_fire (no dense potentials here).
 *   ws         workspace of spk_pool_conv_fire_workspace_size(...) bytes,
 *              256-byte aligned; contents on entry do not matter.
 * Results equal spk_pool followed by spk_conv_fire bit for bit.
 * Errors: those of spk_pool and spk_conv_fire.
 */
size_t spk_pool_conv_fire_workspace_size(int B, int T, int Ci, int H0, int W0, int pool_kh,
                                         int pool_kw, int pool_stride, int pool_pad, int Co,
                                         int Kh, int Kw, int stride, int pad, float theta);
spk_status spk_pool_conv_fire(const uint8_t *in_times, int B, int T, int Ci, int H0, int W0,
                              int pool_kh, int pool_kw, int pool_stride, int pool_pad,
                              uint8_t *pooled_times, const void *w, spk_dtype w_dtype,
                              const void *packed_w, int Co, int Kh, int Kw, int stride, int pad,
                              float theta, uint8_t *out_times, float *out_vkey, void *ws,
                              size_t ws_bytes, spk_stream stream);

/*
 * spk_conv_pack_weights -- the weights of a readout layer as matrix-core B
 * fragments, for spk_pool_conv_fire's packed_w (§II-E.1: V_t = W * S_t is a
 * product with W).  A caller keeps them while w does not change and calls
 * this again after every update of w (spk_stdp_update, spk_quantize).
 *   w        Co x Ci x Kh x Kw (device), SPK_F32 or SPK_F16.
 *   packed   device buffer of spk_conv_packed_weights_size(...) bytes,
 *            16-byte aligned: for each 32-map tile and 16-tap slice of the
 *            depth (taps ordered by kernel row, then column, then channel, the
 *            channels padded to an odd multiple of 8), 64 lanes of 8 halves (lane
 *            l: map l % 32, taps 8*(l/32)..+7); float weights as two such
 *            blocks, hi = half(w) then lo = half(w - hi); padding zero.
 * Errors: SPK_E_ARG, SPK_E_UNSUPPORTED (w_dtype), SPK_E_WORKSPACE (packed
 * smaller than the size), SPK_E_SHAPE (Ci*Kh*Kw*4 above 64 KiB).
 */
size_t spk_conv_packed_weights_size(int Co, int Ci, int Kh, int Kw, spk_dtype w_dtype);
spk_status spk_conv_pack_weights(const void *w, spk_dtype w_dtype, int Co, int Ci, int Kh, int Kw,
                                 void *packed, size_t packed_bytes, spk_stream stream);

/*
 * spk_conv_fire_noalloc -- spk_conv_fire for callers that cannot allocate
 * device memory (code under stream capture, serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, results and errors as spk_conv_fire,
 * without the workspace: its scratch is a static device array of
 * SPK_CONV_FIRE_NOALLOC_MAX_BYTES that the library holds on each GPU it runs
 * on until the process ends.  The call allocates and frees nothing.
 *  - Layers whose spk_conv_fire_workspace_size exceeds the maximum are
 *    rejected with SPK_E_WORKSPACE before anything is launched (64 MiB covers
 *    every layer of the workloads here; the largest, a 200-map 5x5 readout
 *    over 250 x 5 x 5 at batch 256, needs 44.5 MiB).
 *  - The scratch of the current device is used: `stream` must belong to it.
 *    Its address is looked up on the first call on each device
 *    (hipGetSymbolAddress); a failure there is SPK_E_HIP.
 *  - Every call on one GPU shares that GPU's array: calls that overlap in
 *    time on one GPU (on different streams, or from several host threads
 *    without ordering) race and may corrupt each other's results.  Calls
 *    ordered on one stream are safe.
 */
#define SPK_CONV_FIRE_NOALLOC_MAX_BYTES ((size_t)64 << 20)
spk_status spk_conv_fire_noalloc(const uint8_t *in_times, int B, int T, int Ci, int Hi, int Wi,
                                 const void *w, spk_dtype w_dtype, int Co, int Kh, int Kw,
                                 int stride, int pad, float theta,
                                 uint8_t *out_times, float *out_vkey, float *potentials,
                                 spk_stream stream);

/*
 * spk_pool -- max-pooling of spikes under rank-order coding, §II-E.3 (Eq. 3
 * for the size): each output keeps the earliest spike of its Kh x Kw window,
 * i.e. the minimum input time; window cells in the padding never fire.
 *   in_times  uint8 B x C x Hi x Wi (device); out_times uint8 B x C x Ho x Wo.
 * Errors: SPK_E_ARG, SPK_E_SHAPE (Ho or Wo <= 0).
 */
spk_status spk_pool(const uint8_t *in_times, int B, int C, int Hi, int Wi,
                    int Kh, int Kw, int stride, int pad, uint8_t *out_times,
                    spk_stream stream);

/*
 * spk_inhibit_winners -- lateral inhibition and convolutional k-WTA, §II-F.3.
 *   pointwise  1: first keep, at every location (b, y, x), only the map that
 *              fires first (equal times: higher vkey, then lower channel);
 *              the other neurons there count as never firing.
 *   k, radius  per sample, up to k rounds: the best remaining candidate wins
 *              (earliest time, then higher vkey, then lower flat index
 *              (c*H + y)*W + x); its map and every neuron of every map within
 *              Chebyshev distance radius of (y, x) stop being candidates.
 *   readout    1 (a layer with an infinite threshold): every neuron is a
 *              candidate, ranked by vkey (higher first, then lower index),
 *              and winners report t = T-1; pointwise must then be 0.
 *   times, vkey  uint8 / float B x C x H x W (device), from spk_conv_fire.
 *   inhibited  nullable uint8 B x C x H x W (device): times after pointwise
 *              inhibition (may alias times for the in-place form).
 *   winners    spk_winner B x k (device); slots past n_winners[b] get c = -1.
 *   n_winners  int32 B (device).
 *   ws         workspace of spk_inhibit_winners_workspace_size(B, C, H, W).
 * Errors: SPK_E_ARG, SPK_E_SHAPE (H*W > 2^20, k > 4096), SPK_E_UNSUPPORTED
 * (readout with pointwise), SPK_E_WORKSPACE.
 */
size_t spk_inhibit_winners_workspace_size(int B, int C, int H, int W);
spk_status spk_inhibit_winners(const uint8_t *times, const float *vkey,
                               int B, int C, int H, int W, int T,
                               int pointwise, int k, int radius, int readout,
                               uint8_t *inhibited, spk_winner *winners, int32_t *n_winners,
                               void *ws, size_t ws_bytes, spk_stream stream);

/*
 * spk_stdp_update -- STDP (§II-F.1, Eq. 4-6) and R-STDP (§II-F.2, Eq. 7) on
 * the winners' receptive fields.  For winner slot s of sample b with map o,
 * location (y, x), time t_post and configuration q = winner_cfg[b*k + s],
 * every synapse (c, ky, kx) of kernel o sees the input neuron (b, c,
 * y*stride + ky - pad, x*stride + kx - pad) with time t_pre (SPK_NEVER in the
 * padding): t_pre <= t_post takes a_causal, otherwise a_anticausal.  With the
 * stabiliser dW = (a * (W - L)) * (U - W), without it dW = a, always from the
 * weights before the call.  The batch rule equals the single-sample rule
 * (§II-F.1): the dW of all winners are summed in float, then W = min(U,
 * max(L, W + sum)) for every weight that received a change.  The order of
 * the float sum is fixed, so repeated calls agree bit for bit: the winners
 * of map o are listed in (b ascending, slot ascending) order and taken in
 * chunks of the 1024 (b, slot) entries; within a chunk, a kernel of at
 * most 512 synapses splits its n winners into G = min(n, 1024 / synapses)
 * strided groups (winners g, g + G, g + 2G, ... of the chunk's list), sums
 * each group from zero and adds the G sums in group order; otherwise it adds
 * the winners one by one in list order.
 *   w          float Co x Ci x Kh x Kw master weights (device, in/out).
 *   w_f16      nullable IEEE-half Co x Ci x Kh x Kw (device): refreshed with
 *              the round-to-nearest-even half of every updated weight.
 *   in_times   uint8 B x Ci x Hi x Wi (device): the layer's input.
 *   winners, n_winners  from spk_inhibit_winners (device), k slots per sample.
 *   cfg        n_cfg configurations (host); all must share lower and upper.
 *   winner_cfg nullable int32 B x k (device); NULL = configuration 0.
 *   ws         workspace of spk_stdp_update_workspace_size(...) bytes.
 * Errors: SPK_E_ARG, SPK_E_SHAPE (Ci*Kh*Kw > 16384, n_cfg > 16),
 * SPK_E_UNSUPPORTED (configurations with different bounds), SPK_E_WORKSPACE.
 */
size_t spk_stdp_update_workspace_size(int Co, int Ci, int Kh, int Kw, int B, int k);
spk_status spk_stdp_update(float *w, uint16_t *w_f16, int Co, int Ci, int Kh, int Kw,
                           int stride, int pad, const uint8_t *in_times, int B, int Hi, int Wi,
                           const spk_winner *winners, const int32_t *n_winners, int k,
                           const spk_stdp_config *cfg, int n_cfg, const int32_t *winner_cfg,
                           void *ws, size_t ws_bytes, spk_stream stream);

/*
 * spk_rstdp_select -- reward / punish choice of R-STDP, §II-F.2: winner slot s
 * of sample b gets configuration 0 (reward) when its map's class c / group
 * equals labels[b], else 1 (punish); empty slots get 1 and are never used.
 *   winners B x k, n_winners B, labels int32 B, winner_cfg int32 B x k (device).
 * Errors: SPK_E_ARG.
 */
spk_status spk_rstdp_select(const spk_winner *winners, const int32_t *n_winners, int B, int k,
                            const int32_t *labels, int group, int32_t *winner_cfg,
                            spk_stream stream);

/*
 * Cumulative frames <-> first-spike times (§II-D.3, §II-B): frames is uint8
 * B x T x n (1 = on), times uint8 B x n; a neuron's time is its first on
 * frame.  spk_frames_to_times expects cumulative frames; a frame sequence
 * that switches a neuron off again is reduced to its first on frame.
 * Errors: SPK_E_ARG, SPK_E_SHAPE (T out of range).
 */
spk_status spk_frames_to_times(const uint8_t *frames, int B, int T, int64_t n,
                               uint8_t *times, spk_stream stream);
spk_status spk_times_to_frames(const uint8_t *times, int B, int T, int64_t n,
                               uint8_t *frames, spk_stream stream);

/*
 * spk_fc_fire -- fully connected layer with integrate-and-fire neurons,
 * §II-E.2: an I x O kernel over B x T x I input spikes.  For sample b,
 * neuron o and step t, V_t = sum over i of W[o, i] * [in_times[b, i] <= t];
 * the neuron fires once, at the first t with V_t > theta (theta = +inf:
 * readout, never fires).  This is spk_conv_fire with a 1 x 1 kernel over I
 * input channels on a 1 x 1 image, and has its precision and errors.
 *   in_times   uint8 B x I (device), e.g. a flattened B x C x H x W time map.
 *   w          O x I (device): float master weights or IEEE half bits.
 *   out_times  uint8 B x O; out_vkey float B x O (as spk_conv_fire).
 *   potentials nullable float B x T x O (device).
 *   ws         workspace of spk_fc_fire_workspace_size(...) bytes.
 */
size_t spk_fc_fire_workspace_size(int B, int T, int I, int O, float theta, int potentials);
spk_status spk_fc_fire(const uint8_t *in_times, int B, int T, int I, const void *w,
                       spk_dtype w_dtype, int O, float theta, uint8_t *out_times,
                       float *out_vkey, float *potentials, void *ws, size_t ws_bytes,
                       spk_stream stream);

/*
 * spk_fc_winners -- k-winners-take-all of a fully connected layer (the
 * paper's fcwta, §II-F.3).  Per sample, up to k rounds: the best remaining
 * candidate wins (earliest time, then higher vkey, then lower neuron index);
 * it and every neuron whose index is within `radius` of its index stop being
 * candidates.  Candidates are the neurons that fired; with readout = 1 every
 * neuron, ranked by vkey only, reported with t = T-1.
 *   times, vkey  uint8 / float B x O (device), from spk_fc_fire.
 *   winners      spk_winner B x k (device): {c = neuron, y = 0, x = 0, t, v};
 *                slots past n_winners[b] get c = -1.
 *   n_winners    int32 B (device).
 * Errors: SPK_E_ARG, SPK_E_SHAPE (T out of range, O > 65536, k > 4096).
 */
spk_status spk_fc_winners(const uint8_t *times, const float *vkey, int B, int O, int T,
                          int k, int radius, int readout, spk_winner *winners,
                          int32_t *n_winners, spk_stream stream);

/*
 * spk_fc_stdp_update -- STDP / R-STDP of a fully connected layer (§II-F.1,
 * §II-F.2): spk_stdp_update with a 1 x 1 kernel over I input channels; the
 * receptive field of neuron o is the whole input, w is float O x I, w_f16
 * nullable half O x I, in_times uint8 B x I, winners from spk_fc_winners.
 */
size_t spk_fc_stdp_update_workspace_size(int O, int I, int B, int k);
spk_status spk_fc_stdp_update(float *w, uint16_t *w_f16, int O, int I, const uint8_t *in_times,
                              int B, const spk_winner *winners, const int32_t *n_winners, int k,
                              const spk_stdp_config *cfg, int n_cfg, const int32_t *winner_cfg,
                              void *ws, size_t ws_bytes, spk_stream stream);

/*
 * spk_log_filter -- Laplacian-of-Gaussian bank (§II-C.3): each deviation s
 * is approximated by two DoG filters, on-centre (s/sqrt 2, s*sqrt 2) and
 * off-centre (s*sqrt 2, s/sqrt 2), applied as spk_dog_filter does (output
 * channel c*2n + 2i for the on-centre filter of stds[i], + 1 for the off one).
 *   stds   n_std deviations (host), 1 <= n_std <= 4; ksize odd; pad as in
 *          spk_dog_filter.
 * Errors: those of spk_dog_filter, SPK_E_ARG (deviation <= 0 or not finite),
 * SPK_E_SHAPE (n_std > 4).
 */
spk_status spk_log_filter(const uint8_t *img, int B, int C, int H, int W, const float *stds,
                          int n_std, int ksize, int pad, float *out, spk_stream stream);

/*
 * spk_inhibit -- pointwise lateral inhibition on its own (§II-F.3, the
 * paper's inhibit): at each location (b, y, x) only the neuron that fires
 * earliest (then the higher vkey, then the lower map) keeps its time; all
 * others become NEVER.  times, vkey B x C x H x W (device); inhibited B x C x
 * H x W, which may be times itself (in place).  One pass: 6 bytes per neuron.
 * Errors: SPK_E_ARG, SPK_E_SHAPE (C*H*W >= 2^31).
 */
spk_status spk_inhibit(const uint8_t *times, const float *vkey, int B, int C, int H, int W,
                       uint8_t *inhibited, spk_stream stream);

/*
 * spk_fire -- the fire step on its own (§II-E, firing rule of §II-D.3): over
 * dense potentials B x T x n (the dense interface's BTCHW layout, n = C*H*W),
 * per neuron the first step with V > theta and V there (else NEVER and
 * V[T-1]).  The same outputs as spk_conv_fire gives with its potentials; a
 * streaming pass that reads every step.
 * Errors: SPK_E_ARG (NULL, sizes <= 0, theta NaN), SPK_E_SHAPE (T range).
 */
spk_status spk_fire(const float *potentials, int B, int T, int64_t n, float theta,
                    uint8_t *out_times, float *out_vkey, spk_stream stream);

/*
 * spk_threshold -- in place, x = x if x > threshold else value (n floats,
 * device).  Applied to filter outputs before coding, it silences the weak
 * responses (§IV's example uses 0.01); NaN becomes value.
 */
spk_status spk_threshold(float *x, int64_t n, float threshold, float value, spk_stream stream);

/*
 * spk_quantize -- binarize trained weights (§IV): w = lower if w < mid else
 * upper, in place on the float master (n values, device), and the half copy
 * w_f16 (nullable) set to the same values.
 */
spk_status spk_quantize(float *w, uint16_t *w_f16, int64_t n, float lower, float mid, float upper,
                        spk_stream stream);

/*
 * spk_gather -- feature values of a spike output (§IV): per neuron, the
 * number of steps at which its cumulative frame is on, T - t for a neuron
 * that fired at t, else 0.  times uint8 (n, device) -> out float (n, device).
 */
spk_status spk_gather(const uint8_t *times, int64_t n, int T, float *out, spk_stream stream);

/* ---------------------------------------------------------------------- */
/* Rate coding (§II-D.1) and the rate-coded network (§II-E, §II-E.3).      */
/* Layers exchange frames B x T x C x H x W (uint8 0/1, one per step, not  */
/* cumulative) and spike counts B x C x H x W (int32).                     */
/* ---------------------------------------------------------------------- */

/*
 * spk_rate_code -- per sample, a value's firing probability is its ratio to
 * the sample's largest value (values <= min_value never fire, min_value >=
 * 0); at step t the neuron fires when u[b][t][i] < that probability.
 *   x      float B x n (device); u float B x T x n uniform draws on [0, 1)
 *          (device; the caller's random numbers); frames uint8 B x T x n.
 *   ws     B * 4 bytes (per-sample maxima).
 */
spk_status spk_rate_code(const float *x, const float *u, int B, int64_t n, int T, float min_value,
                         uint8_t *frames, void *ws, size_t ws_bytes, spk_stream stream);

/*
 * spk_conv_if_rate -- integrate-and-fire over rate-coded frames: each step
 * adds its current (Eq. 2 on that step's frame) to the potential; above
 * theta the neuron fires at that step and its potential returns to zero.
 *   frames      uint8 B x T x Ci x Hi x Wi (device).
 *   w           Co x Ci x Kh x Kw: float master (two half products) or half.
 *   out_frames  uint8 B x T x Co x Ho x Wo; counts int32 B x Co x Ho x Wo.
 *   ws          spk_conv_if_rate_workspace_size(...) bytes (a padded
 *               channels-last copy of the frames and the weight fragments).
 * Float weights are accumulated in float: exact where the sums are (integer
 * or binarized weights, halves summing below 2^13).
 * Errors: SPK_E_ARG, SPK_E_SHAPE, SPK_E_UNSUPPORTED (dtype; weight slices
 * beyond LDS), SPK_E_WORKSPACE.
 */
size_t spk_conv_if_rate_workspace_size(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh, int Kw,
                                       int stride, int pad, spk_dtype w_dtype);
spk_status spk_conv_if_rate(const uint8_t *frames, int B, int T, int Ci, int Hi, int Wi,
                            const void *w, spk_dtype w_dtype, int Co, int Kh, int Kw, int stride,
                            int pad, float theta, uint8_t *out_frames, int32_t *counts, void *ws,
                            size_t ws_bytes, spk_stream stream);

/*
 * spk_rate_pool -- rate-based max pooling (§II-E.3, Eq. 3 shapes): each
 * window passes on the frames of its neuron with the highest count (the
 * first in row-major window order among equals); padding holds no neuron.
 */
spk_status spk_rate_pool(const uint8_t *in_frames, const int32_t *in_counts, int B, int T, int C,
                         int Hi, int Wi, int Kh, int Kw, int stride, int pad, uint8_t *out_frames,
                         int32_t *out_counts, spk_stream stream);

/* spk_rate_features -- firing rates as features: out = counts / T (float). */
spk_status spk_rate_features(const int32_t *counts, int64_t n, int T, float *out, spk_stream stream);

/* ---------------------------------------------------------------------- */
/* Sparse interface (§II-B): the indices of the spikes instead of full     */
/* buffers.                                                                */
/* ---------------------------------------------------------------------- */

/*
 * A spike list of B samples over T steps:
 *   spikes   uint32 B x cap (device): for sample b, the flat neuron indices
 *            (c*H + y)*W + x of its spikes, grouped by step in ascending
 *            order and by ascending index within a step;
 *   offsets  int32 B x (T + 1) (device): offsets[b*(T+1) + t] = number of
 *            spikes of sample b before step t; the entry at T is its total.
 * A sample with more than cap spikes keeps its first cap (in that order);
 * the offsets still count all of them, so total > cap tells the caller, and
 * every consumer reads only the stored ones.  Under rank-order coding a
 * neuron fires once, so cap = C*H*W always suffices.
 */

/*
 * spk_times_to_spikes -- spike list of a time map (dense -> sparse).
 *   times  uint8 B x C x H x W (device); ws of
 *   spk_times_to_spikes_workspace_size(...) bytes (per-chunk counts).
 * Deterministic: the list is the stable sort of the spiking neurons by step.
 * Errors: SPK_E_ARG, SPK_E_SHAPE (T range, C*H*W >= 2^31, B > 65535),
 * SPK_E_WORKSPACE.
 */
size_t spk_times_to_spikes_workspace_size(int B, int C, int H, int W, int T);
spk_status spk_times_to_spikes(const uint8_t *times, int B, int C, int H, int W, int T, int cap,
                               uint32_t *spikes, int32_t *offsets, void *ws, size_t ws_bytes,
                               spk_stream stream);

/*
 * spk_spikes_to_times -- the time map of a spike list (sparse -> dense):
 * NEVER everywhere, then t at each stored spike of step t.  Indices
 * >= C*H*W are ignored; an index listed twice in one sample is invalid.
 * Errors: SPK_E_ARG, SPK_E_SHAPE (T range, C*H*W >= 2^31, B > 65535).
 */
spk_status spk_spikes_to_times(const uint32_t *spikes, const int32_t *offsets, int cap, int B,
                               int C, int H, int W, int T, uint8_t *times, spk_stream stream);

/*
 * spk_conv_fire_sparse -- spiking convolution + IF fire driven by a spike
 * list (§II-B, §II-E.1 Eq. 2, firing of §II-D.3 / §II-E): the same outputs
 * as spk_conv_fire on the list's time map (first-spike times and V_key,
 * B x Co x Ho x Wo), at a cost that follows the number of spikes times their
 * fan-out rather than B*T*Ho*Wo*Co*Ci*Kh*Kw.  theta = +inf is the readout
 * (V_key = V[T-1], nothing fires).  No dense-potential output.
 *   spikes, offsets, cap  the input spike list over Ci x Hi x Wi neurons.
 *   w      Co x Ci x Kh x Kw (device): float master or IEEE half bits; float
 *          weights are added in float, in step order and tap order
 *          ((ky, kx, c) row-major) within a step.
 *   ws     workspace of spk_conv_fire_sparse_workspace_size(...) bytes (a
 *          padded channels-last time buffer and the weight table).
 * Errors: SPK_E_ARG, SPK_E_SHAPE (T range, empty output, tensors of 2^31
 * elements, B > 65535), SPK_E_UNSUPPORTED (unknown dtype, or a weight table
 * of Kh*Kw*Ci taps x 32 maps that does not fit a block's LDS),
 * SPK_E_WORKSPACE.
 */
size_t spk_conv_fire_sparse_workspace_size(int B, int T, int Ci, int Hi, int Wi, int Co, int Kh,
                                           int Kw, int stride, int pad, spk_dtype w_dtype);
spk_status spk_conv_fire_sparse(const uint32_t *spikes, const int32_t *offsets, int cap, int B,
                                int T, int Ci, int Hi, int Wi, const void *w, spk_dtype w_dtype,
                                int Co, int Kh, int Kw, int stride, int pad, float theta,
                                uint8_t *out_times, float *out_vkey, void *ws, size_t ws_bytes,
                                spk_stream stream);

/* float -> IEEE half bits, round to nearest even (the SPK_F16 conv operand). */
spk_status spk_cast_f16(const float *x, uint16_t *y, int64_t n, spk_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* SPK_H */
