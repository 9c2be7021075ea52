/*
 * libspyke.h -- C ABI of the MI355X (gfx950) hot path for convolutional
 * spiking networks with at most one spike per neuron (Mozafari et al.,
 * "SpykeTorch", Frontiers in Neuroscience 2019).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Tensor arguments are DEVICE pointers owned by the caller, contiguous,
 *   row-major and batch-major.  The library never allocates or frees caller
 *   memory; scratch space comes from a caller-provided device `workspace`
 *   whose size the matching *_workspace_size() function returns (a NULL
 *   workspace is accepted when that size is 0).
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   All work is enqueued asynchronously on it; no call synchronises the host.
 * - Spike waves are u8 [B][T][C][H][W] holding 0/1, cumulative in t
 *   (the paper's Eq.1: S[t] = 1 from the first-spike step on).  First-spike
 *   maps are u8 [B][C][H][W] with the value T meaning "never spiked" (the
 *   paper's infinity).  Hence T <= 255.
 * - A neuron's linear index inside one image is c*H*W + y*W + x.
 * - Every function returns an int status.  Arguments are validated on the
 *   host before anything is enqueued; on an error nothing is launched,
 *   outputs are untouched, and spk_last_error() (thread-local) describes it.
 *   An asynchronous device fault surfaces at the caller's next synchronisation.
 * - Entry points are stateless and re-entrant; calls on different streams
 *   may run concurrently as long as their buffers do not overlap.
 */
#ifndef LIBSPYKE_H
#define LIBSPYKE_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define SPK_API __attribute__((visibility("default")))
#else
#define SPK_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

enum {
    SPK_OK = 0,
    SPK_E_ARG = 1,        /* NULL where a buffer is required, or a bad flag  */
    SPK_E_SHAPE = 2,      /* non-positive or inconsistent sizes              */
    SPK_E_RANGE = 3,      /* a size beyond a documented limit (T > 255, ...) */
    SPK_E_WORKSPACE = 4,  /* workspace smaller than *_workspace_size()       */
    SPK_E_INPUT = 5,      /* bad values in a host-side argument              */
    SPK_E_HIP = 6         /* a HIP launch or runtime call failed             */
};

/* Library version, (major << 16) | (minor << 8) | patch. */
SPK_API int spk_version(void);

/* Message of the last failing call on this thread ("" if none). */
SPK_API const char *spk_last_error(void);

/* ------------------------------------------------------------------------
 * Intensity-to-latency encoding (paper, section "utils Module": Filter,
 * DoGKernel/GaborKernel and Intensity2Latency; threshold as in the
 * "functional Module").
 *   image       u8  [B][H][W], pixel values 0..255.
 *   filters     f32 [C][KF][KF], KF odd, KF <= 31; same-size
 *               cross-correlation (no kernel flip), zero outside the image.
 *   intensities f32 [B][C][H][W] or NULL: filter response, with values
 *               below filter_threshold set to 0.  Accumulated in double and
 *               rounded once to float.
 *   t_first     u8  [B][C][H][W] or NULL: rank-order latency.  Per image,
 *               the n positive intensities of all channels are ranked from
 *               largest to smallest (equal values by ascending linear index)
 *               and the entry of rank rho spikes at floor(rho*T/n); other
 *               entries never spike (value T).
 *   wave        u8  [B][T][C][H][W] or NULL: Eq.1 wave of t_first.
 * Limits: 1 <= T <= 255, C*H*W < 2^31, KF <= 31, and the filters plus an
 * 8-row band of the zero-padded image, as doubles, must fit 64 KiB:
 * 8*(C*KF*KF + (7+KF)*(W+KF-1)) + 16*C <= 65536 (W <= 346 for 6 filters of 13x13).
 * Workspace: spk_encode_latency_workspace_size(B, C, H, W, T) bytes.      */
SPK_API size_t spk_encode_latency_workspace_size(int B, int C, int H, int W, int T);
SPK_API int spk_encode_latency(const uint8_t *image, int B, int H, int W,
                       const float *filters, int C, int KF, float filter_threshold, int T,
                       uint8_t *wave, uint8_t *t_first, float *intensities,
                       void *workspace, size_t ws_bytes, void *stream);

/* Rank-order code of a given intensity map (the second half of
 * spk_encode_latency, for maps prepared otherwise -- e.g. locally normalised):
 * intensities f32 [B][C][H][W] -> wave u8 [B][T][C][H][W] and/or t_first u8
 * [B][C][H][W] (either may be NULL), with the ranking of spk_encode_latency.
 * Workspace: spk_rank_latency_workspace_size(B, C, H, W, T) bytes.         */
SPK_API size_t spk_rank_latency_workspace_size(int B, int C, int H, int W, int T);
SPK_API int spk_rank_latency(const float *intensities, int B, int C, int H, int W, int T,
                             uint8_t *wave, uint8_t *t_first, void *workspace, size_t ws_bytes,
                             void *stream);

/* Local normalisation (section "functional Module": intensities normalised by
 * their regional mean; in the tutorial it sits between the filter and the
 * latency code).  A reading -- the paper gives no formula: per channel,
 *     out = in / (mean + eps),
 * mean over the (2*radius+1)^2 window centred on the entry with zero padding
 * (padding counts in the window size).  Operation order, fixed so that the
 * result is reproducible: row sums in double (dx ascending), their sum in
 * double (dy ascending), mean = float(sum / (2r+1)^2), then float mean + eps
 * and a correctly rounded float division.  intensities, out f32
 * [B][C][H][W], not overlapping.  Limits: radius >= 0 and
 * (2*radius + 1) * (12*W + 8*radius) <= 61440 (the rows of one window in LDS). */
SPK_API int spk_local_normalization(const float *intensities, int B, int C, int H, int W, int radius,
                                    float eps, float *out, void *stream);

/* Eq.1: wave u8 [B][T][C][H][W] from first-spike times u8 [B][C][H][W]
 * (values >= T never spike).  1 <= T <= 255.                               */
SPK_API int spk_expand_wave(const uint8_t *t_first, int B, int T, int C, int H, int W,
                    uint8_t *wave, void *stream);

/* Checks Eq.1's structure: writes to *bad_count (device i32) the number of
 * neurons whose entries are not 0/1 or decrease in t.                      */
SPK_API int spk_validate_wave(const uint8_t *wave, int B, int T, int C, int H, int W,
                      int32_t *bad_count, void *stream);

/* ------------------------------------------------------------------------
 * Convolution + firing (section "snn Module", Eq.2; firing from the
 * "functional Module"; infinite-threshold in-place firing, Eq.5).
 *   wave       u8  [B][T][Cin][H][W], a valid cumulative spike wave
 *              (the result is defined through its first-spike times).
 *   weight     f32 [Cout][Cin][K][K], finite.
 *   pad        zero padding of the input (padded neurons never spike);
 *              Ho = H + 2*pad - K + 1, Wo = W + 2*pad - K + 1 (stride 1).
 *   threshold  finite: spike at step t iff P[t] >= threshold;
 *              +INFINITY: Eq.5 -- P[t] = 0 for t < T-1, spike only at
 *              t = T-1 and only where P[T-1] > 0.
 *   potentials f32 [B][T][Cout][Ho][Wo] or NULL:
 *              P[t,f,y,x] = sum over (ci,ky,kx) of W[f,ci,ky,kx] * S[t,ci,y+ky-pad,x+kx-pad].
 *              Computed on 16-bit matrix cores with float accumulation:
 *              each weight, scaled by a power of two, becomes the sum of
 *              two 16-bit terms whose type is chosen per call on the device
 *              from the layer's largest and smallest non-zero |w| -- fp16
 *              (each weight within 2^-22 of itself) when every non-zero |w|
 *              is at least 2^-15 times the largest one's power of two, else
 *              bf16 (each weight within 2^-17 of itself, exactly when it has
 *              at most 17 significant bits; every float weight when
 *              max|w| < 2^8).  Products with spikes are exact and the
 *              scaling is undone exactly.  Repeated calls give the same
 *              bits; the accumulation order depends on the call's size (in
 *              Eq.5 mode a small batch's sum is split into parts added in
 *              order), so one image's potentials may differ in the last bits
 *              between batch sizes.
 *   spikes     u8  [B][T][Cout][Ho][Wo] or NULL: 1 where the neuron fires.
 *   t_first    u8  [B][Cout][Ho][Wo]: first firing step, T if silent.
 *   v_first    f32 [B][Cout][Ho][Wo]: potential at t_first, 0 if silent.
 * Limits: 1 <= T <= 255, Ho, Wo >= 1, Ho*Wo <= 2^26, Cout <= 4096,
 * K*K*CP <= 16384 and (W+2*pad)*CP <= 32768 where CP is Cin rounded up to 4
 * (Cin <= 4) or to a multiple of 8, and B*(H+2*pad)*(W+2*pad)*CP < 2^32.
 * Workspace: spk_conv_fire_workspace_size(...) bytes.                      */
SPK_API size_t spk_conv_fire_workspace_size(int B, int T, int Cin, int H, int W, int Cout, int K, int pad);
SPK_API int spk_conv_fire(const uint8_t *wave, int B, int T, int Cin, int H, int W,
                  const float *weight, int Cout, int K, int pad, float threshold,
                  float *potentials, uint8_t *spikes, uint8_t *t_first, float *v_first,
                  void *workspace, size_t ws_bytes, void *stream);

/* The same call with the input given by its first-spike map (Eq.1: the
 * wave is 1 at step t exactly where t >= t_first), which is what the
 * contraction consumes; it saves reading the T planes of the wave.
 *   in_t_first u8 [B][Cin][H][W], values in [0, T] (T = never; larger
 *   values count as T).  Outputs, limits, workspace and errors as
 *   spk_conv_fire.                                                          */
SPK_API int spk_conv_fire_first_spike(const uint8_t *in_t_first, int B, int T, int Cin, int H, int W,
             const float *weight, int Cout, int K, int pad, float threshold,
             float *potentials, uint8_t *spikes, uint8_t *t_first, float *v_first,
             void *workspace, size_t ws_bytes, void *stream);

/* The same call for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * no workspace argument, the scratch is a static device array of
 * 64 MiB per GPU inside the library, held until the process ends, and the
 * call allocates nothing.  A call whose spk_conv_fire_workspace_size()
 * exceeds 64 MiB returns SPK_E_RANGE with nothing launched.  Every call on
 * one GPU shares that GPU's scratch: calls that overlap in time on one GPU
 * (concurrent streams, or threads) race and must be serialised by the
 * caller.  Arguments, outputs and errors otherwise as
 * spk_conv_fire_first_spike.                                                */
SPK_API int spk_conv_fire_first_spike_noalloc(const uint8_t *in_t_first, int B, int T, int Cin, int H, int W,
             const float *weight, int Cout, int K, int pad, float threshold,
             float *potentials, uint8_t *spikes, uint8_t *t_first, float *v_first, void *stream);

/* The same call as spk_conv_fire_first_spike with the contraction on fp32
 * matrix cores (v_mfma_f32_16x16x4_f32): each fp32 weight is one term, each
 * product with a spike exact, fp32 accumulation -- the dense fp32 form of the
 * time-parallel convolution, kept as the alternative the 16-bit split is
 * measured against.  threshold must be finite (SPK_E_ARG otherwise); all else
 * as spk_conv_fire_first_spike.                                             */
SPK_API int spk_conv_fire_first_spike_f32mfma(const uint8_t *in_t_first, int B, int T, int Cin, int H, int W,
             const float *weight, int Cout, int K, int pad, float threshold,
             float *potentials, uint8_t *spikes, uint8_t *t_first, float *v_first,
             void *workspace, size_t ws_bytes, void *stream);

/* One layer in one launch: convolution + firing (as
 * spk_conv_fire_first_spike) with the first-spike max-pooling of its output
 * (section "snn Module", Pooling, Eq.3, with window = stride = pool and no
 * padding) fused into it, so that the layer's first-spike map is pooled
 * while it is still on chip (the batching and fewer-round-trips direction of
 * the paper's conclusions).
 *   in_t_first      u8 [B][Cin][H][W], the layer input's first-spike map.
 *   pool            pooling window and stride, >= 1, with pool <= Ho, Wo and
 *                   pool * Wo <= 256 (128 when Ho*Wo is not a multiple of 4
 *                   or an output is not 16-byte aligned).
 *   threshold       finite (Eq.5 mode has no fused form).
 *   potentials, spikes   as spk_conv_fire, or NULL (the compact form).
 *   t_first, v_first     required, as spk_conv_fire.
 *   pooled_t_first  u8 [B][Cout][Ho/pool][Wo/pool] (floor): the earliest
 *                   first spike of each window, T if none -- spk_pool_first_spike
 *                   of t_first with (pool, pool, 0).
 *   pooled_wave     u8 [B][T][Cout][Ho/pool][Wo/pool] or NULL: its Eq.1 wave.
 * Work is cut into bands of whole pooling rows of one image; every output
 * neuron's sum runs in the same order as in spk_conv_fire_first_spike, so
 * all outputs equal that call's (and spk_pool_first_spike's).  Workspace:
 * spk_conv_fire_workspace_size(...) bytes.  Errors as spk_conv_fire, plus
 * SPK_E_ARG for an infinite threshold or a NULL pooled_t_first, SPK_E_SHAPE
 * for a window larger than the map and SPK_E_RANGE for a band that exceeds
 * the limit above.                                                          */
SPK_API int spk_conv_fire_pool(const uint8_t *in_t_first, int B, int T, int Cin, int H, int W,
             const float *weight, int Cout, int K, int pad, float threshold, int pool,
             float *potentials, uint8_t *spikes, uint8_t *t_first, float *v_first,
             uint8_t *pooled_t_first, uint8_t *pooled_wave, void *workspace, size_t ws_bytes, void *stream);

/* Convolution + firing with stride > 1 (section "snn Module" names strides
 * above 1 as the next version's feature): output neuron (y, x) reads the
 * zero-padded input window whose top-left corner is (y*stride, x*stride),
 *   P[t,f,y,x] = sum over (ci,ky,kx) of W[f,ci,ky,kx] * S[t,ci,y*stride+ky-pad,x*stride+kx-pad],
 * and Eq.2 becomes Ho = floor((H + 2*pad - K) / stride) + 1 (likewise Wo).
 *   stride  1..64 (1 is spk_conv_fire / spk_conv_fire_first_spike).
 * Everything else -- arguments, firing, Eq.5 mode, the weight terms, limits,
 * errors -- as spk_conv_fire (the wave form) and spk_conv_fire_first_spike
 * (the first-spike form).  Workspace:
 * spk_conv_fire_strided_workspace_size(...) bytes.                          */
SPK_API size_t spk_conv_fire_strided_workspace_size(int B, int T, int Cin, int H, int W, int Cout, int K,
             int stride, int pad);
SPK_API int spk_conv_fire_strided(const uint8_t *wave, int B, int T, int Cin, int H, int W,
             const float *weight, int Cout, int K, int stride, int pad, float threshold,
             float *potentials, uint8_t *spikes, uint8_t *t_first, float *v_first,
             void *workspace, size_t ws_bytes, void *stream);
SPK_API int spk_conv_fire_first_spike_strided(const uint8_t *in_t_first, int B, int T, int Cin, int H, int W,
             const float *weight, int Cout, int K, int stride, int pad, float threshold,
             float *potentials, uint8_t *spikes, uint8_t *t_first, float *v_first,
             void *workspace, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Spike max-pooling (section "snn Module", Eq.3): on a spike wave each
 * window yields its earliest spike.  Window `kernel`, stride `stride`,
 * zero padding `pad`; Ho = floor((H + 2*pad - kernel)/stride) + 1.
 *   out_wave    u8 [B][T][C][Ho][Wo]
 *   out_t_first u8 [B][C][Ho][Wo] or NULL (T where the window never spikes). */
SPK_API int spk_pool(const uint8_t *wave, int B, int T, int C, int H, int W,
             int kernel, int stride, int pad,
             uint8_t *out_wave, uint8_t *out_t_first, void *stream);

/* The same pooling computed from first-spike times: t_first u8 [B][C][H][W]
 * (values >= T never spike) -> out_t_first u8 [B][C][Ho][Wo] = minimum over
 * the window (T where nothing spikes), and out_wave (or NULL) its Eq.1 wave
 * u8 [B][T][C][Ho][Wo].  For a valid cumulative wave this equals spk_pool on
 * that wave (the earliest spike of a window is the minimum first-spike
 * time), while reading one byte per input neuron instead of T.            */
SPK_API int spk_pool_first_spike(const uint8_t *t_first, int B, int T, int C, int H, int W,
                                 int kernel, int stride, int pad,
                                 uint8_t *out_wave, uint8_t *out_t_first, void *stream);

/* Max-pooling of potentials (section "snn Module": pooling a potentials
 * tensor keeps the largest potential of each window).  potentials f32
 * [B][T][C][H][W] -> out f32 [B][T][C][Ho][Wo], Ho = (H + 2*pad - kernel) /
 * stride + 1.  Zero padding: a padded element is a potential of +0 and takes
 * part in the maximum; of equal values the first in row-major window order
 * is kept.  out must not overlap potentials.                               */
SPK_API int spk_pool_potentials(const float *potentials, int B, int T, int C, int H, int W,
                                int kernel, int stride, int pad, float *out, void *stream);

/* ------------------------------------------------------------------------
 * Pointwise inhibition (section "functional Module": at each location only
 * the neuron of the most salient feature may spike -- the earliest spike,
 * then the highest potential; ties go to the lower feature index, as in
 * spk_kwta).  In: t_first u8 and v_first f32 [B][C][H][W] (t_first >= T:
 * silent).  Out: out_t_first / out_v_first [B][C][H][W] keep the winner of
 * each location and make every other feature silent (T, 0); a location
 * where nothing spikes stays silent.  They may alias the inputs.  Optional
 * (NULL to skip): out_wave u8 [B][T][C][H][W], the Eq.1 wave of out_t_first;
 * potentials f32 [B][T][C][H][W], masked in place: every value of a feature
 * that is not its location's winner becomes 0.  Limits: T <= 255.          */
SPK_API int spk_pointwise_inhibition(const uint8_t *t_first, const float *v_first, int B, int T, int C,
                                     int H, int W, uint8_t *out_t_first, float *out_v_first,
                                     uint8_t *out_wave, float *potentials, void *stream);

/* ------------------------------------------------------------------------
 * k winners-take-all with feature-wise and lateral inhibition (sections
 * "snn Module" and "functional Module": get_k_winners).  Eligible neurons
 * have t_first < T.  Up to k times: the eligible, uninhibited neuron with
 * the earliest t_first, then the largest v_first, then the lowest linear
 * index wins; its whole feature map is inhibited, and so is every position
 * within Chebyshev distance `radius` of it in all maps.
 *   winners   i32 [B][k][4] = (feature, t, y, x) in selection order,
 *             rows beyond the count filled with -1.
 *   n_winners i32 [B].
 * Limits: C*H*W <= 2^24, H*W <= 65536, 1 <= k, 0 <= radius, T <= 255.
 * Workspace: spk_kwta_workspace_size(B, C, H, W) bytes.                    */
SPK_API size_t spk_kwta_workspace_size(int B, int C, int H, int W);
SPK_API int spk_kwta(const uint8_t *t_first, const float *v_first, int B, int T, int C, int H, int W,
             int k, int radius, int32_t *winners, int32_t *n_winners,
             void *workspace, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * STDP (Eq.4) on the winners' weights, in place.  For winner
 * (f, t_i, y, x) of image b and synapse (ci, ky, kx), the pre-synaptic
 * neuron is (ci, y+ky-pad, x+kx-pad) of the layer input; it counts as
 * T_j <= T_i when pre_wave[b][t_i] is 1 there (padding never spikes).
 *   dW = A * (W - lb) * (ub - W), A = a_plus if T_j <= T_i else a_minus;
 * with stabilizer == 0 the product term is 1.  W is clamped to [lb, ub].
 * Batches use frozen-forward, ordered replay: the winners of image 0 are
 * applied first, then image 1, and so on; one image's winners use distinct
 * features, so their order does not matter.  The update of each weight is
 * evaluated in double precision as d = (w-lb)*(ub-w); u = a*d; w = w+u;
 * clamp; and stored as float.  Weights are expected to be finite.
 *   weight    f32 [Cout][Cin][K][K] (updated in place)
 *   pre_wave  u8  [B][T][Cin][H][W]: the layer's (unpadded) input wave
 *   winners / n_winners as produced by spk_kwta with the same k.
 * Limits: T <= 255, Cout*B < 2^31, Cin*K*K <= 65535*256, and
 * ceil(B*min(k,Cout)/32) + Cout <= 65535.
 * Workspace: spk_stdp_workspace_size(Cout, Cin, K, B, k) bytes (per-feature
 * update lists and the packed pre-synaptic bits); calls that run
 * concurrently need separate workspaces.                                  */
SPK_API size_t spk_stdp_workspace_size(int Cout, int Cin, int K, int B, int k);
SPK_API int spk_stdp(float *weight, int Cout, int Cin, int K, int pad,
             const uint8_t *pre_wave, int B, int T, int H, int W,
             const int32_t *winners, const int32_t *n_winners, int k,
             float a_plus, float a_minus, float lb, float ub, int stabilizer,
             void *workspace, size_t ws_bytes, void *stream);

/* R-STDP (section "snn Module": two STDP objects; tutorial: anti-STDP
 * negates the learning rates): as spk_stdp, with reward i8 [B] per image:
 * +1 applies (a_plus, a_minus), -1 applies (-a_plus, -a_minus), 0 skips.
 * Same workspace as spk_stdp.                                              */
SPK_API int spk_rstdp(float *weight, int Cout, int Cin, int K, int pad,
              const uint8_t *pre_wave, int B, int T, int H, int W,
              const int32_t *winners, const int32_t *n_winners, int k, const int8_t *reward,
              float a_plus, float a_minus, float lb, float ub, int stabilizer,
              void *workspace, size_t ws_bytes, void *stream);

/* STDP / R-STDP with the layer input given by its first-spike map
 * pre_t_first u8 [B][Cin][H][W] (values in [0, T], T = never) instead of its
 * wave: T_j <= T_i is read as pre_t_first <= t_i, which is the wave's entry
 * at step t_i by Eq.1.  All else as spk_stdp / spk_rstdp (same workspace);
 * the updates are identical to theirs on the map's Eq.1 wave.  For callers
 * that keep first-spike maps only (the compact inter-layer form).            */
SPK_API int spk_stdp_first_spike(float *weight, int Cout, int Cin, int K, int pad,
             const uint8_t *pre_t_first, int B, int T, int H, int W,
             const int32_t *winners, const int32_t *n_winners, int k,
             float a_plus, float a_minus, float lb, float ub, int stabilizer,
             void *workspace, size_t ws_bytes, void *stream);
SPK_API int spk_rstdp_first_spike(float *weight, int Cout, int Cin, int K, int pad,
             const uint8_t *pre_t_first, int B, int T, int H, int W,
             const int32_t *winners, const int32_t *n_winners, int k, const int8_t *reward,
             float a_plus, float a_minus, float lb, float ub, int stabilizer,
             void *workspace, size_t ws_bytes, void *stream);

/* STDP / R-STDP of a layer with stride > 1 (Eq.4; stride as in
 * spk_conv_fire_strided): the pre-synaptic neuron of winner (f, t_i, y, x)
 * and synapse (ci, ky, kx) is (ci, y*stride+ky-pad, x*stride+kx-pad) of the
 * layer input.  stride 1..64; all else as spk_stdp / spk_rstdp (same
 * workspace).                                                               */
SPK_API int spk_stdp_strided(float *weight, int Cout, int Cin, int K, int stride, int pad,
             const uint8_t *pre_wave, int B, int T, int H, int W,
             const int32_t *winners, const int32_t *n_winners, int k,
             float a_plus, float a_minus, float lb, float ub, int stabilizer,
             void *workspace, size_t ws_bytes, void *stream);
SPK_API int spk_rstdp_strided(float *weight, int Cout, int Cin, int K, int stride, int pad,
             const uint8_t *pre_wave, int B, int T, int H, int W,
             const int32_t *winners, const int32_t *n_winners, int k, const int8_t *reward,
             float a_plus, float a_minus, float lb, float ub, int stabilizer,
             void *workspace, size_t ws_bytes, void *stream);

/* Decision and reward (tutorial: the first winner's feature maps to a
 * class; reward when it equals the label, punish otherwise, nothing for a
 * silent sample).  decision i32 [B] = winners[b][0].feature % n_classes or
 * -1 when n_winners[b] == 0; reward i8 [B] in {+1, -1, 0}.                 */
SPK_API int spk_decide(const int32_t *winners, const int32_t *n_winners, int B, int k,
               const int32_t *labels, int n_classes, int32_t *decision, int8_t *reward,
               void *stream);

/* Synaptic events of a convolution (the throughput unit of the hot path):
 * the number of (spiking pre-synaptic neuron, post-synaptic neuron) pairs,
 * each counted once -- for every output position, Cout times the number of
 * in-bounds receptive-field taps whose input neuron spikes at some step of
 * the wave (u8 [B][T][Cin][H][W]; its last step is 1 exactly there).
 * *count is a device u64, overwritten.  Same size rules as spk_conv_fire.  */
SPK_API int spk_count_events(const uint8_t *wave, int B, int T, int Cin, int H, int W,
                             int Cout, int K, int pad, uint64_t *count, void *stream);
/* The same count for a layer with stride > 1 (receptive fields as in
 * spk_conv_fire_strided; stride 1..64).                                    */
SPK_API int spk_count_events_strided(const uint8_t *wave, int B, int T, int Cin, int H, int W,
                             int Cout, int K, int stride, int pad, uint64_t *count, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* LIBSPYKE_H */
