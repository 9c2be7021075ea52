/*
 * orc.c -- CPU oracle for the one-spike-per-neuron convolutional SNN layer
 * (Mozafari et al., "SpykeTorch", Frontiers in Neuroscience 2019).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this file's library.  The product
 * path (the HIP library) never calls into it, and the two share no code.
 *
 * Every function is a plain, single-threaded transcription of a definition
 * from the paper, in the order the paper states it.  Floating-point sums
 * are accumulated in double precision and rounded once to float, because
 * the method stores potentials and weights as float tensors.
 *
 * Layout conventions (all arrays contiguous, row-major, batch-major):
 *   spike wave     u8  [B][T][C][H][W]   (Eq.1, cumulative)
 *   first spikes   u8  [B][C][H][W]      (value T means "never", the paper's infinity)
 *   potentials     f32 [B][T][C][H][W]
 *   weights        f32 [Cout][Cin][K][K]
 *   winners        i32 [B][k][4] = (feature, t, row, col), -1 where unused
 * A neuron's linear index inside one image is  c*H*W + y*W + x.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_API __attribute__((visibility("default")))

/* ------------------------------------------------------------------ */
/* Eq.1 (section "Time Dimension"): S[t,f,r,c] = 0 if t < T_{f,r,c}, else 1. */
ORC_API void orc_expand_wave(const uint8_t *t_first, int64_t B, int T, int64_t N,
                             uint8_t *wave) {
    for (int64_t b = 0; b < B; ++b)
        for (int t = 0; t < T; ++t)
            for (int64_t i = 0; i < N; ++i)
                wave[(b * T + t) * N + i] = (uint8_t)(t >= t_first[b * N + i]);
}

/* Inverse of Eq.1: the first time-step at which the neuron's entry is 1
 * (T if it never is).  For a valid cumulative wave this is T_{f,r,c}. */
ORC_API void orc_first_spike(const uint8_t *wave, int64_t B, int T, int64_t N,
                             uint8_t *t_first) {
    for (int64_t b = 0; b < B; ++b)
        for (int64_t i = 0; i < N; ++i) {
            int tf = T;
            for (int t = 0; t < T; ++t)
                if (wave[(b * T + t) * N + i]) { tf = t; break; }
            t_first[b * N + i] = (uint8_t)tf;
        }
}

/* Number of entries that break Eq.1's structure: a value other than 0/1,
 * or a 1 followed by a 0 later in time (the wave must be non-decreasing). */
ORC_API int64_t orc_count_invalid(const uint8_t *wave, int64_t B, int T, int64_t N) {
    int64_t bad = 0;
    for (int64_t b = 0; b < B; ++b)
        for (int64_t i = 0; i < N; ++i) {
            int prev = 0, ok = 1;
            for (int t = 0; t < T; ++t) {
                int v = wave[(b * T + t) * N + i];
                if (v > 1 || v < prev) ok = 0;
                prev = v;
            }
            bad += !ok;
        }
    return bad;
}

/* ------------------------------------------------------------------ */
/* Input filtering (section "utils Module": a multi-channel DoG / Gabor
 * filter applied to the image, with padding and a threshold).  Same-size
 * cross-correlation (PyTorch conv2d semantics, no kernel flip), zero
 * outside the image, pixels taken as 0..255.  Then the threshold of the
 * "functional Module": values lower than the threshold become 0. */
ORC_API void orc_filter(const uint8_t *img, int64_t B, int H, int W,
                        const float *filt, int C, int KF, float thr, float *out) {
    int p = (KF - 1) / 2;
    for (int64_t b = 0; b < B; ++b)
        for (int c = 0; c < C; ++c)
            for (int y = 0; y < H; ++y)
                for (int x = 0; x < W; ++x) {
                    double s = 0.0;
                    for (int ky = 0; ky < KF; ++ky)
                        for (int kx = 0; kx < KF; ++kx) {
                            int iy = y + ky - p, ix = x + kx - p;
                            if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;
                            s += (double)filt[(c * KF + ky) * KF + kx] *
                                 (double)img[(b * H + iy) * W + ix];
                        }
                    float v = (float)s;
                    out[((b * C + c) * H + y) * W + x] = (v < thr) ? 0.0f : v;
                }
}

/* ------------------------------------------------------------------ */
/* Local normalisation (section "functional Module": intensities normalised
 * by their regional mean; the tutorial applies it between filtering and the
 * latency code).  A reading, the paper gives no formula: per channel, the
 * mean over the (2r+1)x(2r+1) window centred on the entry, the image
 * zero-padded (padding counts in the window size), then
 *     out = in / (mean + eps).
 * Operation order, fixed: row sums R(y', x) = sum over dx of in(y', x+dx)
 * (double, dx ascending), window sum S = sum over dy of R(y+dy, x) (double,
 * dy ascending), mean = float(S / (2r+1)^2), then float mean + eps and a
 * float division. */
ORC_API void orc_local_normalize(const float *in, int64_t B, int C, int H, int W, int r, float eps,
                                 float *out) {
    double n = (double)(2 * r + 1) * (double)(2 * r + 1);
    for (int64_t b = 0; b < B; ++b)
        for (int c = 0; c < C; ++c) {
            const float *src = in + (b * C + c) * (int64_t)H * W;
            float *dst = out + (b * C + c) * (int64_t)H * W;
            for (int y = 0; y < H; ++y)
                for (int x = 0; x < W; ++x) {
                    double S = 0.0;
                    for (int dy = -r; dy <= r; ++dy) {
                        double R = 0.0;
                        for (int dx = -r; dx <= r; ++dx) {
                            int yy = y + dy, xx = x + dx;
                            if (yy >= 0 && yy < H && xx >= 0 && xx < W) R += (double)src[(int64_t)yy * W + xx];
                            else R += 0.0;
                        }
                        S += R;
                    }
                    float mean = (float)(S / n);
                    float d = mean + eps;
                    dst[(int64_t)y * W + x] = src[(int64_t)y * W + x] / d;
                }
        }
}

/* ------------------------------------------------------------------ */
/* Intensity-to-latency, rank-order coding (sections "utils Module" and the
 * abstract: rank-order encoding).  Per image, all channels together: the n
 * positive intensities are ranked from largest to smallest (equal values by
 * ascending linear index), and the entry of rank rho gets time bin
 * floor(rho*T/n).  Non-positive entries never spike (bin T). */
typedef struct { float v; int64_t idx; } orc_ent;

static int orc_ent_cmp(const void *a, const void *b) {
    const orc_ent *x = (const orc_ent *)a, *y = (const orc_ent *)b;
    if (x->v > y->v) return -1;
    if (x->v < y->v) return 1;
    return (x->idx < y->idx) ? -1 : (x->idx > y->idx);
}

ORC_API void orc_rank_latency(const float *inten, int64_t B, int64_t N, int T,
                              uint8_t *t_first) {
    orc_ent *e = (orc_ent *)malloc((size_t)(N > 0 ? N : 1) * sizeof(orc_ent));
    for (int64_t b = 0; b < B; ++b) {
        const float *I = inten + b * N;
        uint8_t *tf = t_first + b * N;
        int64_t n = 0;
        for (int64_t i = 0; i < N; ++i) {
            tf[i] = (uint8_t)T;
            if (I[i] > 0.0f) { e[n].v = I[i]; e[n].idx = i; ++n; }
        }
        qsort(e, (size_t)n, sizeof(orc_ent), orc_ent_cmp);
        for (int64_t rho = 0; rho < n; ++rho)
            tf[e[rho].idx] = (uint8_t)((rho * (int64_t)T) / n);
    }
    free(e);
}

/* ------------------------------------------------------------------ */
/* Convolution of a spike wave (section "snn Module", Eq.2): for every
 * time-step independently, a valid cross-correlation of the (zero-padded,
 * as in the tutorial's forward pass) input wave with the weights.  Literal
 * form: the sum over all taps of W * S[t] at each t.  The paper's layers
 * have stride 1 and name larger strides as the next version's feature; with
 * stride s the output neuron (y, x) sees the input window whose top-left
 * padded position is (y*s, x*s), and Eq.2 becomes
 * H_out = floor((H_in + 2*pad - K) / s) + 1 (stride 1: H_in + 2*pad - K + 1). */
static inline int orc_out_size(int n, int pad, int K, int stride) { return (n + 2 * pad - K) / stride + 1; }

ORC_API void orc_conv_wave(const uint8_t *wave, int64_t B, int T, int Cin, int H, int W,
                           const float *wt, int Cout, int K, int pad, int stride, float *pot) {
    int Ho = orc_out_size(H, pad, K, stride), Wo = orc_out_size(W, pad, K, stride);
    for (int64_t b = 0; b < B; ++b)
        for (int t = 0; t < T; ++t) {
            const uint8_t *S = wave + (b * T + t) * (int64_t)Cin * H * W;
            for (int f = 0; f < Cout; ++f)
                for (int y = 0; y < Ho; ++y)
                    for (int x = 0; x < Wo; ++x) {
                        double s = 0.0;
                        for (int ci = 0; ci < Cin; ++ci)
                            for (int ky = 0; ky < K; ++ky)
                                for (int kx = 0; kx < K; ++kx) {
                                    int iy = y * stride + ky - pad, ix = x * stride + kx - pad;
                                    if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;
                                    if (S[((int64_t)ci * H + iy) * W + ix])
                                        s += (double)wt[((f * Cin + ci) * K + ky) * K + kx];
                                }
                        pot[(((b * T + t) * Cout + f) * (int64_t)Ho + y) * Wo + x] = (float)s;
                    }
        }
}

/* Same quantity computed a second, independent way from first-spike
 * times: because each input neuron spikes at most once and the wave is
 * cumulative, P[t] is the running sum over t of the weights whose input
 * spiked exactly at t.  Used to cross-check the literal form; it is also
 * the form that stays fast at large T. */
ORC_API void orc_conv_times(const uint8_t *tin, int64_t B, int T, int Cin, int H, int W,
                            const float *wt, int Cout, int K, int pad, int stride, float *pot) {
    int Ho = orc_out_size(H, pad, K, stride), Wo = orc_out_size(W, pad, K, stride);
    double *hist = (double *)malloc((size_t)(T + 1) * sizeof(double));
    for (int64_t b = 0; b < B; ++b)
        for (int f = 0; f < Cout; ++f)
            for (int y = 0; y < Ho; ++y)
                for (int x = 0; x < Wo; ++x) {
                    for (int t = 0; t <= T; ++t) hist[t] = 0.0;
                    for (int ci = 0; ci < Cin; ++ci)
                        for (int ky = 0; ky < K; ++ky)
                            for (int kx = 0; kx < K; ++kx) {
                                int iy = y * stride + ky - pad, ix = x * stride + kx - pad;
                                if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;
                                int tj = tin[((b * Cin + ci) * (int64_t)H + iy) * W + ix];
                                if (tj < T)
                                    hist[tj] += (double)wt[((f * Cin + ci) * K + ky) * K + kx];
                            }
                    double run = 0.0;
                    for (int t = 0; t < T; ++t) {
                        run += hist[t];
                        pot[(((b * T + t) * Cout + f) * (int64_t)Ho + y) * Wo + x] = (float)run;
                    }
                }
    free(hist);
}

/* Potentials of selected neurons only (full-size checks sample outputs):
 * for each of the n requested (b, f, y, x) it writes P[0..T-1], literal form. */
ORC_API void orc_conv_points(const uint8_t *wave, int64_t B, int T, int Cin, int H, int W,
                             const float *wt, int Cout, int K, int pad, int stride,
                             const int32_t *pts, int64_t n, float *out) {
    (void)B; (void)Cout;
    for (int64_t q = 0; q < n; ++q) {
        int64_t b = pts[4 * q]; int f = pts[4 * q + 1], y = pts[4 * q + 2], x = pts[4 * q + 3];
        for (int t = 0; t < T; ++t) {
            const uint8_t *S = wave + (b * T + t) * (int64_t)Cin * H * W;
            double s = 0.0;
            for (int ci = 0; ci < Cin; ++ci)
                for (int ky = 0; ky < K; ++ky)
                    for (int kx = 0; kx < K; ++kx) {
                        int iy = y * stride + ky - pad, ix = x * stride + kx - pad;
                        if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;
                        if (S[((int64_t)ci * H + iy) * W + ix])
                            s += (double)wt[((f * Cin + ci) * K + ky) * K + kx];
                    }
            out[q * T + t] = (float)s;
        }
    }
}

/* ------------------------------------------------------------------ */
/* Firing (section "functional Module": fire / threshold).  A potential at
 * or above the threshold is a spike; the first-spike time is the first
 * such step and v_first the potential there (0 for a silent neuron).
 * inf_mode selects the in-place fire with infinite threshold (Eq.5): every
 * step but the last is zeroed, and the spikes are the non-zero potentials
 * of the last step.  pot is modified in place only in inf_mode. */
ORC_API void orc_fire(float *pot, int64_t B, int T, int64_t N, float thr, int inf_mode,
                      uint8_t *spk, uint8_t *t_first, float *v_first) {
    for (int64_t b = 0; b < B; ++b)
        for (int64_t i = 0; i < N; ++i) {
            int tf = T;
            float vf = 0.0f;
            if (inf_mode) {
                for (int t = 0; t < T - 1; ++t) pot[(b * T + t) * N + i] = 0.0f;
                float last = pot[(b * T + T - 1) * N + i];
                for (int t = 0; t < T - 1; ++t) spk[(b * T + t) * N + i] = 0;
                spk[(b * T + T - 1) * N + i] = (uint8_t)(last > 0.0f);
                if (last > 0.0f) { tf = T - 1; vf = last; }
            } else {
                for (int t = 0; t < T; ++t) {
                    float p = pot[(b * T + t) * N + i];
                    int s = (p >= thr);
                    spk[(b * T + t) * N + i] = (uint8_t)s;
                    if (s && tf == T) { tf = t; vf = p; }
                }
            }
            t_first[b * N + i] = (uint8_t)tf;
            v_first[b * N + i] = vf;
        }
}

/* ------------------------------------------------------------------ */
/* Spike max-pooling (section "snn Module", Eq.3): window P, stride R, zero
 * padding D; on a spike wave the result holds the earliest spike of the
 * window.  Output size floor((H + 2D - P)/R) + 1. */
ORC_API void orc_pool(const uint8_t *wave, int64_t B, int T, int C, int H, int W,
                      int P, int R, int D, uint8_t *out) {
    int Ho = (H + 2 * D - P) / R + 1, Wo = (W + 2 * D - P) / R + 1;
    for (int64_t b = 0; b < B; ++b)
        for (int t = 0; t < T; ++t)
            for (int c = 0; c < C; ++c)
                for (int yo = 0; yo < Ho; ++yo)
                    for (int xo = 0; xo < Wo; ++xo) {
                        int m = 0;
                        for (int dy = 0; dy < P; ++dy)
                            for (int dx = 0; dx < P; ++dx) {
                                int iy = yo * R + dy - D, ix = xo * R + dx - D;
                                if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;
                                int v = wave[(((b * T + t) * C + c) * (int64_t)H + iy) * W + ix];
                                if (v > m) m = v;
                            }
                        out[(((b * T + t) * C + c) * (int64_t)Ho + yo) * Wo + xo] = (uint8_t)m;
                    }
}

/* ------------------------------------------------------------------ */
/* Max-pooling of a potentials tensor (section "snn Module": on potentials the
 * pooling keeps the largest potential of each window).  Window P, stride R,
 * zero padding D: a padded element is a potential of +0 and takes part in the
 * maximum.  Within a window the first of equal values (row-major order) is
 * kept, so -0 and +0 keep the one met first. */
ORC_API void orc_pool_potentials(const float *pot, int64_t B, int T, int C, int H, int W,
                                 int P, int R, int D, float *out) {
    int Ho = (H + 2 * D - P) / R + 1, Wo = (W + 2 * D - P) / R + 1;
    for (int64_t b = 0; b < B; ++b)
        for (int t = 0; t < T; ++t)
            for (int c = 0; c < C; ++c)
                for (int yo = 0; yo < Ho; ++yo)
                    for (int xo = 0; xo < Wo; ++xo) {
                        int first = 1;
                        float m = 0.0f;
                        for (int dy = 0; dy < P; ++dy)
                            for (int dx = 0; dx < P; ++dx) {
                                int iy = yo * R + dy - D, ix = xo * R + dx - D;
                                float v = 0.0f;
                                if (iy >= 0 && iy < H && ix >= 0 && ix < W)
                                    v = pot[(((b * T + t) * C + c) * (int64_t)H + iy) * W + ix];
                                if (first || v > m) m = v;
                                first = 0;
                            }
                        out[(((b * T + t) * C + c) * (int64_t)Ho + yo) * Wo + xo] = m;
                    }
}

/* ------------------------------------------------------------------ */
/* Pointwise inhibition (section "functional Module": at each location only
 * the neuron of the most salient feature may spike -- the earliest spike,
 * then the highest potential; ties go to the lower feature index, a
 * reading).  In the first-spike form: every other feature at that location
 * becomes silent (time T, potential 0); a location where nothing spikes is
 * left silent.  Optional potentials [B][T][C][HW] are masked the same way:
 * every plane value of a feature that is not its location's winner becomes
 * 0 (all of them where nothing spikes). */
ORC_API void orc_pointwise_inhibition(const uint8_t *t_first, const float *v_first, int64_t B, int T, int C,
                                      int64_t HW, uint8_t *out_t, float *out_v, float *pot) {
    for (int64_t b = 0; b < B; ++b)
        for (int64_t p = 0; p < HW; ++p) {
            int best = -1;
            for (int c = 0; c < C; ++c) {
                int64_t i = (b * C + c) * HW + p;
                if (t_first[i] >= T) continue;
                if (best < 0) { best = c; continue; }
                int64_t j = (b * C + best) * HW + p;
                if (t_first[i] < t_first[j] || (t_first[i] == t_first[j] && v_first[i] > v_first[j])) best = c;
            }
            for (int c = 0; c < C; ++c) {
                int64_t i = (b * C + c) * HW + p;
                int keep = c == best;
                out_t[i] = keep ? t_first[i] : (uint8_t)T;
                out_v[i] = keep ? v_first[i] : 0.0f;
                if (pot && !keep)
                    for (int t = 0; t < T; ++t) pot[((b * T + t) * C + c) * HW + p] = 0.0f;
            }
        }
}

/* ------------------------------------------------------------------ */
/* k winners-take-all (sections "snn Module" and "functional Module":
 * get_k_winners).  Eligible neurons are the ones that spiked.  Up to k
 * times: take the eligible, uninhibited neuron with the earliest spike,
 * then the largest potential, then (a reading: the paper is silent on ties)
 * the lowest linear index; record (f, t, y, x); inhibit its whole feature
 * map and, in every feature map, all positions within Chebyshev distance r
 * of (y, x).  Stops early when no eligible neuron is left. */
ORC_API void orc_kwta(const uint8_t *t_first, const float *v_first, int64_t B, int T,
                      int C, int H, int W, int k, int r, int32_t *winners, int32_t *n_win) {
    int64_t N = (int64_t)C * H * W;
    uint8_t *inh = (uint8_t *)malloc((size_t)(N > 0 ? N : 1));
    for (int64_t b = 0; b < B; ++b) {
        const uint8_t *tf = t_first + b * N;
        const float *vf = v_first + b * N;
        memset(inh, 0, (size_t)N);
        for (int j = 0; j < 4 * k; ++j) winners[b * 4 * k + j] = -1;
        int nw = 0;
        for (int round = 0; round < k; ++round) {
            int64_t best = -1;
            for (int64_t i = 0; i < N; ++i) {
                if (inh[i] || tf[i] >= T) continue;
                if (best < 0 || tf[i] < tf[best] ||
                    (tf[i] == tf[best] && vf[i] > vf[best]))
                    best = i;  /* strict comparisons keep the lowest index on ties */
            }
            if (best < 0) break;
            int f = (int)(best / ((int64_t)H * W));
            int y = (int)((best / W) % H), x = (int)(best % W);
            int32_t *o = winners + (b * k + nw) * 4;
            o[0] = f; o[1] = tf[best]; o[2] = y; o[3] = x;
            ++nw;
            for (int64_t i = (int64_t)f * H * W; i < (int64_t)(f + 1) * H * W; ++i) inh[i] = 1;
            for (int c = 0; c < C; ++c)
                for (int yy = y - r; yy <= y + r; ++yy)
                    for (int xx = x - r; xx <= x + r; ++xx)
                        if (yy >= 0 && yy < H && xx >= 0 && xx < W)
                            inh[((int64_t)c * H + yy) * W + xx] = 1;
        }
        n_win[b] = nw;
    }
    free(inh);
}

/* ------------------------------------------------------------------ */
/* STDP (Eq.4) applied to the winners' weights, and R-STDP (section
 * "snn Module": two STDP objects; tutorial: anti-STDP negates the learning
 * rates).  For winner i = (f, t_i, y, x) and each synapse (ci, ky, kx) the
 * pre-synaptic neuron j sits at (ci, y*s+ky-pad, x*s+kx-pad) of the layer
 * input (s the layer's stride);
 * T_j <= T_i holds exactly when the cumulative input wave is 1 there at
 * step t_i (a padded position never spikes).  Then
 *     dW = A * (W - LB) * (UB - W),  A = A+ if T_j <= T_i else A-,
 * with the stabilizer term replaced by 1 when it is switched off, and W kept
 * in [LB, UB].  Batches use frozen-forward, ordered replay: images are
 * applied in ascending order, each weight undergoing its chain of updates
 * sequentially.  reward (nullable) gives +1 (STDP), -1 (anti-STDP: rates
 * negated) or 0 (no update) per image.
 * Evaluation order, in double precision, rounded to float once per update:
 *     d = (w - lb) * (ub - w);  u = a * d;  w = w + u;  clamp to [lb, ub]. */
ORC_API void orc_stdp(float *wt, int Cout, int Cin, int K, int pad, int stride,
                      const uint8_t *pre_wave, int64_t B, int T, int H, int W,
                      const int32_t *winners, const int32_t *n_win, int k,
                      const int8_t *reward, float a_plus, float a_minus,
                      float lb, float ub, int stabilizer) {
    (void)Cout;
    for (int64_t b = 0; b < B; ++b) {
        double sgn = 1.0;
        if (reward) {
            if (reward[b] == 0) continue;
            sgn = (reward[b] > 0) ? 1.0 : -1.0;
        }
        for (int j = 0; j < n_win[b]; ++j) {
            const int32_t *o = winners + (b * k + j) * 4;
            int f = o[0], ti = o[1], y = o[2], x = o[3];
            const uint8_t *S = pre_wave + (b * T + ti) * (int64_t)Cin * H * W;
            for (int ci = 0; ci < Cin; ++ci)
                for (int ky = 0; ky < K; ++ky)
                    for (int kx = 0; kx < K; ++kx) {
                        int iy = y * stride + ky - pad, ix = x * stride + kx - pad;
                        int pre = 0;
                        if (iy >= 0 && iy < H && ix >= 0 && ix < W)
                            pre = S[((int64_t)ci * H + iy) * W + ix] != 0;
                        double a = sgn * (pre ? (double)a_plus : (double)a_minus);
                        float *wp = wt + ((f * Cin + ci) * K + ky) * K + kx;
                        double w = (double)*wp;
                        double d = stabilizer ? ((w - (double)lb) * ((double)ub - w)) : 1.0;
                        double u = a * d;
                        double nw = w + u;
                        if (nw < (double)lb) nw = (double)lb;
                        if (nw > (double)ub) nw = (double)ub;
                        *wp = (float)nw;
                    }
        }
    }
}

/* ------------------------------------------------------------------ */
/* Decision and reward (tutorial: the single winner of the last layer gives
 * the decision through a feature -> class map; reward if it matches the
 * label, punish if not, nothing for a silent sample).  The map is
 * feature mod n_classes. */
ORC_API void orc_decide(const int32_t *winners, const int32_t *n_win, int64_t B, int k,
                        const int32_t *labels, int n_classes, int32_t *decision,
                        int8_t *reward) {
    for (int64_t b = 0; b < B; ++b) {
        if (n_win[b] <= 0) { decision[b] = -1; reward[b] = 0; continue; }
        int d = winners[b * 4 * k] % n_classes;
        decision[b] = d;
        reward[b] = (int8_t)((d == labels[b]) ? 1 : -1);
    }
}

/* ------------------------------------------------------------------ */
/* Synaptic events of one convolution: the number of (spiking pre-synaptic
 * neuron, post-synaptic neuron) pairs, each counted once over the whole
 * simulation, i.e. for every output neuron the number of its input taps
 * whose neuron spikes at some step.  Returns the total over the batch. */
ORC_API int64_t orc_count_events(const uint8_t *tin, int64_t B, int T, int Cin, int H, int W,
                                 int Cout, int K, int pad, int stride) {
    int Ho = orc_out_size(H, pad, K, stride), Wo = orc_out_size(W, pad, K, stride);
    int64_t e = 0;
    for (int64_t b = 0; b < B; ++b)
        for (int y = 0; y < Ho; ++y)
            for (int x = 0; x < Wo; ++x) {
                int64_t c = 0;
                for (int ci = 0; ci < Cin; ++ci)
                    for (int ky = 0; ky < K; ++ky)
                        for (int kx = 0; kx < K; ++kx) {
                            int iy = y * stride + ky - pad, ix = x * stride + kx - pad;
                            if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;
                            c += tin[((b * Cin + ci) * (int64_t)H + iy) * W + ix] < T;
                        }
                e += c * Cout;
            }
    return e;
}
