// Intensity-to-latency encoding and spike-wave utilities (gfx950).
//
// Paper: section "utils Module" (multi-channel DoG/Gabor Filter applied to the
// image, Intensity2Latency = rank-order coding), the threshold semantics of
// the "functional Module", and Eq.1 (cumulative spike wave).
//
// spk_encode_latency runs three kernels on the caller's stream:
//   1. k_filter: same-size cross-correlation of each u8 image with the C
//      filters (double accumulation over the non-zero taps, one rounding to
//      float, then values below the threshold set to 0).  One workgroup per
//      (image, band of rows: the whole image when it fits) stages the
//      zero-padded band in LDS and computes all channels.
//   2. k_rank_select: one workgroup per image finds the T-1 bin boundaries of
//      the rank-order code by an MSD radix select (8 passes of 8 bits) on the
//      unique 64-bit keys  (float bits of I) << 32 | ~index  of the positive
//      intensities; all boundaries share each pass's digit histograms.
//   3. k_expand_latency: every entry counts the boundaries its key does not
//      exceed -- that count is its bin floor(rho*T/n) -- and writes t_first
//      and the T planes of the wave (4 entries per thread, u32 stores).
// When C*H*W <= SORT_MAX, steps 2 and 3 are one kernel instead,
// k_rank_sort: one workgroup per image gathers the keys of the positive
// intensities into LDS, sorts them (bitonic network over the next power of two
// of their count), gives the entry at rank rho the bin floor(rho*T/n) in an
// LDS map of t_first, and writes t_first and the wave from that map.
#include <algorithm>

#include "common.hpp"

namespace {

constexpr int MAX_KF = 31;
constexpr int SEL_THREADS = 1024;
constexpr int MAX_GROUPS = 32;   // bin boundaries resolved per select batch
constexpr int LDS_KEYS = 12288;  // intensities cached in LDS when N fits
constexpr int SORT_MAX = 8192;   // entries per image sorted in LDS
constexpr int SORT_THREADS = 1024;

// ------------------------------------------------------------------ filter
// LDS holds the taps and the zero-padded band of the image as doubles, so the
// tap loop has no bounds checks; padded pixels contribute +0 terms, which
// leave every partial sum unchanged (the sums are never -0), so the result
// equals the sum over the in-image taps in the same ky-then-kx order.  A
// workgroup covers a band of R rows (the whole image when it fits in LDS) and
// all C channels: its work items are (channel, row, group of 4 columns), so
// every thread has work however narrow the image.  An item makes 4
// consecutive outputs of a row: along kx it keeps the 4 pixels under the taps
// in registers and reads one new pixel per tap (3 zero columns pad the band on
// the right for the last group).
__device__ __forceinline__ int wave_min_i32(int v) {
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) v = min(v, __shfl_xor(v, s, 64));
    return v;
}
__device__ __forceinline__ int wave_max_i32(int v) {
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) v = max(v, __shfl_xor(v, s, 64));
    return v;
}

__global__ __launch_bounds__(256) void k_filter(const uint8_t *__restrict__ img, int B, int H, int W,
                                                const float *__restrict__ filt, int C, int KF, float thr, int R,
                                                float *__restrict__ out) {
    extern __shared__ double smem_d[];
    const int nb = (H + R - 1) / R;
    const int b = blockIdx.x / nb, band = blockIdx.x % nb;
    const int y0 = band * R, p = (KF - 1) / 2;
    const int rows = min(R, H - y0);
    const int srows = rows + KF - 1, Wp = W + 2 * p + 3;
    const int KK = KF * KF;
    double *fd = smem_d;                                       // C*KF*KF taps
    double *sim = fd + C * KK;                                 // srows x Wp pixels
    int *bbox = reinterpret_cast<int *>(sim + srows * Wp);     // C x (y0,y1,x0,x1)

    for (int i = threadIdx.x; i < C * KK; i += blockDim.x) fd[i] = (double)filt[i];
    for (int i = threadIdx.x; i < srows * Wp; i += blockDim.x) {
        const int r = i / Wp, xp = i - r * Wp;
        const int y = y0 - p + r, x = xp - p;
        sim[i] = (y >= 0 && y < H && x >= 0 && x < W) ? (double)img[((int64_t)b * H + y) * W + x] : 0.0;
    }
    __syncthreads();
    // bounding box of the non-zero taps of each channel (zero taps add nothing),
    // one wave per channel
    const int lane = threadIdx.x & 63, nw = blockDim.x >> 6;
    for (int c = threadIdx.x >> 6; c < C; c += nw) {
        int ya = KF, yb = -1, xa = KF, xb = -1;
        for (int i = lane; i < KK; i += 64)
            if (fd[c * KK + i] != 0.0) {
                const int ky = i / KF, kx = i - ky * KF;
                ya = min(ya, ky); yb = max(yb, ky); xa = min(xa, kx); xb = max(xb, kx);
            }
        ya = wave_min_i32(ya); yb = wave_max_i32(yb); xa = wave_min_i32(xa); xb = wave_max_i32(xb);
        if (lane == 0) {
            bbox[4 * c] = ya; bbox[4 * c + 1] = yb; bbox[4 * c + 2] = xa; bbox[4 * c + 3] = xb;
        }
    }
    __syncthreads();
    const int xg = (W + 3) / 4, per = rows * xg, items = C * per;
    for (int i = threadIdx.x; i < items; i += blockDim.x) {
        const int c = i / per, rem = i - c * per;
        const int r = rem / xg, x = (rem - r * xg) * 4;
        const int ya = bbox[4 * c], yb = bbox[4 * c + 1], xa = bbox[4 * c + 2], xb = bbox[4 * c + 3];
        const double *fc = fd + c * KK;
        double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
        for (int ky = ya; ky <= yb; ++ky) {
            const double *row = sim + (r + ky) * Wp + x;
            const double *frow = fc + ky * KF;
            double w0 = row[xa], w1 = row[xa + 1], w2 = row[xa + 2];
#pragma unroll 4
            for (int kx = xa; kx <= xb; ++kx) {
                const double w3 = row[kx + 3], f = frow[kx];
                s0 += f * w0;
                s1 += f * w1;
                s2 += f * w2;
                s3 += f * w3;
                w0 = w1;
                w1 = w2;
                w2 = w3;
            }
        }
        float *o = out + (((int64_t)b * C + c) * H + y0 + r) * W + x;
        const double sv[4] = {s0, s1, s2, s3};
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (x + j < W) {
                const float v = (float)sv[j];
                o[j] = (v < thr) ? 0.0f : v;
            }
    }
}

// ------------------------------------------------------------------ rank select
__device__ __forceinline__ uint64_t make_key(float v, uint32_t idx) {
    return ((uint64_t)__float_as_uint(v) << 32) | (uint64_t)(0xFFFFFFFFu - idx);
}

// Output per image: bounds[b][j] (j = 0..T-2) = key at rank ceil((j+1)*n/T)
// in descending order, 0 when that rank is >= n; count[b] = n.
__global__ __launch_bounds__(SEL_THREADS) void k_rank_select(const float *__restrict__ inten, int64_t N, int T,
                                                             uint64_t *__restrict__ bounds,
                                                             uint32_t *__restrict__ count) {
    __shared__ uint32_t hist[MAX_GROUPS][256];
    __shared__ uint64_t gprefix[MAX_GROUPS];
    __shared__ uint64_t tprefix[MAX_GROUPS];
    __shared__ uint32_t trank[MAX_GROUPS];
    __shared__ int tgroup[MAX_GROUPS];
    __shared__ int ngroups, ntarg;
    __shared__ int red[SEL_THREADS / 64];
    __shared__ float cache[LDS_KEYS];

    const int b = blockIdx.x;
    const float *I = inten + (int64_t)b * N;
    const bool cached = N <= LDS_KEYS;
    const int tid = threadIdx.x;

    int cnt = 0;
    for (int64_t i = tid; i < N; i += SEL_THREADS) {
        const float v = I[i];
        if (cached) cache[i] = v;
        cnt += v > 0.0f;
    }
    cnt = spk::wave_sum_i32(cnt);
    if ((tid & 63) == 0) red[tid >> 6] = cnt;
    __syncthreads();
    uint32_t n = 0;
    for (int w = 0; w < SEL_THREADS / 64; ++w) n += (uint32_t)red[w];
    if (tid == 0) count[b] = n;

    for (int j0 = 0; j0 < T - 1; j0 += MAX_GROUPS) {
        const int jn = min(MAX_GROUPS, T - 1 - j0);
        if (tid < jn) {
            const uint64_t r = ((uint64_t)(j0 + tid + 1) * n + T - 1) / T;  // ceil((j+1) n / T)
            trank[tid] = (uint32_t)r;
            tprefix[tid] = 0;
            bounds[(int64_t)b * (T - 1) + j0 + tid] = 0;
        }
        __syncthreads();
        if (tid == 0) {
            int m = 0;
            for (int j = 0; j < jn; ++j) m += trank[j] < n;
            ntarg = m;  // active targets are a prefix (ranks grow with j)
        }
        __syncthreads();
        const int m = ntarg;
        if (m == 0) continue;
        for (int pass = 0; pass < 8; ++pass) {
            const int shift = 56 - 8 * pass;
            // group the active targets by their current prefix (non-increasing in j)
            if (tid == 0) {
                int g = -1;
                for (int j = 0; j < m; ++j) {
                    if (g < 0 || tprefix[j] != gprefix[g]) gprefix[++g] = tprefix[j];
                    tgroup[j] = g;
                }
                ngroups = g + 1;
            }
            __syncthreads();
            const int ng = ngroups;
            for (int i = tid; i < ng * 256; i += SEL_THREADS) (&hist[0][0])[i] = 0;
            __syncthreads();
            for (int64_t i = tid; i < N; i += SEL_THREADS) {
                const float v = cached ? cache[i] : I[i];
                if (!(v > 0.0f)) continue;
                const uint64_t key = make_key(v, (uint32_t)i);
                const uint64_t pre = pass == 0 ? 0 : (key >> (shift + 8));
                // binary search among the group prefixes (sorted descending)
                int lo = 0, hi = ng - 1, g = -1;
                while (lo <= hi) {
                    const int mid = (lo + hi) >> 1;
                    const uint64_t gp = gprefix[mid];
                    if (gp == pre) { g = mid; break; }
                    if (gp > pre) lo = mid + 1; else hi = mid - 1;
                }
                if (g >= 0) atomicAdd(&hist[g][(key >> shift) & 255u], 1u);
            }
            __syncthreads();
            // per group, suffix sums over the digits (digit 255 first): one wave per group
            for (int g = tid >> 6; g < ng; g += SEL_THREADS / 64) {
                const int lane = tid & 63;
                uint32_t h[4], loc = 0;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    h[q] = hist[g][4 * lane + q];
                    loc += h[q];
                }
                uint32_t suf = loc;  // sum over lanes >= lane
#pragma unroll
                for (int d = 1; d < 64; d <<= 1) {
                    const uint32_t o = __shfl_down(suf, d, 64);
                    if (lane + d < 64) suf += o;
                }
                uint32_t above = suf - loc;  // digits held by higher lanes
                for (int q = 3; q >= 0; --q) {
                    above += h[q];
                    hist[g][4 * lane + q] = above;  // now: entries with digit >= 4*lane+q
                }
            }
            __syncthreads();
            if (tid < m) {
                // the digit d with S[d+1] <= r < S[d], where S[d] = entries with digit >= d
                const int g = tgroup[tid];
                const uint32_t r = trank[tid];
                int lo = 0, hi = 255;  // S[0] > r holds: the rank exists in this group
                while (lo < hi) {
                    const int mid = (lo + hi + 1) >> 1;
                    if (hist[g][mid] > r) lo = mid; else hi = mid - 1;
                }
                const int d = lo;
                const uint32_t above = d < 255 ? hist[g][d + 1] : 0u;
                trank[tid] = r - above;
                tprefix[tid] = (tprefix[tid] << 8) | (uint64_t)d;
            }
            __syncthreads();
        }
        if (tid < m) bounds[(int64_t)b * (T - 1) + j0 + tid] = tprefix[tid];
        __syncthreads();
    }
}

// t_first = number of boundaries K_j with key <= K_j (the K_j are non-increasing).
__device__ __forceinline__ int bin_of(uint64_t key, const uint64_t *kb, int nb) {
    int lo = 0, hi = nb;  // first j with kb[j] < key
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (kb[mid] >= key) lo = mid + 1; else hi = mid;
    }
    return lo;
}

__global__ __launch_bounds__(256) void k_expand_latency(const float *__restrict__ inten, int64_t N, int T,
                                                        const uint64_t *__restrict__ bounds,
                                                        uint8_t *__restrict__ tf_out, uint8_t *__restrict__ wave,
                                                        int chunks) {
    __shared__ uint64_t kb[256];
    const int b = blockIdx.x / chunks, ch = blockIdx.x % chunks;
    const int nbnd = T - 1;
    for (int j = threadIdx.x; j < nbnd; j += blockDim.x) kb[j] = bounds[(int64_t)b * nbnd + j];
    __syncthreads();
    const float *I = inten + (int64_t)b * N;
    const bool vec = (N % 4) == 0;
    const int64_t groups = (N + 3) / 4;
    for (int64_t q = (int64_t)ch * blockDim.x + threadIdx.x; q < groups; q += (int64_t)chunks * blockDim.x) {
        uint32_t tv = 0;
        int t4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t i = q * 4 + j;
            int t = T;
            if (i < N) {
                const float v = I[i];
                if (v > 0.0f) t = bin_of(make_key(v, (uint32_t)i), kb, nbnd);
            }
            t4[j] = t;
            tv |= (uint32_t)t << (8 * j);
        }
        if (vec) {
            if (tf_out) *reinterpret_cast<uint32_t *>(tf_out + (int64_t)b * N + q * 4) = tv;
            if (wave)
                for (int t = 0; t < T; ++t)
                    *reinterpret_cast<uint32_t *>(wave + ((int64_t)b * T + t) * N + q * 4) = spk::spikes4(tv, t, T);
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t i = q * 4 + j;
                if (i >= N) break;
                if (tf_out) tf_out[(int64_t)b * N + i] = (uint8_t)t4[j];
                if (wave)
                    for (int t = 0; t < T; ++t) wave[((int64_t)b * T + t) * N + i] = (uint8_t)(t >= t4[j]);
            }
        }
    }
}

// ------------------------------------------------------------------ rank by sorting (small images)
__global__ __launch_bounds__(SORT_THREADS) void k_rank_sort(const float *__restrict__ inten, int N, int T,
                                                            uint8_t *__restrict__ tf_out, uint8_t *__restrict__ wave) {
    __shared__ uint64_t key[SORT_MAX];
    __shared__ uint8_t tmap[SORT_MAX];
    __shared__ int npos;
    const int b = blockIdx.x, tid = threadIdx.x;
    const float *I = inten + (int64_t)b * N;
    if (tid == 0) npos = 0;
    for (int i = tid; i < N; i += SORT_THREADS) tmap[i] = (uint8_t)T;
    __syncthreads();
    // gather the positive entries' keys (their order in LDS does not matter: keys are
    // unique); every load of the thread is issued before the first is used
    float vin[SORT_MAX / SORT_THREADS];
#pragma unroll
    for (int r = 0; r < SORT_MAX / SORT_THREADS; ++r) {
        const int i = r * SORT_THREADS + tid;
        vin[r] = i < N ? I[i] : 0.0f;
    }
#pragma unroll
    for (int r = 0; r < SORT_MAX / SORT_THREADS; ++r) {
        const int i = r * SORT_THREADS + tid;
        const float v = vin[r];
        const bool pos = v > 0.0f;
        const uint64_t m = __ballot(pos);
        int base = 0;
        if ((tid & 63) == 0 && m) base = atomicAdd(&npos, __popcll(m));
        base = __shfl(base, 0, 64);
        if (pos) key[base + __popcll(m & ((1ull << (tid & 63)) - 1ull))] = make_key(v, (uint32_t)i);
    }
    __syncthreads();
    const int n = npos;
    int m = 1;
    while (m < n) m <<= 1;
    for (int i = n + tid; i < m; i += SORT_THREADS) key[i] = 0;  // below every positive key
    __syncthreads();
    // bitonic network, descending overall
    for (int k = 2; k <= m; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = tid; i < m / 2; i += SORT_THREADS) {
                const int lo = ((i & ~(j - 1)) << 1) | (i & (j - 1)), hi = lo + j;
                const uint64_t x = key[lo], y = key[hi];
                const bool desc = (lo & k) == 0;
                if ((x < y) == desc) {
                    key[lo] = y;
                    key[hi] = x;
                }
            }
            __syncthreads();
        }
    }
    for (int p = tid; p < n; p += SORT_THREADS)
        tmap[0xFFFFFFFFu - (uint32_t)key[p]] = (uint8_t)(((int64_t)p * T) / n);
    __syncthreads();
    uint8_t *tf = tf_out ? tf_out + (int64_t)b * N : nullptr;
    uint8_t *wv = wave ? wave + (int64_t)b * T * N : nullptr;
    if ((N & 3) == 0) {
        const int nq = N / 4;
        for (int q = tid; q < nq; q += SORT_THREADS) {
            const uint32_t t4 = *reinterpret_cast<const uint32_t *>(tmap + 4 * q);
            if (tf) *reinterpret_cast<uint32_t *>(tf + 4 * q) = t4;
            if (wv)
                for (int t = 0; t < T; ++t) *reinterpret_cast<uint32_t *>(wv + (int64_t)t * N + 4 * q) = spk::spikes4(t4, t, T);
        }
    } else {
        for (int i = tid; i < N; i += SORT_THREADS)
            if (tf) tf[i] = tmap[i];
        if (wv)
            for (int e = tid; e < T * N; e += SORT_THREADS) {
                const int t = e / N, i = e - t * N;
                wv[(int64_t)t * N + i] = (uint8_t)(t >= (int)tmap[i]);
            }
    }
}

// ------------------------------------------------------------------ local normalisation
// out = in / (float(S / (2r+1)^2) + eps), S the sum of the zero-padded window
// of the entry's channel taken as row sums R(y', x) (double, dx ascending)
// added over the rows (dy ascending) -- the order the definition fixes, so
// the result is reproducible bit for bit.  A row sum is the same value for
// every entry that uses it, so a workgroup computes each once: it takes a
// tile of TR output rows of one plane, stages the TR + 2r input rows with
// their zero margins in LDS, computes their row sums into LDS, then adds
// 2r + 1 of them per entry.
__global__ __launch_bounds__(256) void k_local_norm(const float *__restrict__ in, int H, int W, int r, int TR,
                                                    float eps, float *__restrict__ out) {
#pragma clang fp contract(off)
    extern __shared__ double lnsm[];
    const int ntile = (H + TR - 1) / TR;
    const int64_t pl = blockIdx.x / ntile;
    const int y0 = (int)(blockIdx.x % ntile) * TR;
    const int rows = min(TR, H - y0), srows = rows + 2 * r, Wp = W + 2 * r;
    double *R = lnsm;                                          // srows x W row sums
    float *xs = reinterpret_cast<float *>(R + (size_t)srows * W);  // srows x Wp padded input
    const float *src = in + pl * H * W;
    for (int i = threadIdx.x; i < srows * Wp; i += blockDim.x) {
        const int rr = i / Wp, cc = i - rr * Wp;
        const int y = y0 - r + rr, x = cc - r;
        xs[i] = (y >= 0 && y < H && x >= 0 && x < W) ? src[(int64_t)y * W + x] : 0.0f;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < srows * W; i += blockDim.x) {
        const int rr = i / W, x = i - rr * W;
        const float *row = xs + rr * Wp + x;
        double acc = 0.0;
        for (int dx = 0; dx <= 2 * r; ++dx) acc += (double)row[dx];
        R[i] = acc;
    }
    __syncthreads();
    const double n = (double)(2 * r + 1) * (double)(2 * r + 1);
    float *dst = out + pl * H * W;
    for (int i = threadIdx.x; i < rows * W; i += blockDim.x) {
        const int yy = i / W, x = i - yy * W;
        double S = 0.0;
        for (int dy = 0; dy <= 2 * r; ++dy) S += R[(yy + dy) * W + x];
        const float mean = (float)(S / n);
        const float d = mean + eps;
        dst[(int64_t)(y0 + yy) * W + x] = xs[(yy + r) * Wp + x + r] / d;
    }
}

// Output rows per workgroup of the local normalisation: as many as LDS holds.
int local_norm_rows(int H, int W, int r) {
    const size_t per_row = (size_t)W * sizeof(double) + (size_t)(W + 2 * r) * sizeof(float);
    const size_t cap = 60 * 1024 / per_row;
    return cap > (size_t)(2 * r) ? (int)std::min<size_t>(H, cap - 2 * r) : 0;
}

// ------------------------------------------------------------------ Eq.1 utilities
__global__ __launch_bounds__(256) void k_expand_wave(const uint8_t *__restrict__ tf, int64_t N, int T,
                                                     uint8_t *__restrict__ wave, int64_t total_groups,
                                                     int64_t groups_per_img) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= total_groups) return;
    const int64_t b = q / groups_per_img, g = q % groups_per_img;
    if ((N % 4) == 0) {
        const uint32_t t4 = *reinterpret_cast<const uint32_t *>(tf + b * N + g * 4);
        for (int t = 0; t < T; ++t) *reinterpret_cast<uint32_t *>(wave + (b * T + t) * N + g * 4) = spk::spikes4(t4, t, T);
    } else {
        for (int j = 0; j < 4; ++j) {
            const int64_t i = g * 4 + j;
            if (i >= N) break;
            const int tv = tf[b * N + i];
            for (int t = 0; t < T; ++t) wave[(b * T + t) * N + i] = (uint8_t)(t >= tv);
        }
    }
}

__global__ void k_zero_i32(int32_t *p) { *p = 0; }

__global__ __launch_bounds__(256) void k_validate_wave(const uint8_t *__restrict__ wave, int64_t B, int64_t N, int T,
                                                       int32_t *__restrict__ bad) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int my = 0;
    if (i < B * N) {
        const int64_t b = i / N, e = i % N;
        int prev = 0;
        for (int t = 0; t < T; ++t) {
            const int v = wave[(b * T + t) * N + e];
            if (v > 1 || v < prev) { my = 1; break; }
            prev = v;
        }
    }
    my = spk::wave_sum_i32(my);
    if ((threadIdx.x & 63) == 0 && my) atomicAdd(bad, my);
}

struct EncPlan {
    int64_t N;
    size_t inten_bytes, bound_bytes, count_bytes;
};

int enc_plan(int B, int C, int H, int W, int T, EncPlan &p) {
    SPK_REQUIRE(B >= 0 && C >= 1 && H >= 1 && W >= 1 && T >= 1, SPK_E_SHAPE,
                "spk_encode_latency: bad sizes B=%d C=%d H=%d W=%d T=%d", B, C, H, W, T);
    SPK_REQUIRE(T <= 255, SPK_E_RANGE, "spk_encode_latency: T=%d > 255", T);
    p.N = (int64_t)C * H * W;
    SPK_REQUIRE(p.N < (1LL << 31), SPK_E_RANGE, "spk_encode_latency: C*H*W too large");
    p.inten_bytes = (size_t)B * p.N * sizeof(float);
    p.bound_bytes = (size_t)B * (T > 1 ? T - 1 : 1) * sizeof(uint64_t);
    p.count_bytes = (size_t)B * sizeof(uint32_t);
    return SPK_OK;
}

// The rank-order code of an intensity map: one sorting kernel per image when it
// fits in LDS, else the bin boundaries by radix select and a separate expansion.
void launch_rank(const float *I, int B, int64_t N, int T, uint8_t *t_first, uint8_t *wave, uint64_t *bounds,
                 uint32_t *count, hipStream_t st) {
    if (N <= SORT_MAX) {
        hipLaunchKernelGGL(k_rank_sort, dim3(B), dim3(SORT_THREADS), 0, st, I, (int)N, T, t_first, wave);
        return;
    }
    if (T > 1) hipLaunchKernelGGL(k_rank_select, dim3(B), dim3(SEL_THREADS), 0, st, I, N, T, bounds, count);
    const int64_t groups = (N + 3) / 4;
    const int chunks = (int)std::max<int64_t>(1, std::min<int64_t>(64, spk::ceil_div(groups, 256)));
    hipLaunchKernelGGL(k_expand_latency, dim3((unsigned)(B * chunks)), dim3(256), 0, st, I, N, T, bounds, t_first,
                       wave, chunks);
}

}  // namespace

extern "C" size_t spk_encode_latency_workspace_size(int B, int C, int H, int W, int T) {
    EncPlan p;
    if (enc_plan(B, C, H, W, T, p) != SPK_OK) return 0;
    spk::Carver c(nullptr);
    c.take<float>(p.inten_bytes / sizeof(float));
    c.take<uint64_t>(p.bound_bytes / sizeof(uint64_t));
    c.take<uint32_t>(p.count_bytes / sizeof(uint32_t));
    return spk::align_up(c.off, 256);
}

extern "C" int spk_encode_latency(const uint8_t *image, int B, int H, int W, const float *filters, int C, int KF,
                                  float filter_threshold, int T, uint8_t *wave, uint8_t *t_first,
                                  float *intensities, void *workspace, size_t ws_bytes, void *stream) {
    EncPlan p;
    int rc = enc_plan(B, C, H, W, T, p);
    if (rc != SPK_OK) return rc;
    SPK_REQUIRE(KF >= 1 && (KF % 2) == 1 && KF <= MAX_KF, SPK_E_RANGE,
                "spk_encode_latency: filter size %d must be odd and <= %d", KF, MAX_KF);

    SPK_REQUIRE(!std::isnan(filter_threshold), SPK_E_ARG, "spk_encode_latency: threshold is NaN");
    if (B == 0) return spk::ok();
    SPK_REQUIRE(image && filters, SPK_E_ARG, "spk_encode_latency: image and filters are required");
    const size_t need = spk_encode_latency_workspace_size(B, C, H, W, T);
    SPK_REQUIRE(workspace && ws_bytes >= need, SPK_E_WORKSPACE,
                "spk_encode_latency: workspace of %zu bytes < %zu required", ws_bytes, need);
    hipStream_t st = spk::as_stream(stream);
    spk::Carver cv(workspace);
    float *ws_int = cv.take<float>(p.inten_bytes / sizeof(float));
    uint64_t *bounds = cv.take<uint64_t>(p.bound_bytes / sizeof(uint64_t));
    uint32_t *count = cv.take<uint32_t>(p.count_bytes / sizeof(uint32_t));
    float *I = intensities ? intensities : ws_int;

    // rows per band: the whole image when it fits in LDS, else the most that
    // fit, then evened out over the bands
    auto filter_lds = [&](int rows) {
        return ((size_t)C * KF * KF + (size_t)(rows + KF - 1) * (W + KF - 1 + 3)) * sizeof(double) +
               4 * C * sizeof(int);
    };
    int R = H;
    while (R > 1 && filter_lds(R) > 65536) --R;
    SPK_REQUIRE(filter_lds(R) <= 65536, SPK_E_RANGE, "spk_encode_latency: %d filters of %dx%d on width %d do not fit",
                C, KF, KF, W);
    int nb = (H + R - 1) / R;
    // few images (online steps): more, thinner bands, so that more workgroups share them
    while ((int64_t)B * nb < 128 && nb < H) nb = std::min(H, 2 * nb);
    R = (H + nb - 1) / nb;
    hipLaunchKernelGGL(k_filter, dim3((unsigned)(B * nb)), dim3(256), filter_lds(R), st, image, B, H, W, filters, C,
                       KF, filter_threshold, R, I);
    if (!t_first && !wave) return spk::check_launch("spk_encode_latency");
    launch_rank(I, B, p.N, T, t_first, wave, bounds, count, st);
    return spk::check_launch("spk_encode_latency");
}

extern "C" size_t spk_rank_latency_workspace_size(int B, int C, int H, int W, int T) {
    EncPlan p;
    if (enc_plan(B, C, H, W, T, p) != SPK_OK) return 0;
    spk::Carver c(nullptr);
    c.take<uint64_t>(p.bound_bytes / sizeof(uint64_t));
    c.take<uint32_t>(p.count_bytes / sizeof(uint32_t));
    return spk::align_up(c.off, 256);
}

extern "C" int spk_rank_latency(const float *intensities, int B, int C, int H, int W, int T, uint8_t *wave,
                                uint8_t *t_first, void *workspace, size_t ws_bytes, void *stream) {
    EncPlan p;
    int rc = enc_plan(B, C, H, W, T, p);
    if (rc != SPK_OK) return rc;
    if (B == 0) return spk::ok();
    SPK_REQUIRE(intensities && (wave || t_first), SPK_E_ARG,
                "spk_rank_latency: intensities and wave or t_first are required");
    const size_t need = spk_rank_latency_workspace_size(B, C, H, W, T);
    SPK_REQUIRE(workspace && ws_bytes >= need, SPK_E_WORKSPACE, "spk_rank_latency: workspace of %zu bytes < %zu required",
                ws_bytes, need);
    spk::Carver cv(workspace);
    uint64_t *bounds = cv.take<uint64_t>(p.bound_bytes / sizeof(uint64_t));
    uint32_t *count = cv.take<uint32_t>(p.count_bytes / sizeof(uint32_t));
    launch_rank(intensities, B, p.N, T, t_first, wave, bounds, count, spk::as_stream(stream));
    return spk::check_launch("spk_rank_latency");
}

extern "C" int spk_local_normalization(const float *intensities, int B, int C, int H, int W, int radius, float eps,
                                       float *out, void *stream) {
    SPK_REQUIRE(B >= 0 && C >= 1 && H >= 1 && W >= 1, SPK_E_SHAPE, "spk_local_normalization: bad sizes");
    SPK_REQUIRE(radius >= 0 && radius <= 1024, SPK_E_RANGE, "spk_local_normalization: radius %d", radius);
    SPK_REQUIRE(!std::isnan(eps), SPK_E_ARG, "spk_local_normalization: eps is NaN");
    if (B == 0) return spk::ok();
    SPK_REQUIRE(intensities && out && intensities != out, SPK_E_ARG,
                "spk_local_normalization: intensities and a separate out are required");
    const int TR = local_norm_rows(H, W, radius);
    SPK_REQUIRE(TR >= 1, SPK_E_RANGE, "spk_local_normalization: radius %d on width %d does not fit", radius, W);
    const int64_t blocks = (int64_t)B * C * ((H + TR - 1) / TR);
    SPK_REQUIRE(blocks < (1LL << 31), SPK_E_RANGE, "spk_local_normalization: too large");
    const int srows = std::min(TR, H) + 2 * radius;
    const size_t lds = (size_t)srows * W * sizeof(double) + (size_t)srows * (W + 2 * radius) * sizeof(float);
    hipLaunchKernelGGL(k_local_norm, dim3((unsigned)blocks), dim3(256), lds, spk::as_stream(stream), intensities, H,
                       W, radius, TR, eps, out);
    return spk::check_launch("spk_local_normalization");
}

extern "C" int spk_expand_wave(const uint8_t *t_first, int B, int T, int C, int H, int W, uint8_t *wave,
                               void *stream) {
    SPK_REQUIRE(B >= 0 && C >= 1 && H >= 1 && W >= 1 && T >= 1, SPK_E_SHAPE, "spk_expand_wave: bad sizes");
    SPK_REQUIRE(T <= 255, SPK_E_RANGE, "spk_expand_wave: T=%d > 255", T);
    if (B == 0) return spk::ok();
    SPK_REQUIRE(t_first && wave, SPK_E_ARG, "spk_expand_wave: t_first and wave are required");
    const int64_t N = (int64_t)C * H * W;
    const int64_t gpi = (N + 3) / 4, total = gpi * B;
    hipLaunchKernelGGL(k_expand_wave, dim3((unsigned)spk::ceil_div(total, 256)), dim3(256), 0, spk::as_stream(stream),
                       t_first, N, T, wave, total, gpi);
    return spk::check_launch("spk_expand_wave");
}

extern "C" int spk_validate_wave(const uint8_t *wave, int B, int T, int C, int H, int W, int32_t *bad_count,
                                 void *stream) {
    SPK_REQUIRE(B >= 0 && C >= 1 && H >= 1 && W >= 1 && T >= 1, SPK_E_SHAPE, "spk_validate_wave: bad sizes");
    SPK_REQUIRE(bad_count && (wave || B == 0), SPK_E_ARG, "spk_validate_wave: wave and bad_count are required");
    hipStream_t st = spk::as_stream(stream);
    hipLaunchKernelGGL(k_zero_i32, dim3(1), dim3(1), 0, st, bad_count);
    const int64_t N = (int64_t)C * H * W, total = N * B;
    if (total > 0)
        hipLaunchKernelGGL(k_validate_wave, dim3((unsigned)spk::ceil_div(total, 256)), dim3(256), 0, st, wave,
                           (int64_t)B, N, T, bad_count);
    return spk::check_launch("spk_validate_wave");
}
