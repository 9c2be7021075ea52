// Intensity-to-latency encoding and spike-wave utilities (gfx950).
//
// Paper: section "utils Module" (multi-channel DoG/Gabor Filter applied to the
// image, Intensity2Latency = rank-order coding), the threshold semantics of
// the "functional Module", and Eq.1 (cumulative spike wave).
//
// spk_encode_latency, for maps of C*H*W <= SMALL_MAX entries whose padded
// image fits in LDS (the MNIST-sized and other small inputs), is one kernel,
// k_encode_small (one workgroup per image): filter, rank-order bins by radix
// select, t_first and wave, with the intensity map never leaving LDS (it is
// written out only when the caller asks for it).  Otherwise three kernels:
//   1. k_filter: same-size cross-correlation of each u8 image with the C
//      filters (double accumulation over the non-zero taps, one rounding to
//      float, then values below the threshold set to 0).  One workgroup per
//      (image, band of rows: the whole image when it fits) stages the
//      zero-padded band in LDS and computes all channels.
//   2. rank-order bins: k_encode_small without its filter step when the map
//      has <= SMALL_MAX entries; else k_rank_select, one workgroup per image
//      finding the T-1 bin boundaries by an MSD radix select (8 passes of 8
//      bits) on the unique 64-bit keys  (float bits of I) << 32 | ~index  of
//      the positive intensities, all boundaries sharing each pass's digit
//      histograms, and
//   3. k_expand_latency: every entry counts the boundaries its key does not
//      exceed -- that count is its bin floor(rho*T/n) -- and writes t_first
//      and the T planes of the wave (4 entries per thread, u32 stores).
#include <algorithm>

#include "common.hpp"

namespace {

constexpr int MAX_KF = 31;
constexpr int SEL_THREADS = 1024;
constexpr int MAX_GROUPS = 32;   // bin boundaries resolved per select batch
constexpr int LDS_KEYS = 12288;  // intensities cached in LDS when N fits
constexpr int SMALL_MAX = 8192;  // entries per image coded by one k_encode_small workgroup
constexpr size_t SMALL_LDS = 60 * 1024;  // its dynamic LDS at most

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
// Min / max of two 16-bit halves over the wave, by DPP lane moves (no LDS
// round trips): within quads, eights, rows, then across rows to lane 63, whose
// value is returned to every lane.  All 64 lanes must be active.
template <bool MAX>
__device__ __forceinline__ uint32_t pair_op(uint32_t a, uint32_t b) {
    const uint32_t l = MAX ? max(a & 0xFFFFu, b & 0xFFFFu) : min(a & 0xFFFFu, b & 0xFFFFu);
    const uint32_t h = MAX ? max(a >> 16, b >> 16) : min(a >> 16, b >> 16);
    return l | h << 16;
}
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, CTRL, ROWS, 0xF, false);
}
template <bool MAX>
__device__ __forceinline__ uint32_t wave_reduce_u16x2(uint32_t v) {
    v = pair_op<MAX>(v, dpp_mov<0xB1, 0xF>(v));   // quad_perm [1,0,3,2]
    v = pair_op<MAX>(v, dpp_mov<0x4E, 0xF>(v));   // quad_perm [2,3,0,1]
    v = pair_op<MAX>(v, dpp_mov<0x141, 0xF>(v));  // row_half_mirror
    v = pair_op<MAX>(v, dpp_mov<0x140, 0xF>(v));  // row_mirror
    v = pair_op<MAX>(v, dpp_mov<0x142, 0xA>(v));  // row_bcast15 into rows 1, 3
    v = pair_op<MAX>(v, dpp_mov<0x143, 0xC>(v));  // row_bcast31 into rows 2, 3
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}
__device__ __forceinline__ uint32_t wave_min_u16x2(uint32_t v) { return wave_reduce_u16x2<false>(v); }
__device__ __forceinline__ uint32_t wave_max_u16x2(uint32_t v) { return wave_reduce_u16x2<true>(v); }
// v plus the DPP-moved value of v (0 where the source lane is outside the
// row or the lane's row is not in ROWS)
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_add(uint32_t v) {
    return v + (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROWS, 0xF, false);
}
// Inclusive prefix sum over the lanes of the wave (lane 0 first): shifts by 1,
// 2, 4, 8 within each row of 16, then the totals of earlier rows.  All 64
// lanes must be active.
__device__ __forceinline__ uint32_t wave_prefix_sum(uint32_t v) {
    v = dpp_add<0x111, 0xF>(v);  // row_shr:1
    v = dpp_add<0x112, 0xF>(v);  // row_shr:2
    v = dpp_add<0x114, 0xF>(v);  // row_shr:4
    v = dpp_add<0x118, 0xF>(v);  // row_shr:8
    v = dpp_add<0x142, 0xA>(v);  // row_bcast15: rows 1, 3 add the row before
    v = dpp_add<0x143, 0xC>(v);  // row_bcast31: rows 2, 3 add rows 0 and 1
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

// ------------------------------------------------------------------ one workgroup per image (small maps)
// k_encode_small: for C*H*W <= SMALL_MAX one workgroup of ENC_THREADS threads
// per image keeps the intensity map in LDS and does the whole code there:
//   1. (FILTER) the filter: the zero-padded image (as vertical pixel pairs)
//      and the taps in LDS; a work item is (channel, row, group of 8 columns)
//      with the lanes of a wave on consecutive rows, so their pixel reads fall
//      in distinct banks (odd row stride), and the channels taken in
//      decreasing order of their non-zero tap area.  Each output is the sum
//      over the channel's box of non-zero taps in ky-then-kx order, rounded
//      once to float: as exact int32 sums of (tap 2^s) * pixel by dot2 when
//      every tap allows it (the integer form), else accumulated in double.
//      A channel whose taps are exactly the negated taps of the channel before
//      it (the on/off pairs of a DoG bank) is not computed: its sum is the
//      exact negation, so its float is -v (+0 where v is 0).
//      (!FILTER) the intensities are loaded instead.
//   2. the T-1 bin boundaries: the keys at ranks ceil((j+1) n / T) of the
//      positive entries in descending key order, key = float bits << 13 |
//      (8191 - index) (unique; equal intensities rank in index order), up to
//      SEL_T boundaries at once.  The first 12-bit digit (key bits 43..32) of
//      every positive entry is counted (16-bit counters packed in pairs), and
//      a boundary's digit is found by the thread that holds the digit's
//      suffix count in registers.  When the entries with the boundaries'
//      digits are few (at most KCAP after padding), their low 32 key bits are
//      gathered per digit and a boundary is the key with the boundary's rank
//      among them (the number of larger keys).  Otherwise (many ties) an MSD
//      radix select resolves four more 8-bit digits, each revisiting only the
//      entries that matched (a candidate list, or all entries when it
//      overflows).
//   3. every entry's bin = the number of boundaries its key does not exceed,
//      i.e. floor(rho T / n) for rank rho (T for entries <= 0); t_first and the
//      T planes of the wave are written as 4-entry words.
constexpr int ENC_THREADS = 256;
constexpr int SEL_T = 16;        // boundaries resolved per select batch
constexpr int HBINS = 4096;      // first digit: 12 bits
constexpr int LCAP = 1024;       // candidate list capacity (entries)
constexpr int KCAP = LCAP;       // 32-bit keys of the targets' first digits ranked directly (same LDS)
constexpr int MAX_DERIV_C = 64;  // negated-channel detection and cost order for at most this many channels

// Global-to-LDS staging of n elements by one workgroup: a thread loads up to
// STAGE_U elements into registers before it stores any, so their memory
// latencies overlap (a load followed at once by its store waits each time).
constexpr int STAGE_U = 8;
template <typename Load, typename Store>
__device__ __forceinline__ void stage_batched(int n, Load ld, Store stv) {
    using V = decltype(ld(0));
    for (int i0 = threadIdx.x; i0 < n; i0 += STAGE_U * ENC_THREADS) {
        V v[STAGE_U];
#pragma unroll
        for (int k = 0; k < STAGE_U; ++k) {
            const int i = i0 + k * ENC_THREADS;
            v[k] = i < n ? ld(i) : V{};
        }
#pragma unroll
        for (int k = 0; k < STAGE_U; ++k) {
            const int i = i0 + k * ENC_THREADS;
            if (i < n) stv(i, v[k]);
        }
    }
}

__device__ __forceinline__ uint64_t key44(float v, int i) {
    return ((uint64_t)__float_as_uint(v) << 13) | (uint64_t)(8191 - i);
}

struct SmallFilter {
    int H, W, C, KF, Wp, nxg;  // image, channels, filter size, staged row stride (odd), 8-column groups
};

__host__ __device__ inline size_t up16(size_t v) { return (v + 15) & ~(size_t)15; }
__host__ __device__ inline int small_filter_wp(int W, int KF) {
    const int nxg = (W + 7) / 8;
    return (8 * nxg + KF + 6) | 1;
}
// LDS of the filter step (offsets in bytes): the taps as staged (float), which
// the double form's taps later replace; the zero-padded image as vertical
// pixel pairs (row r, row r + 1, as int16); the integer form's packed taps;
// per-channel integers.
struct SmallFiltLayout {
    size_t taps, pairs, itaps, ints, total;
};
constexpr int SF_INTS = 8;  // per channel: box (4), derived, order, tap offset, tap row stride
__host__ __device__ inline SmallFiltLayout small_filter_layout(int H, int W, int C, int KF) {
    const size_t KK = (size_t)KF * KF, img = (size_t)(H + KF - 1) * small_filter_wp(W, KF);
    SmallFiltLayout L;
    L.taps = 0;
    L.pairs = up16(C * KK * sizeof(double));
    L.itaps = L.pairs + up16(img * sizeof(uint32_t));
    L.ints = L.itaps + up16((size_t)C * ((KF + 1) / 2) * KF * sizeof(uint32_t));
    L.total = L.ints + (size_t)SF_INTS * C * sizeof(int);
    return L;
}
__host__ __device__ inline size_t small_filter_bytes(int H, int W, int C, int KF) {
    return small_filter_layout(H, W, C, KF).total;
}
// packed counters (SEL_T groups x 256 digits, or the 4096 first digits, as
// 16-bit halves), the 12-bit prefix table, two candidate lists
constexpr size_t SEL_HIST = (size_t)SEL_T * 256 * 2;
__host__ __device__ inline size_t small_select_bytes() { return SEL_HIST + HBINS + (size_t)2 * LCAP * 2; }

__device__ __forceinline__ int tap_area(const int *bbox, int c) {
    return max(0, bbox[4 * c + 1] - bbox[4 * c] + 1) * max(0, bbox[4 * c + 3] - bbox[4 * c + 2] + 1);
}
struct FiltCtx {
    int H, W, C, Wp;
    float thr;
    const uint32_t *pairs;  // zero-padded image as (pixel row r, row r + 1) int16 pairs, row stride Wp
    const void *taps;      // each computed channel's box of taps: packed pairs, or doubles in rows of stride tstr
    const int *bbox, *deriv, *toff, *tstr;
    double scale;          // integer form: 2^-s
    float *Ic, *gout;      // intensities in LDS, optionally in global memory
};

// Double form: NU consecutive taps of one filter row applied to 8 consecutive
// outputs; the 8 + NU - 1 pixels under them and the NU taps are all read
// before the first product, then the products in kx order.
template <int NU>
__device__ __forceinline__ void filter_taps(const uint32_t *row, const double *fr, double (&acc)[8]) {
    double a[8 + NU - 1], f[NU];
#pragma unroll
    for (int q = 0; q < 8 + NU - 1; ++q) a[q] = (double)(row[q] & 0xFFFFu);  // the pixel of row r
#pragma unroll
    for (int u = 0; u < NU; ++u) f[u] = fr[u];
#pragma unroll
    for (int u = 0; u < NU; ++u)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = fma(f[u], a[u + j], acc[j]);
}
// Integer form: NU tap pairs (rows ky, ky + 1 of NU consecutive columns)
// against the vertical pixel pairs under them, one dot2 per pair and output.
typedef short short2_t __attribute__((ext_vector_type(2)));
template <int NU>
__device__ __forceinline__ void int_taps(const uint32_t *row, const uint32_t *tr, int (&acc)[8]) {
    uint32_t a[8 + NU - 1], f[NU];
#pragma unroll
    for (int q = 0; q < 8 + NU - 1; ++q) a[q] = row[q];
#pragma unroll
    for (int u = 0; u < NU; ++u) f[u] = tr[u];
#pragma unroll
    for (int u = 0; u < NU; ++u)
#pragma unroll
        for (int j = 0; j < 8; ++j)
            acc[j] = __builtin_amdgcn_sdot2(__builtin_bit_cast(short2_t, a[u + j]), __builtin_bit_cast(short2_t, f[u]),
                                            acc[j], false);
}
// a row of wx taps in chunks of 8 and a last chunk of wx % 8, without a
// branch per tap
template <typename P, typename T, typename A, typename F8, typename FR>
__device__ __forceinline__ void tap_row(const P *row, const T *tr, int wx, A &acc, F8 &&full, FR &&rest) {
    int u0 = 0;
    for (; u0 + 8 <= wx; u0 += 8) full(row + u0, tr + u0, acc);
    rest(wx - u0, row + u0, tr + u0, acc);
}

// 8 consecutive outputs of row y, columns 8*xg.., of computed channel slot k
// (channel c, and the negated channel after it when that one is derived), the
// threshold applied.  Returns the number of positive outputs.
//  * double form: sums in ky-then-kx order over the channel's box of taps,
//    one rounding to float;
//  * integer form: int32 sums of tap 2^s times pixel, exact, times 2^-s and
//    rounded once to float -- the same value, every partial sum of the
//    double form being exact for such taps.
template <bool INT>
__device__ __forceinline__ int filter_item(const FiltCtx &fx, int k, int c, int xg, int y) {
    constexpr int CW = 8;
    const int ya = fx.bbox[4 * c], yb = fx.bbox[4 * c + 1], xa = fx.bbox[4 * c + 2], xb = fx.bbox[4 * c + 3];
    const int wx = xb - xa + 1;
    double val[CW];
    if constexpr (INT) {
        int acc[CW];
#pragma unroll
        for (int j = 0; j < CW; ++j) acc[j] = 0;
        const uint32_t *tp = reinterpret_cast<const uint32_t *>(fx.taps) + fx.toff[k];
        for (int ky = ya; ky <= yb; ky += 2) {
            const uint32_t *row = fx.pairs + (y + ky) * fx.Wp + CW * xg + xa;
            const uint32_t *tr = tp + ((ky - ya) >> 1) * wx;
            tap_row(row, tr, wx, acc, [](const uint32_t *r, const uint32_t *t, int(&a)[8]) { int_taps<8>(r, t, a); },
                    [](int n, const uint32_t *r, const uint32_t *t, int(&a)[8]) {
                        switch (n) {
                            case 1: int_taps<1>(r, t, a); break;
                            case 2: int_taps<2>(r, t, a); break;
                            case 3: int_taps<3>(r, t, a); break;
                            case 4: int_taps<4>(r, t, a); break;
                            case 5: int_taps<5>(r, t, a); break;
                            case 6: int_taps<6>(r, t, a); break;
                            case 7: int_taps<7>(r, t, a); break;
                            default: break;
                        }
                    });
        }
#pragma unroll
        for (int j = 0; j < CW; ++j) val[j] = (double)acc[j] * fx.scale;
    } else {
#pragma unroll
        for (int j = 0; j < CW; ++j) val[j] = 0.0;
        const double *fc = reinterpret_cast<const double *>(fx.taps) + fx.toff[k];
        const int ts = fx.tstr[k];
        for (int ky = ya; ky <= yb; ++ky) {
            const uint32_t *row = fx.pairs + (y + ky) * fx.Wp + CW * xg + xa;
            tap_row(row, fc + (ky - ya) * ts, wx, val,
                    [](const uint32_t *r, const double *t, double(&a)[8]) { filter_taps<8>(r, t, a); },
                    [](int n, const uint32_t *r, const double *t, double(&a)[8]) {
                        switch (n) {
                            case 1: filter_taps<1>(r, t, a); break;
                            case 2: filter_taps<2>(r, t, a); break;
                            case 3: filter_taps<3>(r, t, a); break;
                            case 4: filter_taps<4>(r, t, a); break;
                            case 5: filter_taps<5>(r, t, a); break;
                            case 6: filter_taps<6>(r, t, a); break;
                            case 7: filter_taps<7>(r, t, a); break;
                            default: break;
                        }
                    });
        }
    }
    const bool dn = c + 1 < fx.C && fx.deriv[c + 1];
    const int HW = fx.H * fx.W;
    int npos = 0;
#pragma unroll
    for (int j = 0; j < CW; ++j) {
        const int x = CW * xg + j;
        if (x >= fx.W) break;
        const float v = (float)val[j];
        const float o = v < fx.thr ? 0.0f : v;
        const int e = (c * fx.H + y) * fx.W + x;
        fx.Ic[e] = o;
        npos += o > 0.0f;
        if (fx.gout) fx.gout[e] = o;
        if (dn) {
            const float w = v == 0.0f ? 0.0f : -v;
            const float o2 = w < fx.thr ? 0.0f : w;
            fx.Ic[e + HW] = o2;
            npos += o2 > 0.0f;
            if (fx.gout) fx.gout[e + HW] = o2;
        }
    }
    return npos;
}

template <bool FILTER>
__global__ __launch_bounds__(ENC_THREADS, 4) void k_encode_small(const uint8_t *__restrict__ img, SmallFilter fg,
                                                             const float *__restrict__ filt, float thr,
                                                             const float *__restrict__ inten_in, int N, int T,
                                                             float *__restrict__ inten_out,
                                                             uint8_t *__restrict__ tf_out, uint8_t *__restrict__ wave) {
    static_assert(HBINS / 2 <= SEL_HIST / 4 && HBINS == 16 * ENC_THREADS, "first-digit counters");
    extern __shared__ uint4 lds4[];
    float *Ic = reinterpret_cast<float *>(lds4);  // N intensities
    unsigned char *r2 = reinterpret_cast<unsigned char *>(lds4) + up16((size_t)N * 4);
    __shared__ uint64_t kb[256];              // bin boundaries, zero past the last
    __shared__ uint64_t tpre[2][SEL_T];       // per target: digits found so far (by pass parity)
    __shared__ uint32_t trank[2][SEL_T];      // per target: rank among the keys with that prefix
    __shared__ uint64_t gpre[SEL_T];          // distinct target prefixes, descending
    __shared__ int tgrp[SEL_T];
    __shared__ uint32_t tcnt[SEL_T];          // per target: entries with its first digit
    __shared__ uint32_t gstart[SEL_T + 1], gcur[SEL_T];
    __shared__ int s_n, s_m, s_ng, s_total, s_lc[2], s_wsum[ENC_THREADS / 64];
    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    if (tid == 0) s_n = 0;
    for (int j = tid; j < 256; j += ENC_THREADS) kb[j] = 0;
    int npos = 0;

    if constexpr (FILTER) {
        const int H = fg.H, W = fg.W, C = fg.C, KF = fg.KF, Wp = fg.Wp, nxg = fg.nxg, KK = KF * KF;
        const int p = (KF - 1) / 2, Hs = H + KF - 1;
        const SmallFiltLayout L = small_filter_layout(H, W, C, KF);
        float *ft = reinterpret_cast<float *>(r2 + L.taps);
        uint32_t *pairs = reinterpret_cast<uint32_t *>(r2 + L.pairs);
        int *bbox = reinterpret_cast<int *>(r2 + L.ints);
        int *deriv = bbox + 4 * C;  // 1: the exact negation of the channel before, not computed
        int *order = deriv + C;     // computed channels, largest tap area first
        int *toff = order + C;      // per computed slot: offset of its taps
        int *tstr = toff + C;       // per computed slot: row stride of its taps (double form)
        __shared__ int s_ncomp, s_s;
        __shared__ uint32_t s_ex[MAX_DERIV_C];  // per channel: max fraction bits | (max exponent + 512) << 16
        // taps and the padded image (as vertical pixel pairs, zero past the last
        // row): each thread issues a batch's global loads before its LDS stores, so
        // a batch waits for memory once
        stage_batched(C * KK, [&](int i) { return filt[i]; }, [&](int i, float v) { ft[i] = v; });
        const uint8_t *im = img + (int64_t)b * H * W;
        stage_batched(
            Hs * Wp,
            [&](int i) {
                const int r = i / Wp, xp = i - r * Wp;
                const int y = r - p, x = xp - p;
                const bool in_x = x >= 0 && x < W;
                const uint32_t lo = in_x && y >= 0 && y < H ? im[y * W + x] : 0u;
                const uint32_t hi = in_x && y + 1 >= 0 && y + 1 < H ? im[(y + 1) * W + x] : 0u;
                return uint2{lo, hi};  // (combined at the store: a use here would wait for the load)
            },
            [&](int i, uint2 v) {
                uint32_t hi = v.y;
                asm volatile("" : "+v"(hi));  // keeps the shift here, out of the load's branch
                pairs[i] = v.x | hi << 16;
            });
        const bool order_c = C <= MAX_DERIV_C;  // negated channels, cost order and integer form only then
        __syncthreads();
        // per channel (one wave each): bounding box of the non-zero taps, whether the
        // taps are the exact negation of the previous channel's, and the integer
        // form's statistics (fraction bits and largest binary exponent of the taps)
        for (int c = wid; c < C; c += ENC_THREADS / 64) {
            int ya = KF, yb = -1, xa = KF, xb = -1, fb = 0, em = -400;
            bool neg = c > 0 && order_c;
            for (int i = lane; i < KK; i += 64) {
                const float f = ft[c * KK + i];
                if (f != 0.0f) {
                    const int ky = i / KF, kx = i - ky * KF;
                    ya = min(ya, ky); yb = max(yb, ky); xa = min(xa, kx); xb = max(xb, kx);
                    const uint32_t u = __float_as_uint(f), e = (u >> 23) & 255u, m = u & 0x7FFFFFu;
                    if (e == 255u) {
                        fb = 4095;  // not finite: the double form
                    } else {
                        const uint32_t mm = e ? (m | 0x800000u) : m;
                        const int e0 = (int)(e ? e : 1u) - 150;  // value = mm * 2^e0
                        fb = max(fb, -(e0 + (int)__builtin_ctz(mm)));
                        em = max(em, e0 + 31 - (int)__builtin_clz(mm));
                    }
                }
                if (c > 0) neg = neg && (f == -ft[(c - 1) * KK + i]);
            }
            // three reductions of 16-bit pairs: (ya, xa) by min, (yb + 1, xb + 1) and
            // (fraction bits, exponent + 512) by max
            const uint32_t lo = wave_min_u16x2((uint32_t)ya | ((uint32_t)xa << 16));
            const uint32_t hi = wave_max_u16x2((uint32_t)(yb + 1) | ((uint32_t)(xb + 1) << 16));
            const uint32_t ex = wave_max_u16x2((uint32_t)max(fb, 0) | ((uint32_t)(em + 512) << 16));
            const bool all_neg = __ballot(!neg) == 0;
            if (lane == 0) {
                bbox[4 * c] = (int)(lo & 0xFFFFu); bbox[4 * c + 1] = (int)(hi & 0xFFFFu) - 1;
                bbox[4 * c + 2] = (int)(lo >> 16); bbox[4 * c + 3] = (int)(hi >> 16) - 1;
                deriv[c] = all_neg ? 1 : 0;
                if (order_c) s_ex[c] = ex;
            }
        }
        __syncthreads();
        if (wid == 0) {
            if (order_c) {  // lane c: channel c
                // A negated channel is derived only from a computed one: in a run of
                // channels that each negate the one before, following a channel that
                // does not, every second one is derived.
                const bool neg = lane < C && deriv[lane] != 0;
                const uint64_t upto = lane == 63 ? ~0ull : (2ull << lane) - 1;
                const int c0 = 63 - __clzll(~__ballot(neg) & upto);  // channel 0 never negates
                const bool der = neg && ((lane - c0) & 1);
                const bool comp = lane < C && !der;
                // computed channels in decreasing order of tap area, equal areas by index
                const int area = comp ? tap_area(bbox, lane) : -1;
                // the integer form: every computed tap a multiple of 2^-s, |tap| 2^s <
                // 2^15, and KK * 255 * 2^(exponent + s + 1) < 2^31 bounds every sum
                const uint32_t ex = comp ? s_ex[lane] : 0u;
                const uint32_t exm = wave_max_u16x2(comp ? ex : (uint32_t)(112u << 16));  // (-400 + 512) << 16
                const int sfb = (int)(exm & 0xFFFFu), sem = (int)(exm >> 16) - 512;
                const bool exact = sfb <= 126 && sem + sfb <= 14 &&
                                   (sem + sfb + 1 < 0 || ((int64_t)KK * 255 << (sem + sfb + 1)) < (1LL << 31));
                const int wy = comp ? bbox[4 * lane + 1] - bbox[4 * lane] + 1 : 0;
                const int wxl = comp ? bbox[4 * lane + 3] - bbox[4 * lane + 2] + 1 : 0;
                const int size = area <= 0 ? 0 : exact ? ((wy + 1) >> 1) * wxl : area;
                int rank = 0, off = 0;
                for (int k = 0; k < C; ++k) {
                    const int ak = __builtin_amdgcn_readlane(area, k), sk = __builtin_amdgcn_readlane(size, k);
                    const bool before = ak > area || (ak == area && k < lane);
                    rank += before;
                    off += before && ak >= 0 ? sk : 0;
                }
                if (lane < C) {
                    deriv[lane] = der ? 1 : 0;
                    if (comp) {
                        order[rank] = lane;
                        toff[rank] = off;
                        tstr[rank] = wxl;
                    }
                }
                const int nc = __popcll(__ballot(comp));
                if (lane == 0) {
                    s_ncomp = nc;
                    s_s = exact ? sfb : -1;
                }
                if (exact) {
                    // this wave packs the integer form's taps (int16 pairs of tap rows ky,
                    // ky + 1; zero past the box), slot after slot, while the others wait
                    uint32_t *itp = reinterpret_cast<uint32_t *>(r2 + L.itaps);
                    const int bya = comp ? bbox[4 * lane] : 0, byb = comp ? bbox[4 * lane + 1] : 0;
                    const int bxa = comp ? bbox[4 * lane + 2] : 0;
                    for (int k = 0; k < nc; ++k) {
                        const int c = (int)__builtin_ctzll(__ballot(comp && rank == k));  // slot k's channel
                        const int ya = __builtin_amdgcn_readlane(bya, c), yb = __builtin_amdgcn_readlane(byb, c);
                        const int xa = __builtin_amdgcn_readlane(bxa, c), wk = __builtin_amdgcn_readlane(wxl, c);
                        const int n = ((yb - ya + 2) >> 1) * wk;
                        uint32_t *tp = itp + __builtin_amdgcn_readlane(off, c);
                        for (int e = lane; e < n; e += 64) {
                            const int kp = e / wk, u = e - kp * wk, ky = ya + 2 * kp;
                            const int q0 = (int)ldexpf(ft[c * KK + ky * KF + xa + u], sfb);
                            const int q1 = ky + 1 <= yb ? (int)ldexpf(ft[c * KK + (ky + 1) * KF + xa + u], sfb) : 0;
                            tp[e] = ((uint32_t)q0 & 0xFFFFu) | ((uint32_t)q1 << 16);
                        }
                    }
                }
            } else {  // every channel computed, in index order, double form with full rows
                for (int c = lane; c < C; c += 64) {
                    order[c] = c;
                    toff[c] = c * KK + max(bbox[4 * c], 0) * KF + max(bbox[4 * c + 2], 0);
                    tstr[c] = KF;
                }
                if (lane == 0) {
                    s_ncomp = C;
                    s_s = -1;
                }
            }
        }
        __syncthreads();
        const int ncomp = s_ncomp, sexp = s_s;
        const bool int_form = sexp >= 0;
        void *taps = r2 + (int_form ? L.itaps : L.taps);
        if (!int_form) {  // (the integer form's taps were packed with the order)
            // per computed channel: its box of taps as doubles (whole rows when C is
            // large), read from global memory since they replace the staged floats
            double *tp = reinterpret_cast<double *>(taps);
            for (int k = 0; k < ncomp; ++k) {
                const int c = order[k];
                if (order_c) {
                    const int ya = bbox[4 * c], xa = bbox[4 * c + 2], wxl = tstr[k];
                    const int n = max(0, (bbox[4 * c + 1] - ya + 1)) * wxl;
                    for (int e = tid; e < n; e += ENC_THREADS) {
                        const int r = e / wxl, u = e - r * wxl;
                        tp[toff[k] + e] = (double)filt[c * KK + (ya + r) * KF + xa + u];
                    }
                } else {
                    for (int e = tid; e < KK; e += ENC_THREADS) tp[c * KK + e] = (double)filt[c * KK + e];
                }
            }
            __syncthreads();  // (uniform)
        }
        float *gout = inten_out ? inten_out + (int64_t)b * N : nullptr;
        const FiltCtx fx{H, W, C, Wp, thr, pairs, taps, bbox, deriv, toff, tstr,
                         int_form ? ldexp(1.0, -sexp) : 1.0, Ic, gout};
        const int per_c = H * nxg, items = ncomp * per_c;
        for (int it = tid; it < items; it += ENC_THREADS) {
            const int slot = it / per_c, rem = it - slot * per_c;
            const int xg = rem / H, y = rem - xg * H;
            const int c = order[slot];
            npos += int_form ? filter_item<true>(fx, slot, c, xg, y) : filter_item<false>(fx, slot, c, xg, y);
        }
    } else {
        const float *I = inten_in + (int64_t)b * N;
        if ((N & 3) == 0) {  // four float4 loads in flight per thread before its stores
            const int n4 = N / 4;
            for (int q0 = tid; q0 < n4; q0 += 4 * ENC_THREADS) {
                float4 v[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int q = q0 + k * ENC_THREADS;
                    v[k] = q < n4 ? reinterpret_cast<const float4 *>(I)[q] : make_float4(0.f, 0.f, 0.f, 0.f);
                }
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int q = q0 + k * ENC_THREADS;
                    if (q < n4) reinterpret_cast<float4 *>(Ic)[q] = v[k];
                    npos += (v[k].x > 0.0f) + (v[k].y > 0.0f) + (v[k].z > 0.0f) + (v[k].w > 0.0f);
                }
            }
        } else {
            for (int i = tid; i < N; i += ENC_THREADS) {
                const float v = I[i];
                Ic[i] = v;
                npos += v > 0.0f;
            }
        }
    }
    uint32_t *hist = reinterpret_cast<uint32_t *>(r2);          // packed 16-bit counters
    uint8_t *tab = r2 + SEL_HIST;  // first digit -> group of this batch's targets (0xFF: none)
    uint16_t *lists = reinterpret_cast<uint16_t *>(tab + HBINS);  // two candidate lists of LCAP entries
    // (aliases the lists) key bits 31..0 of the entries with the targets' first digits
    uint32_t *ckey = reinterpret_cast<uint32_t *>(tab + HBINS);
    npos = spk::wave_sum_i32(npos);
    __syncthreads();  // the filter's LDS is free; s_n = 0 is seen by all
    if (lane == 0) atomicAdd(&s_n, npos);
    // first digit (key bits 43..32) of the positive entries, counted once
    for (int i = tid; i < HBINS / 2; i += ENC_THREADS) hist[i] = 0;
    __syncthreads();
    const int n = s_n, nb = T - 1;
    for (int i0 = tid; i0 < N; i0 += 4 * ENC_THREADS) {  // four reads in flight per thread
        float v[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = i0 + k * ENC_THREADS < N ? Ic[i0 + k * ENC_THREADS] : 0.0f;
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (v[k] > 0.0f) {
                const uint32_t d = (uint32_t)(key44(v[k], i0 + k * ENC_THREADS) >> 32);
                atomicAdd(&hist[d >> 1], 1u << (16 * (d & 1)));
            }
    }
    __syncthreads();
    // thread t holds digits 16t..16t+15: suffix counts S[q] = entries with digit >= 16t+q,
    // and beyond = entries with digit >= 16t+16
    uint32_t S[16], beyond;
    {
        uint32_t loc = 0;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const uint32_t w = hist[tid * 8 + q];
            S[2 * q] = w & 0xFFFFu;
            S[2 * q + 1] = w >> 16;
            loc += S[2 * q] + S[2 * q + 1];
        }
        const uint32_t pre = wave_prefix_sum(loc);  // over this wave's lanes <= lane
        const uint32_t wtot = (uint32_t)__builtin_amdgcn_readlane((int)pre, 63);
        if (lane == 0) s_wsum[wid] = (int)wtot;
        __syncthreads();
        uint32_t above = wtot - pre;  // this wave's lanes > lane
        for (int w = wid + 1; w < ENC_THREADS / 64; ++w) above += (uint32_t)s_wsum[w];
        beyond = above;
#pragma unroll
        for (int q = 15; q >= 0; --q) {
            above += S[q];
            S[q] = above;
        }
    }
    for (int j0 = 0; j0 < nb; j0 += SEL_T) {
        const int jn = min(SEL_T, nb - j0);
        if (wid == 0) {  // (j+1) n + T - 1 < 256 * 8192 + 256: 32-bit arithmetic is exact
            const bool act = lane < jn;
            const uint32_t r = act ? ((uint32_t)(j0 + lane + 1) * (uint32_t)n + (uint32_t)(T - 1)) / (uint32_t)T : 0u;
            if (act) {
                trank[0][lane] = r;  // ceil((j+1) n / T)
                tpre[0][lane] = 0;
            }
            // the targets with an entry at their rank are a prefix (ranks grow with j)
            const int m = __popcll(__ballot(act && r < (uint32_t)n));
            if (lane == 0) s_m = m;
        }
        for (int i = tid; i < HBINS / 4; i += ENC_THREADS) reinterpret_cast<uint32_t *>(tab)[i] = 0xFFFFFFFFu;
        for (int i = tid; i < KCAP / 4; i += ENC_THREADS) reinterpret_cast<uint4 *>(ckey)[i] = make_uint4(0, 0, 0, 0);
        __syncthreads();
        const int m = s_m;
        if (m == 0) continue;  // uniform
        {
            // the target whose rank r satisfies S[16t] > r >= S[16t+16] takes its digit
            // here; most threads hold none, and those skip the search
            uint32_t own = 0;
#pragma unroll
            for (int j = 0; j < SEL_T; ++j) {
                const uint32_t r = trank[0][j];
                own |= (j < m && S[0] > r && r >= beyond) ? (1u << j) : 0u;
            }
            while (own) {
                const int j = __builtin_ctz(own);
                own &= own - 1;
                const uint32_t r = trank[0][j];
                int q = 0;
#pragma unroll
                for (int k = 1; k < 16; ++k) q += S[k] > r;
                uint32_t sq = S[0], nxt = beyond;
#pragma unroll
                for (int k = 1; k < 16; ++k) {
                    sq = k == q ? S[k] : sq;
                    nxt = k == q + 1 ? S[k] : nxt;
                }
                trank[1][j] = r - nxt;
                tpre[1][j] = (uint64_t)(16 * tid + q);
                tcnt[j] = sq - nxt;  // entries with this digit
            }
        }
        __syncthreads();
        // The targets' digits, distinct ones numbered g = 0, 1, ... (descending); each
        // digit's entries get a segment of ckey from gstart[g], in that order, its
        // length rounded up to a multiple of 8 (the rest stays 0).
        if (tid < m) {
            uint64_t pp[SEL_T];
            uint32_t cc[SEL_T];
#pragma unroll
            for (int i = 0; i < SEL_T; ++i) {
                pp[i] = tpre[1][i];
                cc[i] = tcnt[i];
            }
            int g = 0;
            uint32_t start = 0;
#pragma unroll
            for (int i = 1; i < SEL_T; ++i)
                if (i <= tid && pp[i] != pp[i - 1]) {
                    ++g;
                    start += (cc[i - 1] + 7u) & ~7u;
                }
            tgrp[tid] = g;
            const uint64_t pt = tpre[1][tid];  // (from LDS: an index into pp or cc by tid would go to scratch)
            if (tid == 0 || pt != tpre[1][tid - 1]) {
                gstart[g] = start;
                gcur[g] = 0;
                gpre[g] = pt;
                tab[pt] = (uint8_t)g;
            }
            if (tid == m - 1) {
                s_ng = g + 1;
                s_total = (int)(start + ((tcnt[tid] + 7u) & ~7u));
                gstart[g + 1] = (uint32_t)s_total;
            }
        }
        __syncthreads();
        if (s_total <= KCAP) {  // uniform: rank the targets' digits' entries directly
            const int total = s_total, ng = s_ng;
            for (int i0 = tid; i0 < N; i0 += 4 * ENC_THREADS) {  // four entries in flight per thread
                float v[4];
                int g[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) v[k] = i0 + k * ENC_THREADS < N ? Ic[i0 + k * ENC_THREADS] : 0.0f;
#pragma unroll
                for (int k = 0; k < 4; ++k) g[k] = v[k] > 0.0f ? tab[key44(v[k], i0 + k * ENC_THREADS) >> 32] : 0xFF;
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    if (g[k] != 0xFF)
                        ckey[gstart[g[k]] + atomicAdd(&gcur[g[k]], 1u)] = (uint32_t)key44(v[k], i0 + k * ENC_THREADS);
            }
            __syncthreads();
            // Within a digit the keys differ in bits 31..0 only, so the rank of a key
            // there is the number of larger low words; the target with that rank takes
            // the key as its boundary.  The padding zeros exceed no key.
            for (int sl = tid; sl < total; sl += ENC_THREADS) {
                int g = 0;
#pragma unroll
                for (int k = 1; k < SEL_T; ++k) g += (k < ng && sl >= (int)gstart[k]) ? 1 : 0;
                const int g0 = (int)gstart[g], e1 = (int)gstart[g + 1];
                if (sl - g0 >= (int)gcur[g]) continue;  // padding
                const uint32_t key = ckey[sl];
                // eight keys per two 16-byte reads, two steps in flight
                const uint4 *c4 = reinterpret_cast<const uint4 *>(ckey);
                uint32_t rho = 0;
                int u = g0 / 4;
                const int u1 = e1 / 4;
                for (; u + 4 <= u1; u += 4) {
                    uint4 kk[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) kk[q] = c4[u + q];
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        rho += (kk[q].x > key) + (kk[q].y > key) + (kk[q].z > key) + (kk[q].w > key);
                }
                if (u < u1) {  // 8 keys left
                    const uint4 ka = c4[u], kc = c4[u + 1];
                    rho += (ka.x > key) + (ka.y > key) + (ka.z > key) + (ka.w > key);
                    rho += (kc.x > key) + (kc.y > key) + (kc.z > key) + (kc.w > key);
                }
                const uint64_t full = gpre[g] << 32 | key;
#pragma unroll
                for (int j = 0; j < SEL_T; ++j)
                    if (j < m && tgrp[j] == g && trank[1][j] == rho) kb[j0 + j] = full;
            }
            __syncthreads();
            continue;
        }
        // Many entries share the targets' digits (ties): resolve the remaining
        // digits 1..4 -- key bits 31..24, 23..16, 15..8, 7..0 -- per group of targets
        // sharing a prefix
        int src = -1;  // candidate list read by this digit (-1: all entries)
        for (int pass = 1; pass <= 4; ++pass) {
            const int shift = 32 - 8 * pass, cur = pass & 1, dst = src == 0 ? 1 : 0;
            if (tid < m) {  // group of target tid: distinct prefixes among targets 0..tid
                uint64_t pp[SEL_T];
#pragma unroll
                for (int i = 0; i < SEL_T; ++i) pp[i] = tpre[cur][i];
                const uint64_t pj = tpre[cur][tid];
                int g = 0;
#pragma unroll
                for (int i = 1; i < SEL_T; ++i) g += (i <= tid && pp[i] != pp[i - 1]) ? 1 : 0;
                tgrp[tid] = g;
                if (tid == 0 || pj != tpre[cur][tid - 1]) gpre[g] = pj;
                if (tid == m - 1) s_ng = g + 1;
            }
            if (tid == 0) s_lc[dst] = 0;
            for (int i = tid; i < SEL_T * 128; i += ENC_THREADS) hist[i] = 0;
            __syncthreads();
            const int ng = s_ng;
            const int cnt = src < 0 ? N : s_lc[src];
            for (int k = tid; k < cnt; k += ENC_THREADS) {
                const int i = src < 0 ? k : (int)lists[src * LCAP + k];
                const float v = Ic[i];
                if (!(v > 0.0f)) continue;
                const uint64_t key = key44(v, i), pre = key >> (shift + 8);
                int g = -1, lo = 0, hi = ng - 1;  // gpre is descending
                while (lo <= hi) {
                    const int mid = (lo + hi) >> 1;
                    const uint64_t gp = gpre[mid];
                    if (gp == pre) { g = mid; break; }
                    if (gp > pre) lo = mid + 1; else hi = mid - 1;
                }
                if (g < 0) continue;
                const uint32_t d = (uint32_t)(key >> shift) & 255u;
                atomicAdd(&hist[g * 128 + (d >> 1)], 1u << (16 * (d & 1)));
                if (pass < 4) {  // a candidate of the next digit
                    const int pos = atomicAdd(&s_lc[dst], 1);
                    if (pos < LCAP) lists[dst * LCAP + pos] = (uint16_t)i;
                }
            }
            __syncthreads();
            // one wave per group; lane l holds digits 4l..4l+3; the targets' ranks and
            // groups are read once, into registers
            uint32_t rr[SEL_T];
            int gg[SEL_T];
#pragma unroll
            for (int j = 0; j < SEL_T; ++j) {
                rr[j] = trank[cur][j];
                gg[j] = j < m ? tgrp[j] : -1;
            }
            for (int g = wid; g < ng; g += ENC_THREADS / 64) {
                uint32_t S[4], loc = 0;
                const uint32_t w0 = hist[g * 128 + 2 * lane], w1 = hist[g * 128 + 2 * lane + 1];
                S[0] = w0 & 0xFFFFu; S[1] = w0 >> 16; S[2] = w1 & 0xFFFFu; S[3] = w1 >> 16;
                loc = S[0] + S[1] + S[2] + S[3];
                const uint32_t pre = wave_prefix_sum(loc);
                const uint32_t beyond = (uint32_t)__builtin_amdgcn_readlane((int)pre, 63) - pre;  // lanes > lane
                uint32_t above = beyond;
#pragma unroll
                for (int q = 3; q >= 0; --q) {
                    above += S[q];
                    S[q] = above;
                }
#pragma unroll
                for (int j = 0; j < SEL_T; ++j) {
                    const uint32_t r = rr[j];
                    if (gg[j] == g && S[0] > r && r >= beyond) {
                        const int q = (S[1] > r) + (S[2] > r) + (S[3] > r);
                        const uint32_t nxt = q == 0 ? S[1] : q == 1 ? S[2] : q == 2 ? S[3] : beyond;
                        trank[cur ^ 1][j] = r - nxt;
                        tpre[cur ^ 1][j] = (tpre[cur][j] << 8) | (uint64_t)(4 * lane + q);
                    }
                }
            }
            __syncthreads();
            src = s_lc[dst] <= LCAP ? dst : -1;
        }
        if (tid < m) kb[j0 + tid] = tpre[1][tid];  // after 4 digits: pass 4 wrote parity 1
        __syncthreads();
    }
    __syncthreads();

    // bins (a fixed-step search over the boundaries padded with zeros to a power of
    // two, four entries interleaved), t_first and the wave
    int nbp = 1;  // a power of two > nb: the search counts 0..nbp-1 boundaries
    while (nbp <= nb) nbp <<= 1;
    uint8_t *tf = tf_out ? tf_out + (int64_t)b * N : nullptr;
    uint8_t *wv = wave ? wave + (int64_t)b * T * N : nullptr;
    if ((N & 3) == 0) {
        for (int q = tid; q < N / 4; q += ENC_THREADS) {
            const float4 v4 = reinterpret_cast<const float4 *>(Ic)[q];
            const float vv[4] = {v4.x, v4.y, v4.z, v4.w};
            uint64_t key[4];
            int pos[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                key[j] = key44(vv[j], 4 * q + j);
                pos[j] = 0;
            }
            for (int step = nbp >> 1; step > 0; step >>= 1)
#pragma unroll
                for (int j = 0; j < 4; ++j) pos[j] += kb[pos[j] + step - 1] >= key[j] ? step : 0;
            uint32_t t4 = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) t4 |= (uint32_t)(vv[j] > 0.0f ? pos[j] : T) << (8 * j);
            if (tf) *reinterpret_cast<uint32_t *>(tf + 4 * q) = t4;
            if (wv)
                for (int t = 0; t < T; ++t)
                    *reinterpret_cast<uint32_t *>(wv + (int64_t)t * N + 4 * q) = spk::spikes4(t4, t, T);
        }
    } else {
        for (int i = tid; i < N; i += ENC_THREADS) {
            const float v = Ic[i];
            const uint64_t key = key44(v, i);
            int pos = 0;
            for (int step = nbp >> 1; step > 0; step >>= 1) pos += kb[pos + step - 1] >= key ? step : 0;
            const int t = v > 0.0f ? pos : T;
            if (tf) tf[i] = (uint8_t)t;
            if (wv)
                for (int s2 = 0; s2 < T; ++s2) wv[(int64_t)s2 * N + i] = (uint8_t)(s2 >= t);
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

size_t small_rank_lds(int64_t N) { return spk::align_up((size_t)N * 4, 16) + small_select_bytes(); }

// The rank-order code of an intensity map: one workgroup per image when the
// map has at most SMALL_MAX entries, else the bin boundaries by radix select
// and a separate expansion.
void launch_rank(const float *I, int B, int64_t N, int T, uint8_t *t_first, uint8_t *wave, uint64_t *bounds,
                 uint32_t *count, hipStream_t st) {
    if (N <= SMALL_MAX) {
        hipLaunchKernelGGL(k_encode_small<false>, dim3(B), dim3(ENC_THREADS), small_rank_lds(N), st, nullptr,
                           SmallFilter{}, nullptr, 0.0f, I, (int)N, T, nullptr, t_first, wave);
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
    if ((t_first || wave) && p.N <= SMALL_MAX) {
        const size_t lds = spk::align_up((size_t)p.N * 4, 16) + std::max(small_filter_bytes(H, W, C, KF), small_select_bytes());
        if (lds <= SMALL_LDS) {  // the whole code in one kernel
            const SmallFilter fg{H, W, C, KF, small_filter_wp(W, KF), (W + 7) / 8};
            hipLaunchKernelGGL(k_encode_small<true>, dim3(B), dim3(ENC_THREADS), lds, st, image, fg, filters,
                               filter_threshold, nullptr, (int)p.N, T, intensities, t_first, wave);
            return spk::check_launch("spk_encode_latency");
        }
    }
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
