// Convolution of a cumulative spike wave + firing, fused (gfx950).
//
// Paper: section "snn Module" (per-step valid convolution over all time
// steps at once, Eq.2), "functional Module" (fire / threshold) and Eq.5
// (infinite threshold, in place).
//
// Formulation.  For output neuron (f, y, x) and step t
//     P[t,f,y,x] = sum_k W[f,k] * [tp_k <= t]
// where k runs over the receptive field and tp_k is the first-spike step of
// that input neuron (Eq.1 makes S[t] = [tp <= t]).  Per image this is a GEMM
// P_t[pos, f] = A_t[pos, k] * W^T[k, f] for every t, with a binary A_t made on
// the fly from the u8 first-spike map.  It runs on the 16-bit matrix cores: a
// spike is produced for two taps at once by one packed fp16 add with clamping,
// clamp((1025 + t) - (1024 + tp)), which is 1.0 exactly when tp <= t and 0
// otherwise.  The same bits (0x3C00) read as bf16 are 2^-7, so one spike
// operand serves both MFMA types.  The fp32 weights, scaled by a power of two,
// become the sum of two 16-bit terms hi = r(v), lo = r(v - hi) (v - hi is
// exact in float), the type chosen per call from the layer's largest and
// smallest non-zero |w| (both reduced on the device):
//   * fp16 terms (v_mfma_f32_16x16x32_f16) when every non-zero |w| is at
//     least 2^-15 times the largest one's power of two: each weight is then
//     carried to within 2^-22 of itself;
//   * otherwise bf16 terms (v_mfma_f32_16x16x32_bf16): bf16 has float's
//     exponent range, and two round-to-nearest 8-bit significands carry every
//     weight to within 2^-17 of itself (exactly when it has at most 17
//     significant bits), for every float weight when the largest |w| is below
//     2^8, else every |w| >= 2^-156 times the largest one's power of two.
// Products with a spike are exact either way; accumulation is fp32, and the
// scale is undone exactly.
//
// Pipeline of one call (all on the caller's stream):
//   1. k_pad_first_spike: wave [B,T,Cin,H,W] -> zero-padded first-spike map in
//      channel-last order, tpad [B][H+2p][W+2p][CP] (CP = Cin rounded up to 4
//      or to a multiple of 8; padding and padded channels hold T = never).
//      Taps are ordered k = (ky*K + kx)*CP + ci, so the 8 taps a lane feeds to
//      one MFMA are two 4-byte words of tpad.
//      The same launch reduces |W| to per-block maxima and non-zero minima
//      (extra workgroups).
//   2. W -> scaled 16-bit B-operand fragments (two terms) and the
//      per-lane word offsets of every 8-tap group: built by the
//      finite-threshold kernel itself when its fragments fit in LDS, else by
//      k_split_weights into the workspace.
//   3. finite threshold: k_conv_fire_fin (below); threshold = +inf (Eq.5):
//      k_conv_fire_inf, which computes only the last step.
#include <algorithm>
#include <cmath>
#include <mutex>
#include <numeric>
#include <type_traits>

#include "common.hpp"

namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int NTILE_ALIGN = 4;  // the N tiles (16 features) are padded to a multiple of this

// 16 bytes per lane from global memory into LDS at byte offset m0 + 16*lane.
// Issued as inline assembly so that the compiler, which cannot tell which LDS
// bytes the transfer writes, does not wait for it before every later LDS read;
// the caller waits for it explicitly (vmcnt) before the barrier that hands the
// buffer to the other waves.
__device__ __forceinline__ void lds_dma16(const uint4 *gsrc, uint32_t m0) {
    asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(gsrc), "{m0}"(m0) : "memory");
}

// A workgroup barrier for LDS hand-offs only: this wave's LDS operations
// complete, its global loads may stay in flight.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// s_waitcnt vmcnt(n) for a wave-uniform n (the immediate must be a constant)
__device__ __forceinline__ void wait_vmcnt(int n) {
    switch (n) {
#define SPK_VMCNT(k) \
    case k:          \
        asm volatile("s_waitcnt vmcnt(" #k ")" ::: "memory"); \
        break;
        SPK_VMCNT(8) SPK_VMCNT(12) SPK_VMCNT(20)
#undef SPK_VMCNT
    default:
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
}


struct ConvGeom {
    int B, T, Cin, H, W, Cout, K, pad;
    int S;           // stride: output (y, x) reads the padded window at (y*S, x*S)
    int CP;          // channels per tpad cell (Cin rounded up)
    int Hp, Wp, Ho, Wo, HoWo;
    int ksteps;      // ceil(K*K*CP / 32)
    int ntiles;      // ceil(Cout/16) rounded up to NTILE_ALIGN
    int mt_per_img;  // ceil(HoWo/16)
    int64_t total_mtiles;
    float thr;
};

// ------------------------------------------------------------------ 1. padded first-spike map
// Grid (chunk of padded rows, images).  A chunk is up to PAD_LDS bytes of
// whole padded rows (Wp*CP bytes each) of one image, contiguous in tpad.  The
// workgroup fills an LDS copy with T, writes T - (number of ones over the T
// steps) for every interior (ci, y, x) of the chunk (byte loads, consecutive
// threads on consecutive x), then stores the chunk with 16-byte stores; the
// LDS copy is shifted by the chunk's address mod 16 so that LDS and global
// 16-byte boundaries coincide.
constexpr int PAD_LDS = 32768;
constexpr int PAD_RAW = 8192;   // input bytes of one image staged in LDS at most

// LDS of the padding kernel: the padded rows of a chunk, then the raw map of a
// whole image when staged (a whole-image chunk of 4-byte words, at most PAD_RAW).
__host__ __device__ inline int pad_raw_offset(const ConvGeom &g, int rows_per_chunk) {
    return (rows_per_chunk * g.Wp * g.CP + 16 + 15) / 16 * 16;
}
__host__ __device__ inline bool pad_raw_fits(const ConvGeom &g, int nchunk) {
    return nchunk == 1 && (g.Cin * g.H * g.W) % 4 == 0 && g.Cin * g.H * g.W <= PAD_RAW;
}

// Workgroups past the nchunk * ny padding ones each write, for one run of wper
// weights, the bit patterns of the largest |w| to wmax[part] and of the
// smallest non-zero |w| to wmin[part] (0xFFFFFFFF if the run is all zeros):
// they fix the weights' scale and split (below).
constexpr int WMAX_PARTS = 2048;  // weight-range partials at most

// TIMES: the input is the first-spike map t_first [B][Cin][H][W] itself (T = never).
// 1D grid: workgroup (chunk, yb) = (id % nchunk, id / nchunk) pads images yb, yb + ny, ...
template <bool TIMES>
__global__ __launch_bounds__(256) void k_pad_first_spike(const uint8_t *__restrict__ wave, ConvGeom g,
                                                         int rows_per_chunk, int nchunk, int ny,
                                                         uint8_t *__restrict__ tpad, const float *__restrict__ w,
                                                         int64_t nw, int wper, unsigned *__restrict__ wmax,
                                                         unsigned *__restrict__ wmin) {
    // dynamic LDS: the chunk's padded rows (+16 for the alignment shift), then,
    // for a whole-image first-spike map that fits, the raw map (pad_lds_split)
    extern __shared__ uint4 pad_lds[];
    uint8_t *buf = reinterpret_cast<uint8_t *>(pad_lds);
    uint8_t *raw = buf + pad_raw_offset(g, rows_per_chunk);
    const int tid = threadIdx.x;
    if ((int)blockIdx.x >= nchunk * ny) {
        const int part = (int)blockIdx.x - nchunk * ny;
        const int64_t i1 = min(nw, (int64_t)(part + 1) * wper);
        unsigned m = 0, mn = 0xFFFFFFFFu;
        // four independent loads per thread and pass (at clamped indices, so that
        // none sits behind a branch that waits for it; the clamped ones count 0)
        for (int64_t i0 = (int64_t)part * wper + tid; i0 < i1; i0 += 1024) {
            float v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = w[min(i0 + 256 * j, i1 - 1)];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = i0 + 256 * j < i1 ? v[j] : 0.0f;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const unsigned b = __float_as_uint(fabsf(v[j]));
                m = max(m, b);
                mn = b ? min(mn, b) : mn;
            }
        }
#pragma unroll
        for (int s = 32; s >= 1; s >>= 1) {
            m = max(m, (unsigned)__shfl_xor((int)m, s, 64));
            mn = min(mn, (unsigned)__shfl_xor((int)mn, s, 64));
        }
        unsigned *red = reinterpret_cast<unsigned *>(buf);
        if ((tid & 63) == 0) {
            red[tid >> 6] = m;
            red[4 + (tid >> 6)] = mn;
        }
        __syncthreads();
        if (tid == 0) {
            wmax[part] = max(max(red[0], red[1]), max(red[2], red[3]));
            wmin[part] = min(min(red[4], red[5]), min(red[6], red[7]));
        }
        return;
    }
    const int row_bytes = g.Wp * g.CP;
    const int r0 = ((int)blockIdx.x % nchunk) * rows_per_chunk;
    const int nr = min(rows_per_chunk, g.Hp - r0);
    const int nbytes = nr * row_bytes;
    const int hw = g.H * g.W;
    // interior input rows of the chunk
    const int y_lo = max(r0 - g.pad, 0), y_hi = min(r0 + nr - g.pad, g.H);
    const int ncell = y_hi > y_lo ? g.Cin * (y_hi - y_lo) * g.W : 0;
    const uint32_t tfill = (uint32_t)g.T * 0x01010101u;
    for (int64_t b = (int)blockIdx.x / nchunk; b < g.B; b += ny) {
        uint8_t *out = tpad + (b * g.Hp + r0) * (int64_t)row_bytes;
        const int shift = (int)((uintptr_t)out & 15);
        for (int i = tid * 4; i < shift + nbytes; i += 1024) *reinterpret_cast<uint32_t *>(buf + i) = tfill;
        __syncthreads();
        const uint8_t *src = wave + b * (TIMES ? 1 : g.T) * (int64_t)g.Cin * hw;
        // A whole image's first-spike map is one contiguous block: it is read
        // with word loads, all issued before any is used, into LDS first.
        const bool staged = TIMES && pad_raw_fits(g, nchunk) && ((uintptr_t)src & 3) == 0;
        if (staged) {
            const int nwd = g.Cin * hw / 4;
            const uint32_t *s4 = reinterpret_cast<const uint32_t *>(src);
            uint32_t *r4 = reinterpret_cast<uint32_t *>(raw);
            for (int i0 = tid; i0 < nwd; i0 += 8 * 256) {
                uint32_t v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) v[u] = s4[min(i0 + 256 * u, nwd - 1)];  // (clamped: unconditional)
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (i0 + 256 * u < nwd) r4[i0 + 256 * u] = v[u];
            }
            __syncthreads();
            // one 4-channel word of the padded map per item: (cell, channel quad)
            const int nq = g.CP / 4;
            for (int wi = tid; wi < hw * nq; wi += 256) {
                const int yx = wi / nq, cq = wi - yx * nq;
                const int y = yx / g.W, x = yx - y * g.W;
                uint32_t word = 0;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int ci = cq * 4 + j;
                    const int tp = ci < g.Cin ? min((int)raw[ci * hw + yx], g.T) : g.T;
                    word |= (uint32_t)tp << (8 * j);
                }
                *reinterpret_cast<uint32_t *>(buf + shift + ((y + g.pad) * g.Wp + x + g.pad) * g.CP + cq * 4) = word;
            }
        }
        for (int i = tid; i < (staged ? 0 : ncell); i += 256) {
            const int x = i % g.W, rest = i / g.W;
            const int yy = rest % (y_hi - y_lo), ci = rest / (y_hi - y_lo);
            const int y = y_lo + yy;
            const uint8_t *p = src + ci * hw + y * g.W + x;
            int tp;
            if (TIMES) {
                tp = min((int)*p, g.T);
            } else {
                int cnt = 0;
#pragma unroll 5
                for (int t = 0; t < g.T; ++t) cnt += p[(int64_t)t * g.Cin * hw] != 0;
                tp = g.T - cnt;  // a cumulative wave has exactly T - t_first ones
            }
            buf[shift + ((y + g.pad - r0) * g.Wp + x + g.pad) * g.CP + ci] = (uint8_t)tp;
        }
        __syncthreads();
        const int head = min(nbytes, (16 - shift) & 15);
        const int body = (nbytes - head) & ~15;
        for (int i = tid; i < head; i += 256) out[i] = buf[shift + i];
        for (int i = head + tid * 16; i < head + body; i += 4096)
            *reinterpret_cast<uint4 *>(out + i) = *reinterpret_cast<const uint4 *>(buf + shift + i);
        for (int i = head + body + tid; i < nbytes; i += 256) out[i] = buf[shift + i];
        __syncthreads();
    }
}

// ------------------------------------------------------------------ 2. weight fragments
// Weight split of a call, from the bit patterns of the largest |w| (maxbits)
// and the smallest non-zero |w| (minbits; 0xFFFFFFFF when all are zero).
// With E the exponent of max|w|, each weight w becomes v = w * 2^e, split into
// hi = r(v) and lo = r(v - hi), r rounding to nearest even (v - hi is exact in
// float):
//   * fp16 terms: e = 12 - E, so the largest |v| lies in [2^12, 2^13).  For
//     |v| >= 2^-3 both terms keep 11 significant bits (lo, if subnormal, is
//     still within 2^-25 <= 2^-22 |v|), so |v - hi - lo| <= 2^-22 |v|.  Taken
//     when every non-zero |w| >= 2^(E-15) and |E| <= 100.
//   * bf16 terms otherwise: e = 60 - max(E, -60), so |v| < 2^61.  With v in
//     [2^m, 2^(m+1)), |v - hi| <= 2^(m-8); below 2^(m-8) v - hi has an ulp of
//     at most 2^(m-16), so |v - hi - lo| <= 2^(m-17) <= 2^-17 |v| (and v - hi
//     is exact at 2^(m-8)).  A v of at most 17 significant bits is carried
//     exactly.  For |w| >= 2^(E-156) (every float when E <= 7) every non-zero
//     term is at least 2^-119, normal even times a spike's 2^-7.  A spike is
//     2^-7 as bf16, so the sums are scaled by 2^(e - 7).
// inv_s undoes the scale (a power of two, exact).
// The fp32 form (arith == 1, finite threshold only: the dense fp32 contraction,
// kept to compare with the split) takes the weights unscaled as one fp32 term
// on v_mfma_f32_16x16x4_f32, eight products per 8-tap fragment.
constexpr int WK_F16 = 0, WK_BF16 = 1, WK_F32 = 2;  // weight term kinds
struct WSplit {
    int kind;
    int e;
    float inv_s;
};

__device__ __forceinline__ WSplit weight_split(unsigned maxbits, unsigned minbits, int arith = 0) {
    if (arith == 1) return {WK_F32, 0, 1.0f};
    const int E = maxbits ? (int)((maxbits >> 23) & 255u) - 127 : 0;  // subnormal maxima count as 2^-127
    if (E >= -100 && E <= 100 && minbits >= ((unsigned)(E - 15 + 127) << 23))
        return {WK_F16, 12 - E, ldexpf(1.0f, E - 12)};
    const int e = 60 - max(E, -60);
    return {WK_BF16, e, ldexpf(1.0f, 7 - e)};
}

// Largest of the n maximum partials and smallest of the n minimum partials,
// returned to every thread of the workgroup (blockDim.x a multiple of 64;
// red: 2 * blockDim.x / 64 words of LDS).
__device__ uint2 reduce_wrange(const unsigned *__restrict__ pmax, const unsigned *__restrict__ pmin, int n,
                               unsigned *red) {
    unsigned m = 0, mn = 0xFFFFFFFFu;
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
        m = max(m, pmax[i]);
        mn = min(mn, pmin[i]);
    }
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) {
        m = max(m, (unsigned)__shfl_xor((int)m, s, 64));
        mn = min(mn, (unsigned)__shfl_xor((int)mn, s, 64));
    }
    const int nw = (int)(blockDim.x >> 6);
    if ((threadIdx.x & 63) == 0) {
        red[threadIdx.x >> 6] = m;
        red[nw + (threadIdx.x >> 6)] = mn;
    }
    __syncthreads();
    m = 0;
    mn = 0xFFFFFFFFu;
    for (int i = 0; i < nw; ++i) {
        m = max(m, red[i]);
        mn = min(mn, red[nw + i]);
    }
    __syncthreads();
    return uint2{m, mn};
}

// bf16 bits of v rounded to nearest even (v finite, |v| < 2^127).
__device__ __forceinline__ uint32_t bf16_bits(float v) {
    const uint32_t u = __float_as_uint(v);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Tap (K-step ks, lane group gq, j) of the padded receptive field -> (cell kyx,
// channel ci).  In general k = ks*32 + 8*gq + j is cell k / CP, channel k % CP.
// When CP is a multiple of 32 the CP/32 K-steps of a cell are laid out so that
// a lane group's channels are contiguous over the whole cell: channel
// gq*CP/4 + 8*(ks mod CP/32) + j, i.e. a lane reads CP/4 consecutive bytes of
// tpad per cell (the same order as the general one when CP == 32).
__device__ __forceinline__ void tap_of(const ConvGeom &g, int ks, int gq, int j, int &kyx, int &ci) {
    if (g.CP % 32 == 0) {
        const int kpc = g.CP / 32;
        kyx = ks / kpc;
        ci = gq * (g.CP / 4) + (ks % kpc) * 8 + j;
    } else {
        const int k = ks * 32 + gq * 8 + j;
        kyx = k / g.CP;
        ci = k % g.CP;
    }
}

// Tap k of the padded receptive field: cell kyx, channel ci (tap_of).
// koff2[q] holds, for the 8-tap group q = 4*ks + gq, the tpad byte offsets (relative
// to the output position's top-left input cell) of its two 4-byte words; with
// CP >= 8 they are adjacent, with CP == 4 they are the cells 2q and 2q+1.
// Groups past the receptive field point at offset 0 (their weights are 0).
//
// Fragment (nt, ks, lane) holds, for feature n = nt*16 + lane%16, the 8 taps
// k = ks*32 + 8*(lane/16) + j, j = 0..7, as two 16-bit terms (each a uint4 of
// 8 fp16 or bf16 values), or as 8 floats (taps 0-3, then 4-7) in the fp32 form.  w holds the weights of features n0, n0 + 1, ...
// ([Cout - n0][Cin][K][K]).
constexpr int NT = 2;  // 16-bit terms per weight

// Tap j (0..7) of a fragment lane: the weight w (unscaled) into the terms'
// words t[q][j / 2] (16-bit halves), or t[j / 4][j % 4] as a float (fp32 form).
__device__ __forceinline__ void split_tap(float w, int j, const WSplit &s, uint32_t (&t)[NT][4]) {
    const float v = ldexpf(w, s.e);
    if (s.kind == WK_F32) {  // taps 0-3 in out[0], 4-7 in out[1], as floats
        t[j >> 2][j & 3] = __float_as_uint(v);
        return;
    }
    uint32_t h[NT];
    if (s.kind == WK_F16) {
        const _Float16 hv = (_Float16)v;
        const float rest = v - (float)hv;  // exact: hv is within half an fp16 ulp of v
        h[0] = __builtin_bit_cast(uint16_t, hv);
        h[1] = __builtin_bit_cast(uint16_t, (_Float16)rest);
    } else {
        h[0] = bf16_bits(v);
        h[1] = bf16_bits(v - __uint_as_float(h[0] << 16));  // v - hi exact, at most 16 significant bits
    }
#pragma unroll
    for (int q = 0; q < NT; ++q) t[q][j >> 1] |= h[q] << (16 * (j & 1));
}

__device__ __forceinline__ void split_fragment(const float *w, int n0, const ConvGeom &g, int nt, int ks, int lane,
                                               const WSplit &s, uint4 (&out)[NT]) {
    const int KK = g.K * g.K;
    const int n = nt * 16 + (lane & 15);
    uint32_t t[NT][4] = {};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        int kyx, ci;
        tap_of(g, ks, lane >> 4, j, kyx, ci);
        const float v = n < g.Cout && kyx < KK && ci < g.Cin ? w[((int64_t)(n - n0) * g.Cin + ci) * KK + kyx] : 0.0f;
        split_tap(v, j, s, t);
    }
#pragma unroll
    for (int q = 0; q < NT; ++q) out[q] = uint4{t[q][0], t[q][1], t[q][2], t[q][3]};
}

// Word offsets of the 8-tap group q (koff2 below).
__device__ __forceinline__ int2 koff_of(const ConvGeom &g, int q) {
    const int KK = g.K * g.K;
    int2 o{0, 0};
    auto cell = [&](int kyx) { return kyx < KK ? ((kyx / g.K) * g.Wp + kyx % g.K) * g.CP : 0; };
    if (g.CP >= 8) {
        int kyx, ci0;
        tap_of(g, q / 4, q % 4, 0, kyx, ci0);
        o.x = kyx < KK ? cell(kyx) + ci0 : 0;
        o.y = kyx < KK ? o.x + 4 : 0;
    } else {
        o.x = cell(2 * q);
        o.y = cell(2 * q + 1);
    }
    return o;
}

// Fragments of every 16-feature tile into the workspace, frag[nt][ks][term][64],
// the tap offsets, and the split's term type (1: bf16) and inverse scale.
__global__ __launch_bounds__(256) void k_split_weights(const float *__restrict__ w, ConvGeom g,
                                                       const unsigned *__restrict__ wmax,
                                                       const unsigned *__restrict__ wmin, int n_wmax,
                                                       uint4 *__restrict__ frag, int2 *__restrict__ koff2,
                                                       float *__restrict__ inv_scale, int *__restrict__ wbf16,
                                                       int arith) {
    __shared__ unsigned red[8];
    const uint2 mm = reduce_wrange(wmax, wmin, n_wmax, red);
    const WSplit ws = weight_split(mm.x, mm.y, arith);
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t total = (int64_t)g.ntiles * g.ksteps * 64;
    if (i == 0) {
        *inv_scale = ws.inv_s;
        *wbf16 = ws.kind;
    }
    if (i < total) {
        const int lane = (int)(i & 63);
        const int64_t r = i >> 6;
        uint4 t[NT];
        split_fragment(w, 0, g, (int)(r / g.ksteps), (int)(r % g.ksteps), lane, ws, t);
#pragma unroll
        for (int q = 0; q < NT; ++q) frag[(r * NT + q) * 64 + lane] = t[q];
    }
    if (i < (int64_t)g.ksteps * 4) koff2[i] = koff_of(g, (int)i);
}

// The same fragments when CP is a multiple of 32 (the cell-contiguous tap
// order of tap_of): there a fragment lane's 8 taps are 8 consecutive channels
// of one cell, so the block of channels 8cb..8cb+7 gives, for every cell, the
// 16 lanes (lane group cb / (CP/32)) of K-step cell * CP/32 + cb % (CP/32).
// One workgroup per (16-feature tile, channel block): per feature the block's
// weights (8 channels x KK cells) are contiguous, read coalesced into LDS;
// each (cell, term) then leaves as 16 consecutive fragment lanes (256 bytes).
constexpr int SPLIT_CELLS = 64;  // cells per LDS pass
__global__ __launch_bounds__(256) void k_split_weights_cells(const float *__restrict__ w, ConvGeom g,
                                                             const unsigned *__restrict__ wmax,
                                                             const unsigned *__restrict__ wmin, int n_wmax,
                                                             uint4 *__restrict__ frag, int2 *__restrict__ koff2,
                                                             float *__restrict__ inv_scale, int *__restrict__ wbf16) {
    __shared__ float wl[8 * SPLIT_CELLS * 17];  // [channel][cell][feature], rows of 17 (distinct banks)
    __shared__ unsigned red[8];
    const uint2 mm = reduce_wrange(wmax, wmin, n_wmax, red);
    const WSplit ws = weight_split(mm.x, mm.y, 0);
    const int tid = threadIdx.x, kpc = g.CP / 32, nb = g.CP / 8, KK = g.K * g.K;
    const int nt = (int)blockIdx.x / nb, cb = (int)blockIdx.x % nb;
    const int lane0 = (cb / kpc) * 16, m = cb % kpc;
    if (blockIdx.x == 0) {
        if (tid == 0) {
            *inv_scale = ws.inv_s;
            *wbf16 = ws.kind;
        }
        for (int i = tid; i < g.ksteps * 4; i += 256) koff2[i] = koff_of(g, i);
    }
    for (int c0 = 0; c0 < KK; c0 += SPLIT_CELLS) {
        const int nc = min(SPLIT_CELLS, KK - c0), nv = 16 * 8 * nc;
        // (feature, channel, cell) with the cell fastest: a feature's block is
        // contiguous in w; eight loads in flight per thread before its stores.
        // The index i = (f * 8 + j) * nc + cl is carried, not divided out.
        const int dcl = 256 % nc, dj = (256 / nc) % 8, dfe = 256 / (8 * nc);
        int cl = tid % nc, j = (tid / nc) % 8, f = tid / (8 * nc);
        auto step = [&](int &a, int &b, int &c) {
            a += dcl;
            if (a >= nc) {
                a -= nc;
                ++b;
            }
            b += dj;
            if (b >= 8) {
                b -= 8;
                ++c;
            }
            c += dfe;
        };
        for (int i0 = tid; i0 < nv; i0 += 8 * 256) {
            float v[8];
            int a = cl, bb = j, c = f;
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int n = nt * 16 + c, ci = cb * 8 + bb;
                v[u] = i0 + u * 256 < nv && n < g.Cout && ci < g.Cin ? w[((int64_t)n * g.Cin + ci) * KK + c0 + a] : 0.0f;
                step(a, bb, c);
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                if (i0 + u * 256 < nv) wl[(j * SPLIT_CELLS + cl) * 17 + f] = v[u];
                step(cl, j, f);
            }
        }
        __syncthreads();
        for (int i = tid; i < nc * 16; i += 256) {
            const int cl = i >> 4, f = i & 15;
            uint32_t t[NT][4] = {};
#pragma unroll
            for (int j = 0; j < 8; ++j) split_tap(wl[(j * SPLIT_CELLS + cl) * 17 + f], j, ws, t);
            const int64_t r = (int64_t)nt * g.ksteps + (c0 + cl) * kpc + m;
#pragma unroll
            for (int q = 0; q < NT; ++q) frag[(r * NT + q) * 64 + lane0 + f] = uint4{t[q][0], t[q][1], t[q][2], t[q][3]};
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------ shared MFMA helpers
// fp16 -(1024 + tp) for the four tap bytes of a word, as two packed pairs.
__device__ __forceinline__ void neg_times(uint32_t w, uint32_t &lo, uint32_t &hi) {
    lo = __builtin_amdgcn_perm(0xE4E4E4E4u, w, 0x05010400u);
    hi = __builtin_amdgcn_perm(0xE4E4E4E4u, w, 0x05030402u);
}

// Spike operand of 8 taps at step t: clamp((1025 + t) - (1024 + tp)) per tap,
// fp16 1.0 / 0 (as bf16: 2^-7 / 0).
__device__ __forceinline__ u4 spike_operand(const uint32_t (&xn)[4], uint32_t ct) {
    u4 a;
    asm("v_pk_add_f16 %0, %1, %2 clamp" : "=v"(a.x) : "v"(ct), "v"(xn[0]));
    asm("v_pk_add_f16 %0, %1, %2 clamp" : "=v"(a.y) : "v"(ct), "v"(xn[1]));
    asm("v_pk_add_f16 %0, %1, %2 clamp" : "=v"(a.z) : "v"(ct), "v"(xn[2]));
    asm("v_pk_add_f16 %0, %1, %2 clamp" : "=v"(a.w) : "v"(ct), "v"(xn[3]));
    return a;
}

// fp16 (1025 + t) in both halves (t <= 1022)
__device__ __forceinline__ uint32_t step_const(int t) { return (0x6401u + (uint32_t)t) * 0x10001u; }

// One 16x16x32 product of a spike operand with one weight term (fp16 or bf16).
template <int KIND>
__device__ __forceinline__ f4 mfma(u4 a, uint4 b, f4 c) {
    if constexpr (KIND == WK_F16)
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8, a), __builtin_bit_cast(half8, b), c, 0,
                                                      0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, a), __builtin_bit_cast(bf8, b), c, 0, 0,
                                                       0);
}

// ------------------------------------------------------------------ 3a. finite threshold
// One workgroup = 8 MFMA waves + 8 store waves, persistent, serving one pair
// of 16-feature tiles (32 features).  A task is a run of up to 16 position
// tiles: a whole image when it has at most 16 tiles, else a chunk of the
// flattened (image, position) space that may span two images (no padded
// tiles); the workgroup takes its tasks from its XCD's slice of the list.
// For every block of TB time steps:
//   * each MFMA wave computes the GEMM of its tiles (local tiles w and w+8)
//     for the 32 features and TB steps -- spike words from the task's rows,
//     staged in LDS one task ahead (or straight from tpad), weight fragments
//     from LDS (or L2 when they do not fit) -- and writes the scaled
//     potentials into the LDS staging area [TB][32 features][row stride];
//   * the store waves then fire the staged potentials (threshold, first spike,
//     potential at the first spike, kept in their registers for the whole
//     task) and write potentials and spikes of each step as contiguous runs
//     (one run per feature row; a whole-image task is one region), while the
//     MFMA waves go on with the next block.
// Keeping every global store in the store waves keeps the MFMA waves' own
// memory counter free of store acknowledgements, so their operand loads never
// wait behind the output stream.  Two barriers per block: "staging free"
// (the store waves are done with the previous block) and "staging full".
// LDS bank conflicts are avoided on both sides of the LDS traffic: the
// staging rows have a stride whose quotient by 4 is odd, and the staged spike
// rows are stored channel-group major (see k_conv_fire_fin's ALDS buffers).
// Two waves per SIMD do the firing and storing: their VALU work and LDS
// waits overlap each other's.
constexpr int FIN_TB = 3;          // time steps per block (staging depth)
constexpr int FIN_CW = 8;          // MFMA waves (waves 0-7)
constexpr int FIN_MT = 2;          // position tiles per MFMA wave
constexpr int FIN_SW = 8;          // store waves (waves 8-15)
constexpr int FIN_THREADS = (FIN_CW + FIN_SW) * 64;
// position tiles per task at most: 16 with 4-element store groups, 8 with single elements
__host__ __device__ constexpr int chunk_tiles_max(int G) { return G == 4 ? 16 : 8; }
// Row stride (floats) of a feature's positions in the staging area: at least np,
// a multiple of 4 with an odd quotient, so that the 16 feature lanes of an
// epilogue 16-byte write fall in distinct LDS bank groups.
__host__ __device__ constexpr int stage_stride(int np) { return (((np + 3) / 4) | 1) * 4; }

// Work of an MFMA wave on (tile slot i, 16-feature half n) in second-slot mode M
// (0 both halves, 1 the first, 2 the second, 3 none): the first slot always has both.
template <int M>
__device__ constexpr bool fin_unit(int i, int n) {
    return i == 0 || M == 0 || (M == 1 && n == 0) || (M == 2 && n == 1);
}
static_assert(FIN_MT == 2, "the tile slots of an MFMA wave are wv and wv + FIN_CW");

// First-spike pooling fused into the finite-threshold call (window P = stride,
// no padding; P == 0: none).  Tasks are then bands of whole pooling rows of one
// image, so every window lies in one task: the store waves put a task's
// first-spike times into an LDS map [32 features][np_max] and pool them after
// the next barrier of the workgroup (the last task's after one more barrier).
// With vec, each thread pools 4 consecutive positions of a feature's run of
// the band (the band's pooled rows, contiguous in the map) and writes them,
// and each step's Eq.1 word of them, as 4-byte stores.
struct PoolOut {
    int P;          // window and stride (0: no pooling)
    int Hpo, Wpo;   // pooled map size, floor(Ho / P) x floor(Wo / P)
    int vec;        // 4 pooled positions per thread (aligned maps, runs of a multiple of 4 at 4-byte offsets)
    uint8_t *tf;    // pooled first-spike times [B][Cout][Hpo][Wpo]
    uint8_t *wave;  // pooled Eq.1 wave [B][T][Cout][Hpo][Wpo], or null
};

// Kernel forms: the 16-bit split (FIN_SPLIT), the split with fused pooling
// (FIN_POOL) and the fp32 form (FIN_F32), each compiled on its own so that the
// code of the others costs the plain form no registers.
constexpr int FIN_SPLIT = 0, FIN_POOL = 1, FIN_F32 = 2;

template <int G, bool BLDS, bool ALDS, int MODE>
__global__ __launch_bounds__(FIN_THREADS, 1) void k_conv_fire_fin(
    const uint8_t *__restrict__ tpad, const uint4 *__restrict__ frag, const int2 *__restrict__ koff2, ConvGeom g,
    int n_pairs, int n_chunks, int cpi, int chunk_tiles, int band_pos, int np_max, int a_words,
    const float *__restrict__ inv_scale, const int *__restrict__ wbf16, const float *__restrict__ wts,
    const unsigned *__restrict__ wmax, const unsigned *__restrict__ wmin, int n_wmax, float *__restrict__ P,
    uint8_t *__restrict__ S, uint8_t *__restrict__ TF, float *__restrict__ VF, PoolOut po, int arith) {
    extern __shared__ uint4 lds[];
    const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63;
    const int gq = lane >> 4, c = lane & 15;
    int2 *koff_l = reinterpret_cast<int2 *>(lds);
    uint4 *frag_l = lds + (g.ksteps * 4 * 8 + 15) / 16;  // [ks][n(2)][term(NT)][64] (BLDS)
    float *stage = reinterpret_cast<float *>(frag_l + (BLDS ? g.ksteps * 2 * NT * 64 : 0));  // [TB][32*np_max]
    const int stage_t = 32 * stage_stride(np_max);
    // ALDS: 2 buffers of a_words words (a multiple of 64) holding a task's
    // padded rows channel-group major, [row][CP/8][Wp][8 bytes], so that the 16
    // consecutive positions of an 8-byte A read are 128 contiguous bytes.
    uint32_t *abuf = reinterpret_cast<uint32_t *>(stage + FIN_TB * stage_t);
    // pooling: a task's first-spike times, [32 features][np_max]
    uint8_t *pool_l = reinterpret_cast<uint8_t *>(abuf + (ALDS ? 2 * a_words : 0));
    const int row_bytes = g.Wp * g.CP;

    const int x = blockIdx.x % 8, j = blockIdx.x / 8;
    const int pair = j % n_pairs, r = j / n_pairs, R = (int)(gridDim.x / 8) / n_pairs;
    const int ntask = n_chunks;
    const int per_x = (ntask + 7) / 8;
    const int t_lo = x * per_x, t_hi = min(ntask, t_lo + per_x);
    const int f0 = pair * 32;
    const int nf = min(32, g.Cout - f0);
    const int npos = g.B * g.HoWo;  // flattened (image, position) index space

    // A task is the flattened positions [p0, p0 + np): with cpi > 0, chunk
    // task % cpi of image task / cpi; with cpi == 0, chunk `task` of the
    // flattened space, which may span two images.  Chunks are band_pos
    // positions (whole rows) when band_pos > 0, else chunk_tiles tiles.
    auto task_range = [&](int task, int &p0, int &np) {
        if (cpi > 0 && band_pos > 0) {
            const int b = task / cpi, q0 = (task - b * cpi) * band_pos;
            p0 = b * g.HoWo + q0;
            np = min(band_pos, g.HoWo - q0);
        } else if (cpi > 0) {
            const int b = task / cpi, q0 = (task - b * cpi) * chunk_tiles * 16;
            p0 = b * g.HoWo + q0;
            np = min(chunk_tiles * 16, g.HoWo - q0);
        } else {
            const int cp = band_pos > 0 ? band_pos : chunk_tiles * 16;
            p0 = task * cp;
            np = min(cp, npos - p0);
        }
    };
    // The padded first-spike rows it reads: from row y_first of its first image
    // to row y_last+K-1 of its last one, one contiguous range of tpad (rows of
    // consecutive images follow each other; a multiple of 4 bytes).
    auto region = [&](int task, int &row0, int &w0, int &nw) {
        int p0, np;
        task_range(task, p0, np);
        const int pa = p0, pb = p0 + np - 1;
        const int ba = pa / g.HoWo, bb = pb / g.HoWo;
        row0 = ba * g.Hp + (pa - ba * g.HoWo) / g.Wo * g.S;
        const int row1 = bb * g.Hp + (pb - bb * g.HoWo) / g.Wo * g.S + g.K - 1;
        w0 = (int)(((int64_t)row0 * row_bytes) >> 2);
        nw = (row1 - row0 + 1) * row_bytes / 4;
    };
    // Direct global-to-LDS loads of a task's rows into `dst` by the MFMA waves
    // (lane i of a load writes word d0 + i); they complete before the barrier
    // that precedes the buffer's first use (s_waitcnt vmcnt(0) ahead of it).
    auto fill_region = [&](int task, uint32_t *dst) {
        int row0, w0, nw;
        region(task, row0, w0, nw);
        const uint32_t *src = reinterpret_cast<const uint32_t *>(tpad) + (uint32_t)w0;
        const int rw = row_bytes / 4, gw = 2 * g.Wp, cw = g.CP / 4;
        for (int d0 = wv * 64; d0 < nw; d0 += FIN_CW * 64) {
            const int d = min(d0 + lane, nw - 1);  // lanes past the region repeat its last word
            const int rr = d / rw, rem = d - rr * rw;
            const int cg = rem / gw, rem2 = rem - cg * gw;
            __builtin_amdgcn_global_load_lds(src + rr * rw + (rem2 >> 1) * cw + cg * 2 + (rem2 & 1), dst + d0, 4, 0,
                                             0);
        }
    };
    if (ALDS && wv < FIN_CW && t_lo + r < t_hi) fill_region(t_lo + r, abuf);
    if (ALDS) {  // tap offsets in the LDS copy: 8 channels (one channel group of a cell) per lane
        const int KK = g.K * g.K;
        for (int i = tid; i < g.ksteps * 4; i += FIN_THREADS) {
            int kyx, ci0;
            tap_of(g, i >> 2, i & 3, 0, kyx, ci0);
            const int ox = kyx < KK ? (kyx / g.K) * row_bytes + (ci0 >> 3) * g.Wp * 8 + (kyx % g.K) * 8 : 0;
            koff_l[i] = int2{ox, ox + 4};
        }
    } else {
        for (int i = tid; i < g.ksteps * 4; i += FIN_THREADS) koff_l[i] = koff_of(g, i);
    }
    float inv_s;
    int kind;
    if (BLDS) {  // the pair's fragments, split here from the weights: [ks][n][term][64]
        // (the staging area, unused until the main loop, holds the reduction's words)
        const uint2 mm = reduce_wrange(wmax, wmin, n_wmax, reinterpret_cast<unsigned *>(stage));
        const WSplit ws = weight_split(mm.x, mm.y, arith);
        inv_s = ws.inv_s;
        kind = ws.kind;
        // the pair's weights, contiguous in W, go through the staging area when
        // they fit (coalesced loads instead of one load per tap)
        const int per_f = g.Cin * g.K * g.K, nwp = nf * per_f;
        const bool wl = nwp <= FIN_TB * stage_t;
        if (wl) {
            for (int i = tid; i < nwp; i += FIN_THREADS) stage[i] = wts[(int64_t)f0 * per_f + i];
            __syncthreads();
        }
        const float *wsrc = wl ? stage : wts + (int64_t)f0 * per_f;
        for (int i = tid; i < g.ksteps * 2 * 64; i += FIN_THREADS) {
            const int ln = i & 63, rr = i >> 6;  // rr = ks*2 + n
            uint4 t[NT];
            split_fragment(wsrc, f0, g, pair * 2 + (rr & 1), rr >> 1, ln, ws, t);
#pragma unroll
            for (int q = 0; q < NT; ++q) frag_l[(rr * NT + q) * 64 + ln] = t[q];
        }
    } else {
        inv_s = *inv_scale;
        kind = *wbf16;
    }
    if (ALDS) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    const int64_t tplane = (int64_t)g.Cout * g.HoWo;

    if (wv < FIN_CW) {
        // ------------------------------------------------ MFMA waves
        // Every wave computes up to two tiles of 16 positions for the 32 features;
        // positions of a tile past the chunk repeat its last position and are
        // never stored, which keeps the MFMA stream free of branches.  The K-step
        // loop is compiled once per term kind (fp16 / bf16 / fp32) and second-slot
        // mode (below).
        const uint4 *gf = frag + (int64_t)(pair * 2) * g.ksteps * NT * 64 + lane;
        auto mfma_waves = [&](auto kind_c) {
        constexpr int KIND = decltype(kind_c)::value;
        int abuf_sel = 0;
        for (int task = t_lo + r; task < t_hi; task += R) {
            int pos0, np;
            task_range(task, pos0, np);
            const uint8_t *abase[FIN_MT];
            uint32_t alds[FIN_MT];
            int row0_t, w0_t, nw_t;
            region(task, row0_t, w0_t, nw_t);
            const uint8_t *abuf_t = reinterpret_cast<const uint8_t *>(abuf + abuf_sel * a_words);
            // Local tiles: wv, and wv + 8 when the task has it.  The task's tiles are
            // spread over the four SIMDs as waves (s, s + 4) for SIMD s.  With m = ntl - 8
            // second slots in use (0 < m < 8), SIMD s carries 2 + [s < m] + [s + 4 < m]
            // tiles.  When m is 1 or 5 the SIMD holding the last tile carries a whole
            // tile more than the others, so its two 16-feature halves go to two SIMDs:
            // the owner wave computes features 0-15 of it and the next wave, whose
            // second slot is empty, features 16-31.  When m is 2 or 6 two SIMDs carry a
            // tile more than the other two: the last two tiles are split the same way,
            // their second halves going to the two waves after them (SIMDs then carry
            // 5 or 7 halves each).  A second slot past the task is skipped.
            const int ntl = (np + 15) / 16;
            int tile1 = wv + FIN_CW;
            int mode1 = tile1 < ntl ? 0 : 3;  // 0 both halves, 1 first half, 2 second half, 3 none
            const int m2 = ntl - FIN_CW;
            if (ntl > FIN_CW && (ntl & 3) == 1) {
                if (wv == m2 - 1) {
                    mode1 = 1;
                } else if (wv == m2) {
                    tile1 = ntl - 1;
                    mode1 = 2;
                }
            } else if (ntl > FIN_CW && (ntl & 3) == 2) {
                if (wv == m2 - 2 || wv == m2 - 1) {
                    mode1 = 1;
                } else if (wv == m2 || wv == m2 + 1) {
                    tile1 = ntl - 2 + (wv - m2);
                    mode1 = 2;
                }
            }
            if (!BLDS) {  // weight fragments from L2: one code path, the old assignment
                tile1 = wv + FIN_CW;
                mode1 = 0;
            }
            const int tl[FIN_MT] = {wv, tile1};
#pragma unroll
            for (int i = 0; i < FIN_MT; ++i) {
                const int gp = min(pos0 + tl[i] * 16 + c, pos0 + np - 1);
                const int b = gp / g.HoWo, pos = gp - b * g.HoWo;
                const int y = pos / g.Wo, xx = (pos - y * g.Wo) * g.S;  // the window's padded column
                const int row = b * g.Hp + y * g.S;
                abase[i] = tpad + (uint32_t)(((int64_t)row * g.Wp + xx) * g.CP);
                alds[i] = (uint32_t)((row - row0_t) * row_bytes + xx * 8);
            }
            const bool has_next = ALDS && task + R < t_hi;
            if (has_next) fill_region(task + R, abuf + (abuf_sel ^ 1) * a_words);  // read from the next task on
            auto blocks = [&](auto mode_c) {
            constexpr int M = decltype(mode_c)::value;
            constexpr int MT = M == 3 ? 1 : FIN_MT;  // slots with work
            constexpr int TB = FIN_TB;
            for (int tb0 = (g.T - 1) / TB * TB; tb0 >= 0; tb0 -= TB) {  // latest steps first
                const bool last_block = tb0 == 0;
                f4 acc[FIN_MT][2][TB];
#pragma unroll
                for (int i = 0; i < FIN_MT; ++i)
#pragma unroll
                    for (int n = 0; n < 2; ++n)
#pragma unroll
                        for (int t = 0; t < TB; ++t) acc[i][n][t] = f4{0.f, 0.f, 0.f, 0.f};
                // Software pipeline, unrolled by two K-steps with two register sets:
                // while K-step ks runs on the matrix cores, the spike words and weight
                // fragments of ks+1 are in flight and the tap offsets of ks+2 are read.
                auto koff_at = [&](int ks) { return koff_l[min(ks, g.ksteps - 1) * 4 + gq]; };
                auto load_a = [&](uint32_t (&an)[FIN_MT][2], int2 o) {
#pragma unroll
                    for (int i = 0; i < MT; ++i) {
                        if (ALDS) {  // CP >= 8: the lane's 8 taps are 8 contiguous bytes (o.y == o.x + 4)
                            const uint2 w2 = *reinterpret_cast<const uint2 *>(abuf_t + alds[i] + (uint32_t)o.x);
                            an[i][0] = w2.x;
                            an[i][1] = w2.y;
                        } else {
                            an[i][0] = *reinterpret_cast<const uint32_t *>(abase[i] + (uint32_t)o.x);
                            an[i][1] = *reinterpret_cast<const uint32_t *>(abase[i] + (uint32_t)o.y);
                        }
                    }
                };
                // B fragments of a K-step: bn[n * NT + q] = term q of feature tile n
                auto load_b = [&](uint4 (&bn)[2 * NT], int ks) {
                    // (one base address per K-step and constant offsets: per-fragment
                    // addresses would each hold a register through the loop)
                    const uint4 *fr = frag_l + ks * (2 * NT * 64) + lane;
#pragma unroll
                    for (int n = 0; n < 2; ++n)
#pragma unroll
                        for (int q = 0; q < NT; ++q)
                            bn[n * NT + q] = BLDS ? fr[(n * NT + q) * 64] : gf[((n * g.ksteps + ks) * NT + q) * 64];
                };
                // one K-step: spike operands from the words, then TB x 4 tiles x 2 features x NT terms
                auto kstep = [&](const uint32_t (&an)[FIN_MT][2], const uint4 (&bc)[2 * NT]) {
                    if constexpr (KIND == WK_F32) {
                        // fp32 form: instruction j takes tap 8*(lane/16) + j of every lane
                        // group, spike 1.0f / 0.0f against that tap's weight
#pragma unroll
                        for (int t = 0; t < TB; ++t) {
                            const int tt = tb0 + t;
                            float af[FIN_MT][8];
#pragma unroll
                            for (int i = 0; i < MT; ++i)
#pragma unroll
                                for (int j = 0; j < 8; ++j)
                                    af[i][j] = (int)((an[i][j >> 2] >> (8 * (j & 3))) & 255u) <= tt ? 1.0f : 0.0f;
#pragma unroll
                            for (int j = 0; j < 8; ++j)
#pragma unroll
                                for (int i = 0; i < MT; ++i)
#pragma unroll
                                    for (int n = 0; n < 2; ++n)
                                        if (fin_unit<M>(i, n)) {
                                            const uint4 b4 = bc[n * NT + (j >> 2)];
                                            const uint32_t bw = (j & 3) == 0 ? b4.x : (j & 3) == 1 ? b4.y
                                                              : (j & 3) == 2 ? b4.z : b4.w;
                                            acc[i][n][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                                af[i][j], __uint_as_float(bw), acc[i][n][t], 0, 0, 0);
                                        }
                        }
                        return;
                    }
                    uint32_t xn[FIN_MT][4];
#pragma unroll
                    for (int i = 0; i < MT; ++i) {
                        neg_times(an[i][0], xn[i][0], xn[i][1]);
                        neg_times(an[i][1], xn[i][2], xn[i][3]);
                    }
#pragma unroll
                    for (int t = 0; t < TB; ++t) {
                        const uint32_t ct = step_const(tb0 + t);
                        u4 a[FIN_MT];
#pragma unroll
                        for (int i = 0; i < MT; ++i) a[i] = spike_operand(xn[i], ct);
                        // one term of every unit after the other: dependent MFMAs are 8 apart
#pragma unroll
                        for (int q = 0; q < NT; ++q)
#pragma unroll
                            for (int i = 0; i < MT; ++i)
#pragma unroll
                                for (int n = 0; n < 2; ++n)
                                    if (fin_unit<M>(i, n))
                                        acc[i][n][t] = mfma<KIND>(a[i], bc[n * NT + q], acc[i][n][t]);
                    }
                };
                uint32_t a0[FIN_MT][2], a1[FIN_MT][2];
                uint4 b0[2 * NT], b1[2 * NT];
                int2 o2 = koff_at(0);
                load_a(a0, o2);
                load_b(b0, 0);
                o2 = koff_at(1);
                load_a(a1, o2);
                load_b(b1, min(1, g.ksteps - 1));
                o2 = koff_at(2);
                // pairs of K-steps without branches (the loads past the last K-step
                // re-read it), so the LDS waits count exactly; an odd last one after
                int ks = 0;
                for (; ks + 1 < g.ksteps; ks += 2) {
                    kstep(a0, b0);
                    const int2 o3 = koff_at(ks + 3);
                    load_a(a0, o2);
                    load_b(b0, min(ks + 2, g.ksteps - 1));
                    kstep(a1, b1);
                    o2 = koff_at(ks + 4);
                    load_a(a1, o3);
                    load_b(b1, min(ks + 3, g.ksteps - 1));
                }
                if (ks < g.ksteps) kstep(a0, b0);
                lds_barrier();  // staging free: the store waves are done with the previous block
                // Staging offset = the lane's part (feature c, positions 4*gq..) plus a
                // wave-uniform part; the lane part is made opaque here so that the
                // compiler forms the addresses at the writes instead of keeping one
                // register per (step, tile, half) alive through the K-step loop.
                const int sp = stage_stride(np);
                int lofs = c * sp + gq * 4;
                asm volatile("" : "+v"(lofs));
#pragma unroll
                for (int t = 0; t < TB; ++t) {
                    if (tb0 + t >= g.T) break;
                    float *st = stage + t * stage_t + lofs;
#pragma unroll
                    for (int i = 0; i < MT; ++i) {
                        const int pl = tl[i] * 16 + gq * 4;  // first of this lane's 4 positions
#pragma unroll
                        for (int n = 0; n < 2; ++n) {
                            if (!fin_unit<M>(i, n)) continue;
                            const int uo = n * 16 * sp + tl[i] * 16;  // wave-uniform part
                            const f4 v = acc[i][n][t] * inv_s;  // undo the weight scaling (a power of two)
                            if (G == 4) {
                                if (pl < np) *reinterpret_cast<f4 *>(st + uo) = v;
                            } else {
#pragma unroll
                                for (int q = 0; q < 4; ++q)
                                    if (pl + q < np) st[uo + q] = v[q];
                            }
                        }
                    }
                }
                if (has_next && last_block) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                lds_barrier();  // staging full
            }
            };
            if (!BLDS) {
                blocks(std::integral_constant<int, 0>{});
            } else if (G == 1) {  // at most 8 tiles per task: never split
                if (mode1 == 0) blocks(std::integral_constant<int, 0>{});
                else blocks(std::integral_constant<int, 3>{});
            } else {
                switch (mode1) {
                    case 0: blocks(std::integral_constant<int, 0>{}); break;
                    case 1: blocks(std::integral_constant<int, 1>{}); break;
                    case 2: blocks(std::integral_constant<int, 2>{}); break;
                    default: blocks(std::integral_constant<int, 3>{}); break;
                }
            }
            abuf_sel ^= 1;
        }
        };
        if constexpr (MODE == FIN_F32) {
            mfma_waves(std::integral_constant<int, WK_F32>{});
        } else {
            if (kind == WK_BF16)
                mfma_waves(std::integral_constant<int, WK_BF16>{});
            else
                mfma_waves(std::integral_constant<int, WK_F16>{});
        }
        if (MODE == FIN_POOL) __syncthreads();  // the store waves' last pooled map is complete in LDS
    } else {
        // ------------------------------------------------ store waves
        const int s = tid - FIN_CW * 64;
        // Pooling of the task whose first-spike times are in pool_l (after a
        // barrier): window (yo, xo) of feature fl is the min over its P x P
        // positions; outputs of consecutive threads are consecutive in xo.
        int pend_pos0 = -1, pend_np = 0;
        auto pool_pending = [&]() {
            if (MODE != FIN_POOL || pend_pos0 < 0) return;
            const int64_t pplane = (int64_t)po.Hpo * po.Wpo, wplane = (int64_t)g.Cout * pplane;
            // one segment per image the task covers (whole rows; a segment starts at
            // a row that is a multiple of P)
            for (int p = pend_pos0; p < pend_pos0 + pend_np;) {
                const int b = p / g.HoWo, q0 = p - b * g.HoWo;
                const int seg = min(pend_pos0 + pend_np, (b + 1) * g.HoWo) - p;
                const uint8_t *map = pool_l + (p - pend_pos0);  // + fl * np_max
                const int y0 = q0 / g.Wo, y1 = (q0 + seg) / g.Wo;  // the segment's output rows [y0, y1)
                const int yo0 = y0 / po.P, nyo = min(po.Hpo, y1 / po.P) - yo0;
                const int per_f = max(nyo, 0) * po.Wpo;
                if (po.vec) {
                    // per_f is a multiple of 4: groups of 4 consecutive pooled positions of one feature
                    const int gpf = per_f >> 2;
                    for (int i = s; i < nf * gpf; i += FIN_SW * 64) {
                        const int fl = i / gpf, q = (i - fl * gpf) * 4;
                        uint32_t t4 = 0;
#pragma unroll
                        for (int u = 0; u < 4; ++u) {
                            const int yo = yo0 + (q + u) / po.Wpo, xo = (q + u) - ((q + u) / po.Wpo) * po.Wpo;
                            const uint8_t *src = map + fl * np_max + (yo * po.P - y0) * g.Wo + xo * po.P;
                            int tmin = g.T;
                            for (int dy = 0; dy < po.P; ++dy)
                                for (int dx = 0; dx < po.P; ++dx) tmin = min(tmin, (int)src[dy * g.Wo + dx]);
                            t4 |= (uint32_t)tmin << (8 * u);
                        }
                        const int64_t o = ((int64_t)b * g.Cout + f0 + fl) * pplane + (int64_t)yo0 * po.Wpo + q;
                        *reinterpret_cast<uint32_t *>(po.tf + o) = t4;
                        if (po.wave) {
                            uint8_t *wv0 = po.wave + (int64_t)b * g.T * wplane + (int64_t)(f0 + fl) * pplane +
                                           (int64_t)yo0 * po.Wpo + q;
                            for (int tt = 0; tt < g.T; ++tt)
                                *reinterpret_cast<uint32_t *>(wv0 + tt * wplane) = spk::spikes4(t4, tt, g.T);
                        }
                    }
                } else {
                    for (int i = s; i < nf * per_f; i += FIN_SW * 64) {
                        const int fl = i / per_f, rr = i - fl * per_f;
                        const int yo = yo0 + rr / po.Wpo, xo = rr - (rr / po.Wpo) * po.Wpo;
                        const uint8_t *src = map + fl * np_max + (yo * po.P - y0) * g.Wo + xo * po.P;
                        int tmin = g.T;
                        for (int dy = 0; dy < po.P; ++dy)
                            for (int dx = 0; dx < po.P; ++dx) tmin = min(tmin, (int)src[dy * g.Wo + dx]);
                        const int64_t o = ((int64_t)b * g.Cout + f0 + fl) * pplane + (int64_t)yo * po.Wpo + xo;
                        po.tf[o] = (uint8_t)tmin;
                        if (po.wave) {
                            uint8_t *wv0 = po.wave + (int64_t)b * g.T * wplane + (int64_t)(f0 + fl) * pplane +
                                           (int64_t)yo * po.Wpo + xo;
                            for (int tt = 0; tt < g.T; ++tt) wv0[tt * wplane] = (uint8_t)(tt >= tmin);
                        }
                    }
                }
                p += seg;
            }
            pend_pos0 = -1;
        };
        for (int task = t_lo + r; task < t_hi; task += R) {
            int pos0, np;
            task_range(task, pos0, np);
            const int nel = nf * np;  // staged elements of the task
            constexpr int NSLOT = 32 * chunk_tiles_max(G) * 16 / (FIN_SW * 64) / G;  // staged groups per thread
            // per slot: the output element (feature f0+fl of flattened position pos0+pl) at step 0
            // relative to (image b0, feature f0), or -1; slots past the task read element 0 and are
            // never stored.  A group of G never straddles two images (G = 4 needs HoWo % 4 == 0).
            const int b0 = pos0 / g.HoWo;
            const int64_t base0 = (int64_t)b0 * g.T * tplane + (int64_t)f0 * g.HoWo;
            int off[NSLOT], src[NSLOT];
#pragma unroll
            for (int m = 0; m < NSLOT; ++m) {
                const int e = (s + FIN_SW * 64 * m) * G;  // first staged element of the slot
                const int fl = e / np, pl = e - fl * np;
                const int gp = pos0 + pl, b = gp / g.HoWo, pos = gp - b * g.HoWo;
                off[m] = e < nel ? (b - b0) * g.T * (int)tplane + fl * g.HoWo + pos : -1;
                src[m] = e < nel ? fl * stage_stride(np) + pl : 0;
            }
            // The steps arrive latest first, so the first spike is the last firing
            // seen: tf (4 bytes per slot) and vf are overwritten on every firing.
            uint32_t tf4[NSLOT];
            float vfirst[NSLOT][G];
#pragma unroll
            for (int m = 0; m < NSLOT; ++m) {
                tf4[m] = (uint32_t)g.T * 0x01010101u;
#pragma unroll
                for (int q = 0; q < G; ++q) vfirst[m][q] = 0.0f;
            }
            // The previous task's map is complete in LDS after this task's first
            // barrier.  It is pooled after the first block's firing, so that the
            // MFMA waves compute the second block meanwhile; with a single block,
            // between that block's two barriers (the map is rewritten right after
            // the block).  A no-op without pooling, and after its first call.
            const bool one_block = g.T <= FIN_TB;
            for (int tb0 = (g.T - 1) / FIN_TB * FIN_TB; tb0 >= 0; tb0 -= FIN_TB) {
                lds_barrier();  // staging free
                if (one_block) pool_pending();
                lds_barrier();  // staging full
                for (int t = min(FIN_TB, g.T - tb0) - 1; t >= 0; --t) {
                    const int tt = tb0 + t;
                    const float *st = stage + t * stage_t;
                    float *Pt = P ? P + base0 + (int64_t)tt * tplane : nullptr;
                    uint8_t *St = S ? S + base0 + (int64_t)tt * tplane : nullptr;
#pragma unroll
                    for (int m = 0; m < NSLOT; ++m) {
                        if (off[m] < 0) continue;
                        const uint32_t o = (uint32_t)off[m];
                        float v[G];
                        if (G == 4) {
                            const f4 x4 = *reinterpret_cast<const f4 *>(st + src[m]);
#pragma unroll
                            for (int q = 0; q < G; ++q) v[q] = x4[q];
                        } else {
                            v[0] = st[src[m]];
                        }
                        uint32_t bm = 0;  // 0xFF in the bytes that fire
#pragma unroll
                        for (int q = 0; q < G; ++q) {
                            const bool fire = v[q] >= g.thr;
                            vfirst[m][q] = fire ? v[q] : vfirst[m][q];
                            bm |= fire ? (0xFFu << (8 * q)) : 0u;
                        }
                        const uint32_t sp = bm & 0x01010101u;
                        tf4[m] = (tf4[m] & ~bm) | ((uint32_t)tt * 0x01010101u & bm);
                        if (G == 4) {
                            if (Pt) *reinterpret_cast<f4 *>(Pt + o) = f4{v[0], v[1], v[2], v[3]};
                            if (St) *reinterpret_cast<uint32_t *>(St + o) = sp;
                        } else {
                            if (Pt) Pt[o] = v[0];
                            if (St) St[o] = (uint8_t)sp;
                        }
                    }
                }
                if (!one_block) pool_pending();
            }
            // first-spike time and the potential there
#pragma unroll
            for (int m = 0; m < NSLOT; ++m) {
                if (off[m] < 0) continue;
                const int e = (s + FIN_SW * 64 * m) * G;
                const int fl = e / np, pl = e - fl * np;
                const int gp = pos0 + pl, b = gp / g.HoWo, pos = gp - b * g.HoWo;
                const int64_t o = ((int64_t)b * g.Cout + f0 + fl) * g.HoWo + pos;
                uint8_t *TFt = TF;
                float *VFt = VF;
                if (G == 4) {
                    *reinterpret_cast<uint32_t *>(TFt + o) = tf4[m];
                    *reinterpret_cast<f4 *>(VFt + o) = f4{vfirst[m][0], vfirst[m][1], vfirst[m][2], vfirst[m][3]};
                } else {
                    TFt[o] = (uint8_t)tf4[m];
                    VFt[o] = vfirst[m][0];
                }
                if (MODE == FIN_POOL) {  // this task's map for pooling (read after the next barrier)
                    if (G == 4)
                        *reinterpret_cast<uint32_t *>(pool_l + fl * np_max + pl) = tf4[m];
                    else
                        pool_l[fl * np_max + pl] = (uint8_t)tf4[m];
                }
            }
            if (MODE == FIN_POOL) {
                pend_pos0 = pos0;
                pend_np = np;
            }
        }
        if (MODE == FIN_POOL) {
            __syncthreads();  // matches the MFMA waves' last barrier
            pool_pending();
        }
    }
}

// ------------------------------------------------------------------ 3b. infinite threshold (Eq.5)
// Only the last step is computed: P[T-1] = sum_k W[f,k] [tp_k <= T-1], spike
// where P[T-1] > 0.  Every earlier step holds zero potential and no spike;
// those planes are contiguous per image and written by k_zero_planes.
// Persistent workgroups of 8 waves; a task is (group of 4 16-feature tiles,
// block of 16 position tiles), tasks ordered feature-group major and split
// into 8 contiguous XCD slices, so an XCD's L2 holds the fragments of about
// one feature group.  The fragments stream through two LDS buffers of KC
// K-steps, filled with direct global-to-LDS loads one chunk ahead; the spike
// words of a chunk are fetched before the next chunk's fill is issued, so
// the MFMA loop never waits behind it.
// Position-major form (small maps whose receptive fields are mostly padding,
// e.g. 4x4 maps under a 5x5 kernel): a 16-row tile is 16 images at one output
// position, a task is (feature group, position, block of 256 images), and
// the K loop runs only over the K-steps that touch the image at that
// position (9, 12 or 16 of 25 taps on a 4x4 map), listed per task in LDS.
constexpr int INF_WAVES = 8;
constexpr int INF_MW = 2;   // position tiles per wave
constexpr int INF_NW = 4;   // 16-feature tiles per workgroup
constexpr int INF_KC = 8;     // K-steps per LDS chunk
constexpr int INF_CHUNK_U4 = INF_KC * INF_NW * NT * 64;  // uint4 per chunk buffer
constexpr int INF_KPART = INF_KC;  // a K part is a multiple of this many K-steps (whole chunks)
constexpr int INF_ZW = 4;   // zero waves (waves 8-11)
constexpr int64_t INF_PART_MAX = 1 << 21;  // floats of split partial sums at most
constexpr int INF_KLMAX = 512;  // K-steps at most (16384 / 32)
constexpr int INF_PM_IMG = 16 * INF_WAVES * INF_MW;  // images per position-major task

// Does K-step ks touch the image (not only padding) for output position (y, x)?
__host__ __device__ inline bool kstep_valid(const ConvGeom &g, int y, int x, int ks) {
    const int KK = g.K * g.K;
    int c0, c1;
    if (g.CP % 32 == 0) {
        c0 = c1 = ks / (g.CP / 32);
    } else {
        c0 = ks * 32 / g.CP;
        c1 = (ks * 32 + 31) / g.CP;
        c1 = c1 < KK - 1 ? c1 : KK - 1;
    }
    for (int cell = c0; cell <= c1 && cell < KK; ++cell) {
        const int iy = y * g.S + cell / g.K - g.pad, ix = x * g.S + cell % g.K - g.pad;
        if (iy >= 0 && iy < g.H && ix >= 0 && ix < g.W) return true;
    }
    return false;
}

// K-steps of position pos that touch the image, counted by one wave
__device__ __forceinline__ int count_valid_ksteps(const ConvGeom &g, int pos, int lane) {
    const int y = pos / g.Wo, x = pos - y * g.Wo;
    int n = 0;
    for (int k0 = 0; k0 < g.ksteps; k0 += 64) n += __popcll(__ballot(k0 + lane < g.ksteps && kstep_valid(g, y, x, k0 + lane)));
    return n;
}

// With VEC, INF_ZW more waves write the zero planes of steps 0..T-2 (potentials
// and spikes of images blockIdx.x, blockIdx.x + gridDim.x, ...) while the MFMA
// waves compute: they pass the same barriers, one slice of their stores between
// two barriers.
template <bool VEC, bool PM>
__global__ __launch_bounds__((INF_WAVES + INF_ZW) * 64, 1) void k_conv_fire_inf(
    const uint8_t *__restrict__ tpad, const uint4 *__restrict__ frag, const int2 *__restrict__ koff2, ConvGeom g,
    int n_mb, int n_ng, int ksplit, int kpp, int pm_nib, float *__restrict__ part, const float *__restrict__ inv_scale,
    const int *__restrict__ wbf16, float *__restrict__ P, uint8_t *__restrict__ S, uint8_t *__restrict__ TF,
    float *__restrict__ VF) {
    extern __shared__ uint4 lds[];
    int2 *koff_l = reinterpret_cast<int2 *>(lds);
    uint4 *cbuf = lds + (g.ksteps * 4 * 8 + 15) / 16;  // 2 chunk buffers [ksl][n][term][64]
    uint16_t *klist = reinterpret_cast<uint16_t *>(cbuf + 2 * INF_CHUNK_U4);  // [2][INF_KLMAX] (position-major)
    int2 *koffp = reinterpret_cast<int2 *>(klist + 2 * INF_KLMAX);            // [2][ksteps][4] (position-major)
    // LDS byte address of the chunk buffers (for the position-major transfers)
    const uint32_t cbuf_lds = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)cbuf;
    constexpr bool pm = PM;  // position-major tasks (pm_nib image blocks)
    constexpr int KCH = PM ? INF_KC / 2 : INF_KC;  // K-steps per chunk (position-major: fewer, no spills)
    constexpr int GPW_PM = KCH * INF_NW * NT / INF_WAVES;  // position-major fill loads per wave and chunk
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int gq = lane >> 4, c = lane & 15;
    for (int i = tid; i < g.ksteps * 4; i += (INF_WAVES + INF_ZW) * 64) koff_l[i] = koff2[i];
    const float inv_s = *inv_scale;
    const bool use_bf = *wbf16 == WK_BF16;
    const uint32_t ct = step_const(g.T - 1);
    const int x = blockIdx.x % 8, j = blockIdx.x / 8, per_xcd = (int)gridDim.x / 8;
    const int ntask = n_mb * n_ng * ksplit, per_x = (ntask + 7) / 8;
    const int t_lo = x * per_x, t_hi = min(ntask, t_lo + per_x);
    const int64_t tstride = (int64_t)g.Cout * g.HoWo;
    // With ksplit > 1 a task is (feature group, position block, part of the K
    // steps: kpp of them, a multiple of INF_KPART): its raw sums go to
    // part[kp][B][Cout][HoWo], added up in part order by k_inf_reduce.
    // position-major: task -> (feature group, block of images, position); its
    // K-steps are the valid ones of that position (nvalid of them)
    auto pm_pos = [&](int task) { return (task % n_mb) % g.HoWo; };
    auto chunk_range = [&](int task, int kc, int &c_lo, int &c_hi, int nvalid) {
        if (pm) {
            c_lo = 0;
            c_hi = (nvalid + kc - 1) / kc;
            return;
        }
        const int k_lo = (task % ksplit) * kpp, k_hi = min(g.ksteps, k_lo + kpp);
        c_lo = k_lo / kc;
        c_hi = k_hi > k_lo ? (k_hi + kc - 1) / kc : c_lo;
    };

    if (wv >= INF_WAVES) {
        // zero waves: 16-byte units of potentials (4 per unit) and 4-byte units of spikes
        // (4 per unit); images b = blockIdx.x + i * gridDim.x; one slice per barrier interval
        const int zt = tid - INF_WAVES * 64;
        const int64_t zp = VEC && P && g.T > 1 ? (g.T - 1) * tstride / 4 : 0;  // units per image
        const int64_t zs = VEC && S && g.T > 1 ? (g.T - 1) * tstride / 4 : 0;
        const int64_t nimg = g.B > (int)blockIdx.x ? (g.B - 1 - (int)blockIdx.x) / gridDim.x + 1 : 0;
        const int64_t total = nimg * (zp + zs);
        int nint = 1;  // barrier intervals (the last one after the loop)
        for (int task = t_lo + j; task < t_hi; task += per_xcd) {
            int c_lo, c_hi;
            chunk_range(task, KCH, c_lo, c_hi, pm ? count_valid_ksteps(g, pm_pos(task), lane) : 0);
            nint += 1 + max(0, c_hi - c_lo);
        }
        const int64_t per = (total + nint - 1) / nint;
        // lane zt writes units zt, zt + 256, ... in order, as (image im, unit r of it)
        const int64_t zpz = zp + zs;
        int64_t u0 = 0, cu = zt, cim = zpz > 0 ? cu / zpz : 0, cr = cu - cim * zpz;
        auto slice = [&]() {
            if (!VEC) return;  // a separate fill kernel writes the zeros
            const int64_t u1 = min(total, u0 + per);
            for (; cu < u1; cu += INF_ZW * 64) {
                const int64_t b = blockIdx.x + cim * gridDim.x;
                if (cr < zp)
                    *reinterpret_cast<f4 *>(P + b * g.T * tstride + 4 * cr) = f4{0.f, 0.f, 0.f, 0.f};
                else
                    *reinterpret_cast<uint32_t *>(S + b * g.T * tstride + 4 * (cr - zp)) = 0u;
                for (cr += INF_ZW * 64; zpz > 0 && cr >= zpz; ++cim) cr -= zpz;
            }
            u0 = u1;
        };
        for (int task = t_lo + j; task < t_hi; task += per_xcd) {
            int c_lo, c_hi;
            chunk_range(task, KCH, c_lo, c_hi, pm ? count_valid_ksteps(g, pm_pos(task), lane) : 0);
            slice();
            __syncthreads();  // the MFMA waves' "buffers free"
            for (int ch = c_lo; ch < c_hi; ++ch) {
                slice();
                // the MFMA waves' chunk barrier; in the position-major form it does
                // not wait for this wave's stores
                if constexpr (PM)
                    lds_barrier();
                else
                    __syncthreads();
            }
        }
        slice();
        return;
    }

    auto mfma_waves = [&](auto bf_c) {
    constexpr int KIND = decltype(bf_c)::value ? WK_BF16 : WK_F16;
    constexpr int KC = KCH;
    constexpr int CHUNK_U4 = INF_CHUNK_U4;
    int tpar = 0;  // task parity: the K-step list buffer
    for (int task = t_lo + j; task < t_hi; task += per_xcd, tpar ^= 1) {
        const int tq = task / ksplit, kp = task % ksplit;
        const int ng = tq / n_mb, mb = tq % n_mb;
        const int ppos = pm ? pm_pos(task) : 0, pib = pm ? mb / g.HoWo : 0;
        int nks = g.ksteps;
        uint16_t *kl = klist + tpar * INF_KLMAX;
        if constexpr (pm) {  // the valid K-steps of the position, in order (wave 0 lists them)
            const int py = ppos / g.Wo, px = ppos - py * g.Wo;
            nks = 0;
            for (int k0 = 0; k0 < g.ksteps; k0 += 64) {
                const bool v = k0 + lane < g.ksteps && kstep_valid(g, py, px, k0 + lane);
                const uint64_t m = __ballot(v);
                if (wv == 0 && v) {
                    const int at = nks + __popcll(m & ((1ull << lane) - 1ull));
                    kl[at] = (uint16_t)(k0 + lane);
#pragma unroll
                    for (int q = 0; q < 4; ++q) koffp[(tpar * g.ksteps + at) * 4 + q] = koff_l[(k0 + lane) * 4 + q];
                }
                nks += __popcll(m);
            }
        }
        auto kidx = [&](int i) {
            if constexpr (pm) return (int)kl[i];
            else return i;
        };
        int c_lo, c_hi;
        chunk_range(task, KC, c_lo, c_hi, nks);
        const uint4 *fg = frag + (int64_t)ng * INF_NW * g.ksteps * NT * 64;
        // chunk ch -> buffer: wave w issues the 64-lane groups w, w+8, ... (16 bytes per lane)
        auto fill = [&](int ch) {
            if constexpr (pm) {
                // three chunk buffers; every wave issues the same number of loads per
                // chunk (groups past the chunk's last K-step load a valid one that is
                // never read), so the waits can count them
                constexpr int GPW = KC * INF_NW * NT / INF_WAVES;
                const uint32_t dst = cbuf_lds + (uint32_t)((ch % 3) * (KC * INF_NW * NT * 64)) * 16u;
                const int k0 = ch * KC;
#pragma unroll
                for (int u = 0; u < GPW; ++u) {
                    const int grp = wv + u * INF_WAVES;
                    const int q = grp % NT, n = (grp / NT) % INF_NW, ksl = grp / (NT * INF_NW);
                    const uint4 *src = fg + (((int64_t)n * g.ksteps + kidx(min(k0 + ksl, nks - 1))) * NT + q) * 64 + lane;
                    lds_dma16(src, __builtin_amdgcn_readfirstlane(dst + (uint32_t)grp * 64u * 16u));
                }
                return;
            }
            uint4 *dst = cbuf + (ch & 1) * CHUNK_U4;
            const int k0 = ch * KC, nk = min(KC, nks - k0);
            for (int grp = wv; grp < nk * INF_NW * NT; grp += INF_WAVES) {
                const int q = grp % NT, n = (grp / NT) % INF_NW, ksl = grp / (NT * INF_NW);
                const uint4 *src = fg + (((int64_t)n * g.ksteps + kidx(k0 + ksl)) * NT + q) * 64 + lane;
                __builtin_amdgcn_global_load_lds(src, dst + grp * 64, 16, 0, 0);
            }
        };
        const uint8_t *abase[INF_MW];
        int64_t img[INF_MW];
        int mpos0[INF_MW];
#pragma unroll
        for (int i = 0; i < INF_MW; ++i) {
            if constexpr (pm) {  // rows: images pib*INF_PM_IMG + (wv*MW + i)*16 + row, all at position ppos
                const int64_t b0 = (int64_t)pib * INF_PM_IMG + (wv * INF_MW + i) * 16;
                const int64_t b = min<int64_t>(b0 + c, g.B - 1);  // rows past the batch are computed, not stored
                const int y = ppos / g.Wo, xx = ppos % g.Wo;
                abase[i] = tpad + (uint32_t)(((b * g.Hp + y * g.S) * g.Wp + xx * g.S) * g.CP);
                img[i] = b0 < g.B ? b0 : -1;
                mpos0[i] = ppos;
                continue;
            }
            const int64_t gm = ((int64_t)mb * INF_WAVES + wv) * INF_MW + i;
            const bool v = gm < g.total_mtiles;
            const int64_t b = v ? gm / g.mt_per_img : 0;
            const int mt = v ? (int)(gm % g.mt_per_img) : 0;
            const int pos = min(mt * 16 + c, g.HoWo - 1);  // rows past the image are computed, not stored
            const int y = pos / g.Wo, xx = pos % g.Wo;
            abase[i] = tpad + (uint32_t)(((b * g.Hp + y * g.S) * g.Wp + xx * g.S) * g.CP);
            img[i] = v ? b : -1;
            mpos0[i] = mt * 16 + gq * 4;
        }
        f4 acc[INF_MW][INF_NW];
#pragma unroll
        for (int i = 0; i < INF_MW; ++i)
#pragma unroll
            for (int n = 0; n < INF_NW; ++n) acc[i][n] = f4{0.f, 0.f, 0.f, 0.f};
        // the spike words of a chunk are loaded with its fill, one chunk ahead; two
        // register sets, the loop unrolled by two chunks so that both are static
        uint32_t aw0[KC][INF_MW][2], aw1[KC][INF_MW][2];
        // With CP a multiple of 64 a cell has an even number of K-steps and K-steps
        // 2m, 2m+1 of it are 16 consecutive, aligned bytes of a lane's run; with
        // CP >= 8 a K-step's two words are adjacent; with CP == 4 separate cells.
        const int wide = g.CP % 64 == 0 ? 2 : (g.CP >= 8 ? 1 : 0);
        auto load_aw = [&](int ch, uint32_t (&dst)[KC][INF_MW][2]) {
            if (wide == 2) {
#pragma unroll
                for (int kl = 0; kl < KC; kl += 2) {
                    const int2 o = pm ? koffp[(tpar * g.ksteps + max(0, min(ch * KC + kl, nks - 2))) * 4 + gq]
                                      : koff_l[kidx(max(0, min(ch * KC + kl, nks - 2))) * 4 + gq];
#pragma unroll
                    for (int i = 0; i < INF_MW; ++i) {
                        const uint4 v = *reinterpret_cast<const uint4 *>(abase[i] + (uint32_t)o.x);
                        dst[kl][i][0] = v.x;
                        dst[kl][i][1] = v.y;
                        dst[kl + 1][i][0] = v.z;
                        dst[kl + 1][i][1] = v.w;
                    }
                }
            } else {
#pragma unroll
                for (int kl = 0; kl < KC; ++kl) {
                    const int2 o = pm ? koffp[(tpar * g.ksteps + max(0, min(ch * KC + kl, nks - 1))) * 4 + gq]
                                      : koff_l[kidx(max(0, min(ch * KC + kl, nks - 1))) * 4 + gq];
#pragma unroll
                    for (int i = 0; i < INF_MW; ++i) {
                        if (wide == 1) {
                            const uint2 v = *reinterpret_cast<const uint2 *>(abase[i] + (uint32_t)o.x);
                            dst[kl][i][0] = v.x;
                            dst[kl][i][1] = v.y;
                        } else {
                            dst[kl][i][0] = *reinterpret_cast<const uint32_t *>(abase[i] + (uint32_t)o.x);
                            dst[kl][i][1] = *reinterpret_cast<const uint32_t *>(abase[i] + (uint32_t)o.y);
                        }
                    }
                }
            }
        };
        auto mma = [&](const uint4 *fr, int nk, const uint32_t (&awc)[KC][INF_MW][2]) {
#pragma unroll
            for (int kl = 0; kl < KC; ++kl) {
                if (kl >= nk) break;  // uniform
                uint4 bt[NT][INF_NW];
#pragma unroll
                for (int n = 0; n < INF_NW; ++n)
#pragma unroll
                    for (int q = 0; q < NT; ++q) bt[q][n] = fr[((kl * INF_NW + n) * NT + q) * 64];
                u4 a[INF_MW];
#pragma unroll
                for (int i = 0; i < INF_MW; ++i) {
                    uint32_t xn[4];
                    neg_times(awc[kl][i][0], xn[0], xn[1]);
                    neg_times(awc[kl][i][1], xn[2], xn[3]);
                    a[i] = spike_operand(xn, ct);
                }
#pragma unroll
                for (int q = 0; q < NT; ++q)
#pragma unroll
                    for (int i = 0; i < INF_MW; ++i)
#pragma unroll
                        for (int n = 0; n < INF_NW; ++n) acc[i][n] = mfma<KIND>(a[i], bt[q][n], acc[i][n]);
            }
        };
        if constexpr (pm) {
            // two chunks ahead: chunk ch's words and fill are waited for while chunk
            // ch+1's loads (a fixed number per wave) stay in flight
            uint32_t aw2[KC][INF_MW][2];
            const int ahead = GPW_PM + (wide == 2 ? KC / 2 : wide == 1 ? KC : 2 * KC) * INF_MW;
            auto chunk3 = [&](int ch, const uint32_t (&awc)[KC][INF_MW][2], uint32_t (&awn)[KC][INF_MW][2]) {
                if (ch + 1 < c_hi)
                    wait_vmcnt(ahead);
                else
                    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                lds_barrier();  // every wave's part of chunk ch is in LDS; chunk ch-1's buffer is free
                if (ch + 2 < c_hi) {
                    load_aw(ch + 2, awn);
                    fill(ch + 2);
                }
                mma(cbuf + (ch % 3) * (KC * INF_NW * NT * 64) + lane, min(KC, nks - ch * KC), awc);
            };
            __syncthreads();  // the buffers are free (previous task done), the lists are visible
            if (c_hi > 0) {
                load_aw(0, aw0);
                fill(0);
            }
            if (c_hi > 1) {
                load_aw(1, aw1);
                fill(1);
            }
            for (int ch = 0; ch < c_hi; ch += 3) {
                chunk3(ch, aw0, aw2);
                if (ch + 1 < c_hi) chunk3(ch + 1, aw1, aw0);
                if (ch + 2 < c_hi) chunk3(ch + 2, aw2, aw1);
            }
        } else {
            auto chunk = [&](int ch, const uint32_t (&awc)[KC][INF_MW][2], uint32_t (&awn)[KC][INF_MW][2]) {
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's words and fill of chunk ch landed
                __syncthreads();  // every wave's part of chunk ch is in LDS; chunk ch-1's buffer is free
                if (ch + 1 < c_hi) {
                    load_aw(ch + 1, awn);
                    fill(ch + 1);
                }
                mma(cbuf + (ch & 1) * CHUNK_U4 + lane, min(KC, nks - ch * KC), awc);
            };
            __syncthreads();  // the buffers are free (previous task done), koff is visible
            if (c_lo < c_hi) {
                load_aw(c_lo, aw0);
                fill(c_lo);
            }
            for (int ch = c_lo; ch < c_hi; ch += 2) {
                chunk(ch, aw0, aw1);
                if (ch + 1 < c_hi) chunk(ch + 1, aw1, aw0);
            }
        }
        // the last step's potentials and spikes, the first-spike time and potential
        if constexpr (pm) {
            // accumulator rows 4*gq + q are images img + 4*gq + q at position ppos: the
            // raw sums go to part[ppos][b][f] (16 features contiguous), and
            // k_inf_pm_finish writes them out per image
#pragma unroll
            for (int i = 0; i < INF_MW; ++i)
#pragma unroll
                for (int n = 0; n < INF_NW; ++n) {
                    const int f = (ng * INF_NW + n) * 16 + c;
                    if (img[i] < 0 || f >= g.Cout) continue;
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int64_t b = img[i] + gq * 4 + q;
                        if (b < g.B) part[((int64_t)ppos * g.B + b) * g.Cout + f] = acc[i][n][q];
                    }
                }
            continue;
        }
#pragma unroll
        for (int i = 0; i < INF_MW; ++i)
#pragma unroll
            for (int n = 0; n < INF_NW; ++n) {
                const int f = (ng * INF_NW + n) * 16 + c;
                if (img[i] < 0 || f >= g.Cout || mpos0[i] >= g.HoWo) continue;
                const int lim = g.HoWo - mpos0[i];
                if (ksplit > 1) {  // this part's raw sums
                    const int64_t op = (((int64_t)kp * g.B + img[i]) * g.Cout + f) * g.HoWo + mpos0[i];
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        if (q < lim) part[op + q] = acc[i][n][q];
                    continue;
                }
                const f4 v = acc[i][n] * inv_s;
                const int64_t o = (img[i] * g.T + g.T - 1) * tstride + (int64_t)f * g.HoWo + mpos0[i];
                const int64_t of = (img[i] * (int64_t)g.Cout + f) * g.HoWo + mpos0[i];
                uint32_t sp = 0, tv = 0;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    sp |= (uint32_t)(v[q] > 0.0f) << (8 * q);
                    tv |= (uint32_t)(v[q] > 0.0f ? g.T - 1 : g.T) << (8 * q);
                }
                if (VEC) {  // HoWo % 4 == 0: the 4 positions are in the image and aligned
                    if (P) *reinterpret_cast<f4 *>(P + o) = v;
                    if (S) *reinterpret_cast<uint32_t *>(S + o) = sp;
                    *reinterpret_cast<uint32_t *>(TF + of) = tv;
                    *reinterpret_cast<f4 *>(VF + of) = v;
                } else {
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        if (q < lim) {
                            if (P) P[o + q] = v[q];
                            if (S) S[o + q] = (uint8_t)(sp >> (8 * q));
                            TF[of + q] = (uint8_t)(tv >> (8 * q));
                            VF[of + q] = v[q];
                        }
                }
            }
    }
    };
    if (use_bf)
        mfma_waves(std::integral_constant<bool, true>{});
    else
        mfma_waves(std::integral_constant<bool, false>{});
}

// Zero potentials (f32) and spikes (u8) of steps 0..T-2 of every image: per
// image one contiguous run of (T-1)*Cout*Ho*Wo elements.  Grid (chunk, image).
__global__ __launch_bounds__(256) void k_zero_planes(ConvGeom g, float *__restrict__ P, uint8_t *__restrict__ S) {
    const int64_t plane = (int64_t)g.Cout * g.HoWo;
    const int64_t n = (int64_t)(g.T - 1) * plane;
    for (int64_t b = blockIdx.y; b < g.B; b += gridDim.y) {
        if (P) {
            float *p = P + b * g.T * plane;
            const int64_t head = min<int64_t>(n, (int64_t)((16 - ((uintptr_t)p & 15)) & 15) / 4);
            const int64_t body = (n - head) & ~(int64_t)3;
            for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < head; i += (int64_t)gridDim.x * 256) p[i] = 0.0f;
            for (int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4; i < body; i += (int64_t)gridDim.x * 1024)
                *reinterpret_cast<f4 *>(p + head + i) = f4{0.f, 0.f, 0.f, 0.f};
            for (int64_t i = head + body + (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
                p[i] = 0.0f;
        }
        if (S) {
            uint8_t *q = S + b * g.T * plane;
            const int64_t head = min<int64_t>(n, (int64_t)((16 - ((uintptr_t)q & 15)) & 15));
            const int64_t body = (n - head) & ~(int64_t)15;
            for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < head; i += (int64_t)gridDim.x * 256) q[i] = 0;
            for (int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 16; i < body; i += (int64_t)gridDim.x * 4096)
                *reinterpret_cast<uint4 *>(q + head + i) = uint4{0u, 0u, 0u, 0u};
            for (int64_t i = head + body + (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
                q[i] = 0;
        }
    }
}



// The Eq.5 outputs from split sums: P[T-1] = (sum of the parts, in part order)
// / scale; one thread per (image, feature, position).
__global__ __launch_bounds__(256) void k_inf_reduce(const float *__restrict__ part, int ksplit, ConvGeom g,
                                                    const float *__restrict__ inv_scale, float *__restrict__ P,
                                                    uint8_t *__restrict__ S, uint8_t *__restrict__ TF,
                                                    float *__restrict__ VF) {
    const int64_t plane = (int64_t)g.Cout * g.HoWo, n = g.B * plane;
    const int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (o >= n) return;
    float sum = part[o];
    for (int k = 1; k < ksplit; ++k) sum += part[k * n + o];
    const float v = sum * *inv_scale;
    const int64_t b = o / plane, r = o - b * plane;
    const int64_t ot = (b * g.T + g.T - 1) * plane + r;
    if (P) P[ot] = v;
    if (S) S[ot] = (uint8_t)(v > 0.0f);
    TF[o] = (uint8_t)(v > 0.0f ? g.T - 1 : g.T);
    VF[o] = v;
}

// Position-major Eq.5 outputs: one workgroup per image reads the raw sums
// part[pos][b][f] (contiguous in f), transposes them through LDS to the
// image's [f][pos] order and writes P[T-1] = sum / scale, its spikes, the
// first-spike time (T-1 where it fires, else T) and the potential there.
constexpr int INF_PM_OUT = 16384;  // Cout * HoWo at most (the LDS transpose)
__global__ __launch_bounds__(256) void k_inf_pm_finish(const float *__restrict__ part, ConvGeom g,
                                                       const float *__restrict__ inv_scale, float *__restrict__ P,
                                                       uint8_t *__restrict__ S, uint8_t *__restrict__ TF,
                                                       float *__restrict__ VF, int vec4) {
    extern __shared__ float buf[];  // Cout rows of HoWo + 1 (odd stride: the transposing stores hit distinct banks)
    const int64_t b = blockIdx.x, plane = (int64_t)g.Cout * g.HoWo;
    const float inv_s = *inv_scale;
    // sixteen loads in flight per thread before its LDS stores (a load followed
    // at once by its store waits for memory each time); element i = pos * Cout + f
    // with (pos, f) carried, not divided out
    constexpr int U = 16;
    int pos = (int)threadIdx.x / g.Cout, f = (int)threadIdx.x - pos * g.Cout;
    const int dpos = 256 / g.Cout, df = 256 - dpos * g.Cout;
    auto step = [&](int &ps, int &ff) {
        ps += dpos;
        ff += df;
        if (ff >= g.Cout) {
            ff -= g.Cout;
            ++ps;
        }
    };
    for (int i0 = threadIdx.x; i0 < plane; i0 += U * 256) {
        float v[U];
        int ps = pos, ff = f;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            v[u] = i0 + u * 256 < plane ? part[((int64_t)ps * g.B + b) * g.Cout + ff] : 0.0f;
            step(ps, ff);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (i0 + u * 256 < plane) buf[f * (g.HoWo + 1) + pos] = v[u];
            step(pos, f);
        }
    }
    __syncthreads();
    const int64_t o0 = (b * g.T + g.T - 1) * plane, of0 = b * plane;
    if (vec4) {
        // four positions of one feature per thread and pass: 16-byte potential and
        // 4-byte spike / first-spike stores (HoWo a multiple of 4 and the buffers
        // aligned: checked by the host)
        const int q4 = g.HoWo / 4;
        for (int i4 = threadIdx.x; i4 < plane / 4; i4 += 256) {
            const int fo = i4 / q4, i = 4 * i4;
            float4 v;
            v.x = buf[i + fo] * inv_s;
            v.y = buf[i + fo + 1] * inv_s;
            v.z = buf[i + fo + 2] * inv_s;
            v.w = buf[i + fo + 3] * inv_s;
            const uint32_t fire = (v.x > 0.0f) | (v.y > 0.0f) << 8 | (v.z > 0.0f) << 16 | (uint32_t)(v.w > 0.0f) << 24;
            if (P) *reinterpret_cast<float4 *>(P + o0 + i) = v;
            if (S) *reinterpret_cast<uint32_t *>(S + o0 + i) = fire;
            *reinterpret_cast<uint32_t *>(TF + of0 + i) = (uint32_t)g.T * 0x01010101u - fire;  // T - 1 where fired
            *reinterpret_cast<float4 *>(VF + of0 + i) = v;
        }
        return;
    }
    // element i = f * HoWo + q: buf[i + f]
    const int dq = 256 / g.HoWo, dr = 256 - dq * g.HoWo;
    int fo = (int)threadIdx.x / g.HoWo, qo = (int)threadIdx.x - fo * g.HoWo;
    for (int i = threadIdx.x; i < plane; i += 256) {
        const float v = buf[i + fo] * inv_s;
        fo += dq;
        qo += dr;
        if (qo >= g.HoWo) {
            qo -= g.HoWo;
            ++fo;
        }
        const bool fire = v > 0.0f;
        if (P) P[o0 + i] = v;
        if (S) S[o0 + i] = (uint8_t)fire;
        TF[of0 + i] = (uint8_t)(fire ? g.T - 1 : g.T);
        VF[of0 + i] = v;
    }
}

int inf_pm_nib(const ConvGeom &g, int ksplit);

struct ConvPlan {
    ConvGeom g;
    size_t tpad_bytes, frag_count, koff_count;
    int ksplit;         // K parts of the Eq.5 kernel (1: not split)
    int kpp;            // K-steps per part (a multiple of INF_KPART when split)
    size_t part_count;  // floats of its partial sums
};

int make_plan(int B, int T, int Cin, int H, int W, int Cout, int K, int stride, int pad, ConvPlan &pl) {
    SPK_REQUIRE(B >= 0 && T >= 1 && Cin >= 1 && H >= 1 && W >= 1 && Cout >= 1 && K >= 1 && pad >= 0 && stride >= 1,
                SPK_E_SHAPE, "spk_conv_fire: bad sizes B=%d T=%d Cin=%d H=%d W=%d Cout=%d K=%d stride=%d pad=%d",
                B, T, Cin, H, W, Cout, K, stride, pad);
    SPK_REQUIRE(stride <= 64, SPK_E_RANGE, "spk_conv_fire: stride=%d > 64", stride);
    SPK_REQUIRE(T <= 255, SPK_E_RANGE, "spk_conv_fire: T=%d > 255", T);
    SPK_REQUIRE(Cin <= 4096 && K <= 64 && pad <= 64 && H <= 65536 && W <= 65536, SPK_E_RANGE,
                "spk_conv_fire: Cin, K, pad or the image too large");
    ConvGeom &g = pl.g;
    g.B = B; g.T = T; g.Cin = Cin; g.H = H; g.W = W; g.Cout = Cout; g.K = K; g.pad = pad; g.S = stride;
    g.CP = Cin <= 4 ? 4 : (Cin + 7) / 8 * 8;
    g.Hp = H + 2 * pad;
    g.Wp = W + 2 * pad;
    SPK_REQUIRE(g.Hp >= K && g.Wp >= K, SPK_E_SHAPE, "spk_conv_fire: kernel %d larger than padded input %dx%d",
                K, g.Hp, g.Wp);
    g.Ho = (g.Hp - K) / stride + 1;  // Eq.2 with stride: floor((H + 2 pad - K) / stride) + 1
    g.Wo = (g.Wp - K) / stride + 1;
    SPK_REQUIRE((int64_t)K * K * g.CP <= 16384, SPK_E_RANGE,
                "spk_conv_fire: K*K*Cin (Cin rounded up to %d) = %lld > 16384", g.CP, (long long)K * K * g.CP);
    SPK_REQUIRE(Cout <= 4096, SPK_E_RANGE, "spk_conv_fire: Cout=%d > 4096", Cout);
    SPK_REQUIRE((int64_t)g.Ho * g.Wo <= (1LL << 26), SPK_E_RANGE, "spk_conv_fire: %lld output positions > 2^26",
                (long long)g.Ho * g.Wo);
    SPK_REQUIRE((int64_t)g.Wp * g.CP <= PAD_LDS, SPK_E_RANGE,
                "spk_conv_fire: padded input row of %lld bytes exceeds %d", (long long)g.Wp * g.CP, PAD_LDS);
    // the MFMA kernels address the padded first-spike map with 32-bit offsets
    SPK_REQUIRE((int64_t)B * g.Hp * g.Wp * g.CP < (1LL << 32), SPK_E_RANGE,
                "spk_conv_fire: padded input of %lld bytes exceeds 4 GiB", (long long)B * g.Hp * g.Wp * g.CP);
    SPK_REQUIRE((int64_t)B * ((g.Ho * (int64_t)g.Wo + 15) / 16) * 16 + 256 < (1LL << 31), SPK_E_RANGE,
                "spk_conv_fire: B * Ho * Wo too large");
    g.HoWo = g.Ho * g.Wo;
    g.ksteps = (K * K * g.CP + 31) / 32;
    g.ntiles = (int)spk::ceil_div(spk::ceil_div(Cout, 16), NTILE_ALIGN) * NTILE_ALIGN;
    g.mt_per_img = (g.HoWo + 15) / 16;
    g.total_mtiles = (int64_t)B * g.mt_per_img;
    pl.tpad_bytes = (size_t)B * g.Hp * g.Wp * g.CP;
    pl.frag_count = (size_t)g.ntiles * g.ksteps * NT * 64;
    pl.koff_count = (size_t)g.ksteps * 4;
    // Eq.5 mode on few tasks (a small batch): the K chunks are split into parts
    // run by separate workgroups, so that more than a handful of CUs work; the
    // partial sums take at most INF_PART_MAX floats.
    const int64_t n_mb = spk::ceil_div(g.total_mtiles, INF_WAVES * INF_MW);
    const int64_t n_ng = spk::ceil_div(spk::ceil_div(Cout, 16), INF_NW);
    const int64_t nch = spk::ceil_div(g.ksteps, INF_KPART), outs = (int64_t)B * Cout * g.HoWo;
    int64_t ks = n_mb * n_ng > 0 && n_mb * n_ng < 128 ? std::min<int64_t>(nch, spk::ceil_div(256, n_mb * n_ng)) : 1;
    if (outs > 0) ks = std::min<int64_t>(ks, INF_PART_MAX / outs);
    if (ks >= 2) ks = spk::ceil_div(nch, spk::ceil_div(nch, ks));  // no part without K-steps
    pl.ksplit = ks >= 2 ? (int)ks : 1;
    pl.kpp = pl.ksplit > 1 ? (int)spk::ceil_div(nch, pl.ksplit) * INF_KPART : g.ksteps;
    pl.part_count = pl.ksplit > 1 ? (size_t)(pl.ksplit * outs) : 0;
    if (inf_pm_nib(g, pl.ksplit)) pl.part_count = (size_t)outs;  // position-major sums of an Eq.5 call
    return SPK_OK;
}

size_t plan_workspace(const ConvPlan &pl) {
    spk::Carver c(nullptr);
    c.take<uint8_t>(pl.tpad_bytes);
    c.take<uint4>(pl.frag_count);
    c.take<int2>(pl.koff_count);
    c.take<float>(1);                // 1/scale
    c.take<int>(1);                  // weight term type
    c.take<unsigned>(WMAX_PARTS);    // weight-range partials: maxima
    c.take<unsigned>(WMAX_PARTS);    //                        non-zero minima
    c.take<float>(pl.part_count);    // Eq.5 split sums
    return spk::align_up(c.off, 256);
}

int max_lds_per_block() {
    int dev = 0, v = 65536;
    if (hipGetDevice(&dev) != hipSuccess) return 65536;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) return 65536;
    return v;
}

template <int G, bool BLDS, bool ALDS, int MODE>
void launch_fin(const uint8_t *tpad, const uint4 *frag, const int2 *koff2, const float *inv_scale, const int *wbf16,
                const float *wts, const unsigned *wmax, const unsigned *wmin, int n_wmax, const ConvGeom &g,
                int n_pairs, int n_chunks, int cpi, int chunk_tiles, int band_pos, int np_max, int a_words, size_t lds,
                float *P, uint8_t *S, uint8_t *TF, float *VF, const PoolOut &po, int arith, hipStream_t st) {
    // one workgroup per CU: a multiple of the feature pairs on every XCD
    const int per_xcd = (int)spk::ceil_div(std::max(32, n_pairs), n_pairs) * n_pairs;
    hipLaunchKernelGGL((k_conv_fire_fin<G, BLDS, ALDS, MODE>), dim3((unsigned)(per_xcd * 8)), dim3(FIN_THREADS), lds, st,
                       tpad, frag, koff2, g, n_pairs, n_chunks, cpi, chunk_tiles, band_pos, np_max, a_words, inv_scale,
                       wbf16, wts, wmax, wmin, n_wmax, P, S, TF, VF, po, arith);
}

// Position-major Eq.5 tasks pay when most of the receptive fields' K-steps are
// padding and there are enough (feature group, position, image block) tasks.
int inf_pm_nib(const ConvGeom &g, int ksplit) {
    if (ksplit > 1 || g.HoWo > 64 || (int64_t)g.Cout * g.HoWo > INF_PM_OUT || g.ksteps > 256) return 0;
    int64_t valid = 0;
    for (int pos = 0; pos < g.HoWo; ++pos)
        for (int ks = 0; ks < g.ksteps; ++ks) valid += kstep_valid(g, pos / g.Wo, pos % g.Wo, ks);
    const int nib = (int)spk::ceil_div(g.B, INF_PM_IMG);
    const int64_t n_ng = spk::ceil_div(spk::ceil_div(g.Cout, 16), INF_NW);
    const bool sparse = valid * 100 <= (int64_t)g.HoWo * g.ksteps * 85;
    return sparse && n_ng * g.HoWo * nib >= 128 ? nib : 0;
}

template <bool VEC>
void launch_inf(const uint8_t *tpad, const uint4 *frag, const int2 *koff2, const float *inv_scale, const int *wbf16,
                const ConvGeom &g, int ksplit, int kpp, float *part, float *P, uint8_t *S, uint8_t *TF, float *VF,
                hipStream_t st) {
    const int pm_nib = inf_pm_nib(g, ksplit);
    const int n_mb = pm_nib ? g.HoWo * pm_nib : (int)spk::ceil_div(g.total_mtiles, INF_WAVES * INF_MW);
    const int n_ng = (int)spk::ceil_div(spk::ceil_div(g.Cout, 16), INF_NW);
    const size_t lds = spk::align_up((size_t)g.ksteps * 4 * sizeof(int2), 16) + 2 * (size_t)INF_CHUNK_U4 * 16 +
                       2 * INF_KLMAX * sizeof(uint16_t) + (pm_nib ? 2 * (size_t)g.ksteps * 4 * sizeof(int2) : 0);
    if (!VEC && g.T > 1 && (P || S)) {  // (with VEC the conv kernel's zero waves write them)
        const int64_t n = (int64_t)(g.T - 1) * g.Cout * g.HoWo;
        const unsigned gx = (unsigned)std::max<int64_t>(1, std::min<int64_t>(64, spk::ceil_div(n, 256 * 16)));
        hipLaunchKernelGGL(k_zero_planes, dim3(gx, (unsigned)std::min(g.B, 65535)), dim3(256), 0, st, g, P, S);
    }
    if (pm_nib) {
        hipLaunchKernelGGL((k_conv_fire_inf<VEC, true>), dim3(256), dim3((INF_WAVES + INF_ZW) * 64), lds, st, tpad,
                           frag, koff2, g, n_mb, n_ng, ksplit, kpp, pm_nib, part, inv_scale, wbf16, P, S, TF, VF);
        hipLaunchKernelGGL(k_inf_pm_finish, dim3((unsigned)g.B), dim3(256), (size_t)g.Cout * (g.HoWo + 1) * sizeof(float), st,
                           part, g, inv_scale, P, S, TF, VF, VEC ? 1 : 0);
        return;
    }
        hipLaunchKernelGGL((k_conv_fire_inf<VEC, false>), dim3(256), dim3((INF_WAVES + INF_ZW) * 64), lds, st, tpad,
                           frag, koff2, g, n_mb, n_ng, ksplit, kpp, pm_nib, part, inv_scale, wbf16, P, S, TF, VF);
    if (ksplit > 1) {
        const int64_t n = (int64_t)g.B * g.Cout * g.HoWo;
        hipLaunchKernelGGL(k_inf_reduce, dim3((unsigned)spk::ceil_div(n, 256)), dim3(256), 0, st, part, ksplit, g,
                           inv_scale, P, S, TF, VF);
    }
}

}  // namespace

extern "C" size_t spk_conv_fire_workspace_size(int B, int T, int Cin, int H, int W, int Cout, int K, int pad) {
    ConvPlan pl;
    if (make_plan(B, T, Cin, H, W, Cout, K, 1, pad, pl) != SPK_OK) return 0;
    return plan_workspace(pl);
}

extern "C" size_t spk_conv_fire_strided_workspace_size(int B, int T, int Cin, int H, int W, int Cout, int K,
                                                       int stride, int pad) {
    ConvPlan pl;
    if (make_plan(B, T, Cin, H, W, Cout, K, stride, pad, pl) != SPK_OK) return 0;
    return plan_workspace(pl);
}

namespace {
// The conv call on either input form (times: in = first-spike map, else the
// wave); pool.P > 0 fuses first-spike pooling (window = stride = pool.P).
int conv_fire(const uint8_t *wave, bool times, int B, int T, int Cin, int H, int W, const float *weight, int Cout,
              int K, int stride, int pad, float threshold, float *potentials, uint8_t *spikes, uint8_t *t_first,
              float *v_first, void *workspace, size_t ws_bytes, void *stream,
              PoolOut pool = PoolOut{0, 0, 0, 0, nullptr, nullptr}, int arith = 0) {
    ConvPlan pl;
    int rc = make_plan(B, T, Cin, H, W, Cout, K, stride, pad, pl);
    if (rc != SPK_OK) return rc;
    SPK_REQUIRE(!std::isnan(threshold) && !(std::isinf(threshold) && threshold < 0), SPK_E_ARG,
                "spk_conv_fire: threshold must be a number or +INFINITY");
    const bool inf_mode = std::isinf(threshold);
    SPK_REQUIRE(arith == 0 || !inf_mode, SPK_E_ARG, "spk_conv_fire: the fp32 form needs a finite threshold");
    // 4-element store groups need aligned outputs and groups that never straddle a task
    bool vec = (pl.g.HoWo % 4) == 0 && ((uintptr_t)potentials & 15) == 0 && ((uintptr_t)v_first & 15) == 0 &&
               ((uintptr_t)spikes & 3) == 0 && ((uintptr_t)t_first & 3) == 0;
    const bool pooled = pool.P > 0;
    int band_pos = 0, band_rows = 0;
    bool flat_band = false;
    if (pooled) {  // tasks: bands of whole pooling rows, at most as many positions as a task holds
        SPK_REQUIRE(!inf_mode, SPK_E_ARG, "spk_conv_fire_pool: the threshold must be finite");
        SPK_REQUIRE(pl.g.Ho >= pool.P && pl.g.Wo >= pool.P, SPK_E_SHAPE,
                    "spk_conv_fire_pool: pooling window %d larger than the %dx%d map", pool.P, pl.g.Ho, pl.g.Wo);
        auto band = [&](bool v) {
            const int limit = 16 * chunk_tiles_max(v ? 4 : 1);
            band_rows = pool.P * std::max(1, limit / (pool.P * pl.g.Wo));
            band_pos = band_rows * pl.g.Wo;
            return limit;
        };
        band(vec);
        if (vec && band_pos % 4 != 0) vec = false;
        const int limit = band(vec);
        SPK_REQUIRE(pool.P * pl.g.Wo <= limit, SPK_E_RANGE,
                    "spk_conv_fire_pool: a band of %d rows of %d positions exceeds %d positions", pool.P, pl.g.Wo,
                    limit);
        pool.Hpo = pl.g.Ho / pool.P;
        pool.Wpo = pl.g.Wo / pool.P;
        // Bands run over the flattened (image, row) space -- every task full, a task
        // may end in the next image -- when every image starts on a window row
        // (Ho a multiple of P) and an image is more than one band; else per image.
        flat_band = pl.g.Ho % pool.P == 0 && pl.g.HoWo > band_pos &&
                    ((int64_t)T * Cout + 32) * pl.g.HoWo < (1LL << 31);
        // word stores of the pooled maps: every segment's run (its pooled rows of one
        // feature in one image) starts at a multiple of 4 bytes and has a multiple of
        // 4 positions; the segments repeat every lcm(band rows, Ho) flattened rows
        const int64_t pplane = (int64_t)pool.Hpo * pool.Wpo;
        bool runs4 = pplane % 4 == 0;
        const int64_t Ho = pl.g.Ho;
        const int64_t period_rows = flat_band ? band_rows / std::gcd((int64_t)band_rows, Ho) * Ho : Ho;
        for (int64_t r0 = 0; runs4 && r0 < period_rows; r0 += band_rows) {
            const int64_t r1 = flat_band ? r0 + band_rows : std::min(r0 + band_rows, Ho);
            for (int64_t r = r0; r < r1;) {  // segments of [r0, r1) by image
                const int64_t y0 = r % Ho, y1 = std::min(Ho, y0 + (r1 - r));
                const int64_t yo0 = y0 / pool.P, nyo = std::max<int64_t>(0, std::min<int64_t>(pool.Hpo, y1 / pool.P) - yo0);
                runs4 = runs4 && (yo0 * pool.Wpo) % 4 == 0 && (nyo * pool.Wpo) % 4 == 0;
                r += y1 - y0;
            }
        }
        pool.vec = runs4 && ((uintptr_t)pool.tf & 3) == 0 && ((uintptr_t)pool.wave & 3) == 0;
    }

    if (B == 0) return spk::ok();
    SPK_REQUIRE(wave && weight && t_first && v_first, SPK_E_ARG,
                "spk_conv_fire: the input, weight, t_first and v_first are required");
    const size_t need = plan_workspace(pl);
    SPK_REQUIRE(workspace && ws_bytes >= need, SPK_E_WORKSPACE,
                "spk_conv_fire: workspace of %zu bytes < %zu required", ws_bytes, need);
    ConvGeom g = pl.g;
    g.thr = inf_mode ? 0.0f : threshold;
    spk::Carver cv(workspace);
    uint8_t *tpad = cv.take<uint8_t>(pl.tpad_bytes);
    uint4 *frag = cv.take<uint4>(pl.frag_count);
    int2 *koff2 = cv.take<int2>(pl.koff_count);
    float *inv_scale = cv.take<float>(1);
    int *wbf16 = cv.take<int>(1);
    unsigned *wmax = cv.take<unsigned>(WMAX_PARTS);
    unsigned *wmin = cv.take<unsigned>(WMAX_PARTS);
    float *part = cv.take<float>(pl.part_count);
    hipStream_t st = spk::as_stream(stream);

    // finite-threshold launch configuration (validated before anything is enqueued)
    // Tasks: chunks of up to ct_max position tiles.  An image of at most ct_max
    // tiles is one task (each step's outputs of a feature pair are then one
    // contiguous region); larger images are cut into chunks of the flattened
    // (image, position) space, which may span two images, so that no tile slot
    // is padding (store offsets relative to the chunk's first image fit 32 bits).
    const int n_pairs = (int)spk::ceil_div(spk::ceil_div(Cout, 16), 2);
    // Few tiles in all (small batches, online steps): smaller chunks, so that
    // more workgroups share the call (at least 4 tiles per task).
    int ct_max = chunk_tiles_max(vec ? 4 : 1);
    while (ct_max > 4 && (int64_t)n_pairs * B * g.mt_per_img / ct_max < 256) ct_max /= 2;
    const int64_t npos = (int64_t)B * g.HoWo;
    const bool flat = pooled ? flat_band : g.mt_per_img > ct_max && ((int64_t)T * Cout + 32) * g.HoWo < (1LL << 31);
    int cpi, chunk_tiles, n_chunks;
    if (pooled && flat) {
        cpi = 0;
        chunk_tiles = (band_pos + 15) / 16;
        n_chunks = (int)spk::ceil_div(npos, band_pos);
    } else if (pooled) {
        cpi = (g.Ho + band_rows - 1) / band_rows;
        chunk_tiles = (std::min(band_pos, g.HoWo) + 15) / 16;
        n_chunks = B * cpi;
    } else if (flat) {
        cpi = 0;
        chunk_tiles = ct_max;
        n_chunks = (int)spk::ceil_div(npos, ct_max * 16);
    } else {
        cpi = (g.mt_per_img + ct_max - 1) / ct_max;
        chunk_tiles = (g.mt_per_img + cpi - 1) / cpi;
        n_chunks = B * cpi;
    }
    const int np_max = chunk_tiles * 16;
    const size_t koff_lds = spk::align_up((size_t)g.ksteps * 4 * sizeof(int2), 16);
    const size_t stage_lds = (size_t)FIN_TB * 32 * stage_stride(np_max) * sizeof(float);
    const size_t frag_lds = (size_t)g.ksteps * 2 * NT * 64 * 16;
    const size_t lds_limit = (size_t)max_lds_per_block();
    // spike rows of the largest task, staged in LDS (double-buffered) when small enough
    // (the row count of a chunk depends on its first position modulo HoWo, which repeats
    // every HoWo / gcd(HoWo, np_max) chunks; past 65536 of them a bound is used)
    const int cpos = pooled ? band_pos : np_max;  // positions per chunk
    auto chunk_rows = [&](int64_t p0) {
        const int64_t pb = std::min(p0 + cpos, npos) - 1;
        const int64_t ba = p0 / g.HoWo, bb = pb / g.HoWo;
        return (int)((bb * g.Hp + (pb - bb * g.HoWo) / g.Wo * stride + K) -
                     (ba * g.Hp + (p0 - ba * g.HoWo) / g.Wo * stride));
    };
    const int64_t period = g.HoWo / std::gcd((int64_t)g.HoWo, (int64_t)cpos);
    int a_rows = 0;
    if (!flat) {
        for (int ch = 0; ch < cpi; ++ch) {
            const int p0 = ch * cpos, np = std::min(cpos, g.HoWo - p0);
            a_rows = std::max(a_rows, ((p0 + np - 1) / g.Wo - p0 / g.Wo) * stride + K);
        }
    } else if (period <= 65536) {
        for (int64_t ch = 0; ch < std::min<int64_t>(n_chunks, period); ++ch)
            a_rows = std::max(a_rows, chunk_rows(ch * cpos));
    } else {  // HoWo > 65536 > cpos: a chunk touches at most two images
        a_rows = (cpos + g.Wo - 1) / g.Wo * stride + 2 * g.Hp + K;
    }
    // staged spike rows: CP >= 8 (8-byte reads of one channel group), buffers rounded to 64 words
    const int a_words = (int)spk::align_up((size_t)a_rows * g.Wp * g.CP / 4, 64);
    const size_t a_lds = 2 * (size_t)a_words * 4;
    const size_t pool_lds = pooled ? (size_t)32 * np_max : 0;
    const bool alds = g.CP >= 8 && koff_lds + stage_lds + a_lds + pool_lds <= lds_limit;
    const bool blds = koff_lds + frag_lds + stage_lds + (alds ? a_lds : 0) + pool_lds <= lds_limit;
    const size_t fin_lds = koff_lds + (blds ? frag_lds : 0) + stage_lds + (alds ? a_lds : 0) + pool_lds;
    const size_t inf_lds = koff_lds + 2 * (size_t)INF_CHUNK_U4 * 16 + 2 * INF_KLMAX * sizeof(uint16_t) +
                           (inf_pm_nib(g, pl.ksplit) ? 2 * (size_t)g.ksteps * 4 * sizeof(int2) : 0);
    SPK_REQUIRE(!inf_mode || inf_lds <= lds_limit, SPK_E_RANGE,
                "spk_conv_fire: needs %zu bytes of LDS per workgroup, the device has %zu", inf_lds, lds_limit);
    SPK_REQUIRE(inf_mode || fin_lds <= lds_limit, SPK_E_RANGE,
                "spk_conv_fire: needs %zu bytes of LDS per workgroup, the device has %zu", fin_lds, lds_limit);

    const int row_bytes = g.Wp * g.CP;
    const int rows_per_chunk = std::min(g.Hp, PAD_LDS / row_bytes);
    const int nchunk = (int)spk::ceil_div(g.Hp, rows_per_chunk), ny = std::min(B, 65535);
    const int64_t nw = (int64_t)Cout * Cin * K * K;
    const int wper = (int)spk::align_up((size_t)std::max<int64_t>(4096, spk::ceil_div(nw, WMAX_PARTS)), 1024);
    const size_t pad_lds =
        (size_t)pad_raw_offset(g, rows_per_chunk) + (pad_raw_fits(g, nchunk) ? (size_t)Cin * H * W : 0);
    const int n_wmax = (int)spk::ceil_div(nw, wper);
    const dim3 pad_grid((unsigned)((int64_t)nchunk * ny + n_wmax));
    if (times)
        hipLaunchKernelGGL(k_pad_first_spike<true>, pad_grid, dim3(256), pad_lds, st, wave, g, rows_per_chunk, nchunk, ny,
                           tpad, weight, nw, wper, wmax, wmin);
    else
        hipLaunchKernelGGL(k_pad_first_spike<false>, pad_grid, dim3(256), pad_lds, st, wave, g, rows_per_chunk, nchunk, ny,
                           tpad, weight, nw, wper, wmax, wmin);
    if (inf_mode || !blds) {  // fragments in the workspace (the finite-threshold kernel with LDS room builds its own)
        if (g.CP % 32 == 0 && arith != 1) {
            hipLaunchKernelGGL(k_split_weights_cells, dim3((unsigned)(g.ntiles * (g.CP / 8))), dim3(256), 0, st, weight,
                               g, wmax, wmin, n_wmax, frag, koff2, inv_scale, wbf16);
        } else {
            const int64_t n2 = std::max<int64_t>((int64_t)pl.frag_count, (int64_t)pl.koff_count);
            hipLaunchKernelGGL(k_split_weights, dim3((unsigned)spk::ceil_div(n2, 256)), dim3(256), 0, st, weight, g,
                               wmax, wmin, n_wmax, frag, koff2, inv_scale, wbf16, arith);
        }
    }
    if (inf_mode) {
        if (vec)
            launch_inf<true>(tpad, frag, koff2, inv_scale, wbf16, g, pl.ksplit, pl.kpp, part, potentials, spikes,
                             t_first, v_first, st);
        else
            launch_inf<false>(tpad, frag, koff2, inv_scale, wbf16, g, pl.ksplit, pl.kpp, part, potentials, spikes,
                              t_first, v_first, st);
    } else {
#define SPK_FIN(G, BL, AL)                                                                                        \
    do {                                                                                                          \
        if (arith == 1)                                                                                           \
            launch_fin<G, BL, AL, FIN_F32>(tpad, frag, koff2, inv_scale, wbf16, weight, wmax, wmin, n_wmax, g,      \
                                           n_pairs, n_chunks, cpi, chunk_tiles, band_pos, np_max, a_words, fin_lds, \
                                           potentials, spikes, t_first, v_first, pool, arith, st);                  \
        else if (pooled)                                                                                          \
            launch_fin<G, BL, AL, FIN_POOL>(tpad, frag, koff2, inv_scale, wbf16, weight, wmax, wmin, n_wmax, g,     \
                                            n_pairs, n_chunks, cpi, chunk_tiles, band_pos, np_max, a_words,         \
                                            fin_lds, potentials, spikes, t_first, v_first, pool, arith, st);        \
        else                                                                                                      \
            launch_fin<G, BL, AL, FIN_SPLIT>(tpad, frag, koff2, inv_scale, wbf16, weight, wmax, wmin, n_wmax, g,    \
                                             n_pairs, n_chunks, cpi, chunk_tiles, band_pos, np_max, a_words,        \
                                             fin_lds, potentials, spikes, t_first, v_first, pool, arith, st);       \
    } while (0)
        const int sel = (vec ? 4 : 0) + (blds ? 2 : 0) + (alds ? 1 : 0);
        switch (sel) {
            case 0: SPK_FIN(1, false, false); break;
            case 1: SPK_FIN(1, false, true); break;
            case 2: SPK_FIN(1, true, false); break;
            case 3: SPK_FIN(1, true, true); break;
            case 4: SPK_FIN(4, false, false); break;
            case 5: SPK_FIN(4, false, true); break;
            case 6: SPK_FIN(4, true, false); break;
            default: SPK_FIN(4, true, true); break;
        }
#undef SPK_FIN
    }
    return spk::check_launch("spk_conv_fire");
}
}  // namespace

extern "C" int spk_conv_fire(const uint8_t *wave, int B, int T, int Cin, int H, int W, const float *weight,
                             int Cout, int K, int pad, float threshold, float *potentials, uint8_t *spikes,
                             uint8_t *t_first, float *v_first, void *workspace, size_t ws_bytes, void *stream) {
    return conv_fire(wave, false, B, T, Cin, H, W, weight, Cout, K, 1, pad, threshold, potentials, spikes, t_first,
                     v_first, workspace, ws_bytes, stream);
}

extern "C" int spk_conv_fire_first_spike(const uint8_t *in_t_first, int B, int T, int Cin, int H, int W,
                                         const float *weight, int Cout, int K, int pad, float threshold,
                                         float *potentials, uint8_t *spikes, uint8_t *t_first, float *v_first,
                                         void *workspace, size_t ws_bytes, void *stream) {
    return conv_fire(in_t_first, true, B, T, Cin, H, W, weight, Cout, K, 1, pad, threshold, potentials, spikes,
                     t_first, v_first, workspace, ws_bytes, stream);
}

extern "C" int spk_conv_fire_first_spike_f32mfma(const uint8_t *in_t_first, int B, int T, int Cin, int H, int W,
                                                 const float *weight, int Cout, int K, int pad, float threshold,
                                                 float *potentials, uint8_t *spikes, uint8_t *t_first,
                                                 float *v_first, void *workspace, size_t ws_bytes, void *stream) {
    return conv_fire(in_t_first, true, B, T, Cin, H, W, weight, Cout, K, 1, pad, threshold, potentials, spikes,
                     t_first, v_first, workspace, ws_bytes, stream, PoolOut{0, 0, 0, 0, nullptr, nullptr}, 1);
}

extern "C" int spk_conv_fire_pool(const uint8_t *in_t_first, int B, int T, int Cin, int H, int W,
                                  const float *weight, int Cout, int K, int pad, float threshold, int pool,
                                  float *potentials, uint8_t *spikes, uint8_t *t_first, float *v_first,
                                  uint8_t *pooled_t_first, uint8_t *pooled_wave, void *workspace, size_t ws_bytes,
                                  void *stream) {
    SPK_REQUIRE(pool >= 1, SPK_E_SHAPE, "spk_conv_fire_pool: pooling window %d < 1", pool);
    SPK_REQUIRE(pooled_t_first || B == 0, SPK_E_ARG, "spk_conv_fire_pool: pooled_t_first is required");
    return conv_fire(in_t_first, true, B, T, Cin, H, W, weight, Cout, K, 1, pad, threshold, potentials, spikes,
                     t_first, v_first, workspace, ws_bytes, stream, PoolOut{pool, 0, 0, 0, pooled_t_first, pooled_wave});
}

extern "C" int spk_conv_fire_strided(const uint8_t *wave, int B, int T, int Cin, int H, int W, const float *weight,
                                     int Cout, int K, int stride, int pad, float threshold, float *potentials,
                                     uint8_t *spikes, uint8_t *t_first, float *v_first, void *workspace,
                                     size_t ws_bytes, void *stream) {
    return conv_fire(wave, false, B, T, Cin, H, W, weight, Cout, K, stride, pad, threshold, potentials, spikes,
                     t_first, v_first, workspace, ws_bytes, stream);
}

extern "C" int spk_conv_fire_first_spike_strided(const uint8_t *in_t_first, int B, int T, int Cin, int H, int W,
                                                 const float *weight, int Cout, int K, int stride, int pad,
                                                 float threshold, float *potentials, uint8_t *spikes,
                                                 uint8_t *t_first, float *v_first, void *workspace, size_t ws_bytes,
                                                 void *stream) {
    return conv_fire(in_t_first, true, B, T, Cin, H, W, weight, Cout, K, stride, pad, threshold, potentials, spikes,
                     t_first, v_first, workspace, ws_bytes, stream);
}

// ------------------------------------------------------------------ allocation-free variant
// The workspace of spk_conv_fire_first_spike_noalloc: a static device array,
// one copy per GPU, held until the process ends.  In host code `scratch` is
// only a stand-in for the symbol: its device address, per device, comes from
// hipGetSymbolAddress and is what the kernels receive.  Nothing in the conv
// workspace needs to start at zero (every byte a kernel reads was written
// earlier in the same call), so calls do not clear it.
constexpr size_t SPK_NOALLOC_SCRATCH_BYTES = size_t(64) << 20;
static __device__ __align__(256) uint8_t scratch[SPK_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int SPK_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[SPK_MAX_DEVICES] = {};

// Device address of the current device's scratch (looked up once per device).
int current_scratch(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= SPK_MAX_DEVICES)
        return spk::fail(SPK_E_HIP, "spk_conv_fire_first_spike_noalloc: no usable current device (%d)", dev);
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return spk::fail(SPK_E_HIP, "spk_conv_fire_first_spike_noalloc: hipGetSymbolAddress failed on device %d: %s",
                             dev, hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return SPK_OK;
}
}  // namespace

extern "C" int spk_conv_fire_first_spike_noalloc(const uint8_t *in_t_first, int B, int T, int Cin, int H, int W,
                                                 const float *weight, int Cout, int K, int pad, float threshold,
                                                 float *potentials, uint8_t *spikes, uint8_t *t_first,
                                                 float *v_first, void *stream) {
    ConvPlan pl;
    int rc = make_plan(B, T, Cin, H, W, Cout, K, 1, pad, pl);
    if (rc != SPK_OK) return rc;
    const size_t need = plan_workspace(pl);
    SPK_REQUIRE(need <= SPK_NOALLOC_SCRATCH_BYTES, SPK_E_RANGE,
                "spk_conv_fire_first_spike_noalloc: the call needs %zu bytes of scratch, the static scratch holds %zu "
                "(use spk_conv_fire_first_spike with a workspace)",
                need, SPK_NOALLOC_SCRATCH_BYTES);
    if (B == 0) return conv_fire(in_t_first, true, B, T, Cin, H, W, weight, Cout, K, 1, pad, threshold, potentials,
                                 spikes, t_first, v_first, nullptr, 0, stream);
    void *ws = nullptr;
    rc = current_scratch(&ws);
    if (rc != SPK_OK) return rc;
    return conv_fire(in_t_first, true, B, T, Cin, H, W, weight, Cout, K, 1, pad, threshold, potentials, spikes,
                     t_first, v_first, ws, SPK_NOALLOC_SCRATCH_BYTES, stream);
}
