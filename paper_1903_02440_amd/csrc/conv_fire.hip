// Convolution of a cumulative spike wave + firing, fused (gfx950).
//
// Paper: section "snn Module" (per-step valid convolution over all time
// steps at once, Eq.2), "functional Module" (fire / threshold) and Eq.5
// (infinite threshold, in place).
//
// Formulation.  For output neuron (f, y, x) and step t
//     P[t,f,y,x] = sum_k W[f,k] * [tp_k <= t]
// where k = (ci, ky, kx) runs over the receptive field and tp_k is the
// first-spike step of that input neuron (Eq.1 makes S[t] = [tp <= t]).
// Per image this is a GEMM  P_t[pos, f] = A_t[pos, k] * W^T[k, f]  for every
// t, with a binary A_t generated on the fly from the u8 first-spike map.
// It runs on the fp16 matrix cores (v_mfma_f32_16x16x32_f16): A_t is exact
// in fp16 (we use the value 2.0 for a spike, a single bit), and every fp32
// weight, scaled by a power of two so that the layer's largest weight lies in
// [2^12, 2^13) and halved, is split into hi = fp16(v), lo = fp16(v - hi):
// each product pair carries 22 significant bits of w for every weight down to
// 2^-17 times the largest; accumulation is fp32 and the result is scaled back
// exactly.
//
// Pipeline of one call (all on the caller's stream):
//   1. k_pad_first_spike: wave [B,T,Cin,H,W] -> zero-padded first-spike map
//      tpad [B,Cin,H+2p,W+2p] (border = T: padding never spikes).
//   2. k_weight_absmax + k_split_weights: W -> scaled hi/lo fp16 B-operand
//      fragments + the receptive field offset table koff[k] = (ci*Hp + ky)*Wp + kx.
//   3. k_conv_fire: the GEMM for all steps of a block of TB time steps, with
//      threshold, spike, first-spike time and potential-at-first-spike in the
//      epilogue; potentials and spikes are stored straight from registers.
#include <algorithm>
#include <cmath>

#include "common.hpp"

namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int WAVES = 4;  // waves per workgroup
constexpr int NW_MAX = 4;  // N tiles per wave never exceed this; ntiles is padded to a multiple

struct ConvGeom {
    int B, T, Cin, H, W, Cout, K, pad;
    int Hp, Wp, Ho, Wo, HoWo;
    int Kc;          // Cin*K*K
    int ksteps;      // ceil(Kc/32)
    int ntiles;      // ceil(Cout/16) rounded up to a multiple of NW_MAX
    int mt_per_img;  // ceil(HoWo/16)
    int64_t total_mtiles;
    float thr;
    int inf_mode;
    int vec4;        // HoWo % 4 == 0: 16-byte potential / 4-byte spike stores
};

// 1. first-spike times of the padded input.  Grid (chunk of padded rows,
// images).  A chunk is up to PAD_LDS bytes of whole padded rows of one image;
// its interior cells come from one contiguous range of the input plane.  The
// workgroup fills an LDS copy of the chunk with T (padding never spikes),
// counts the ones of every interior cell over the T steps (4 cells per 4-byte
// load when the wave pointer and the plane size are multiples of 4), drops
// t_first = T - count into LDS, then writes the chunk out with 16-byte stores.
// The LDS copy is shifted by the chunk's address mod 16, so LDS and global
// 16-byte boundaries coincide.  32-bit index arithmetic within an image.
constexpr int PAD_LDS = 32768;

__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t w) {  // 1 in every nonzero byte
    return ((((w & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | w) & 0x80808080u) >> 7;
}

__global__ __launch_bounds__(256) void k_pad_first_spike(const uint8_t *__restrict__ wave, ConvGeom g,
                                                         int rows_per_chunk, int words, uint8_t *__restrict__ tpad) {
    __shared__ __attribute__((aligned(16))) uint8_t buf[PAD_LDS + 16];
    const int tid = threadIdx.x;
    const int plane = g.Cin * g.H * g.W, hw = g.H * g.W;
    const int rows_img = g.Cin * g.Hp;
    const int r0 = blockIdx.x * rows_per_chunk;
    const int nr = min(rows_per_chunk, rows_img - r0);
    const int nbytes = nr * g.Wp;
    // the input range [i_begin, i_end) of the chunk's interior rows
    int ci = r0 / g.Hp, py = r0 - ci * g.Hp;
    if (py < g.pad) py = g.pad;
    else if (py >= g.pad + g.H) { ++ci; py = g.pad; }
    const int i_begin = ci * hw + (py - g.pad) * g.W;
    ci = (r0 + nr - 1) / g.Hp;
    py = r0 + nr - 1 - ci * g.Hp;
    if (py >= g.pad + g.H) py = g.pad + g.H - 1;
    else if (py < g.pad) { --ci; py = g.pad + g.H - 1; }
    const int i_end = ci * hw + (py - g.pad + 1) * g.W;
    const uint32_t tfill = (uint32_t)g.T * 0x01010101u;
    for (int64_t b = blockIdx.y; b < g.B; b += gridDim.y) {
        uint8_t *out = tpad + (b * rows_img + r0) * g.Wp;
        const int shift = (int)((uintptr_t)out & 15);
        for (int i = tid * 4; i < shift + nbytes; i += 1024) *reinterpret_cast<uint32_t *>(buf + i) = tfill;
        __syncthreads();
        const uint8_t *src = wave + b * g.T * plane;
        for (int w = (i_begin & ~3) + tid * 4; w < i_end; w += 1024) {
            uint32_t cnt = 0;  // four byte counters (T <= 255)
            const uint8_t *p = src + w;
            if (words) {
#pragma unroll 8
                for (int tt = 0; tt < g.T; ++tt, p += plane) cnt += nonzero_bytes(*reinterpret_cast<const uint32_t *>(p));
            } else {
                for (int tt = 0; tt < g.T; ++tt, p += plane)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        if (w + q >= i_begin && w + q < i_end) cnt += (uint32_t)(p[q] != 0) << (8 * q);
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int i = w + q;
                if (i < i_begin || i >= i_end) continue;
                const int c = i / hw, pix = i - c * hw;
                const int y = pix / g.W, x = pix - y * g.W;
                // a cumulative wave has exactly T - t_first ones
                buf[shift + (c * g.Hp + y + g.pad - r0) * g.Wp + x + g.pad] =
                    (uint8_t)(g.T - (int)((cnt >> (8 * q)) & 0xFFu));
            }
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

// 2. weight fragments.  Every weight is scaled by a power of two
// s = 2^(12 - E), E = the exponent of max|w|, so the largest scaled weight lies
// in [2^12, 2^13): then both terms of the split are normal fp16 for every
// weight down to max|w| * 2^-17, i.e. w*s = hi + lo + e with |e| <= 2^-22 |w*s|.
// The GEMM result is multiplied back by 1/s (exact).  The factor also carries
// the 1/2 that compensates the spike operand 2.0.  Fragment (nt, ks, lane)
// holds, for feature n = nt*16 + lane%16, the 8 taps k = ks*32 + 8*(lane/16) + j.
__global__ __launch_bounds__(256) void k_weight_absmax(const float *__restrict__ w, int64_t n,
                                                       unsigned *__restrict__ maxbits) {
    unsigned m = 0;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
        m = max(m, __float_as_uint(fabsf(w[i])));
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) m = max(m, (unsigned)__shfl_xor((int)m, s, 64));
    if ((threadIdx.x & 63) == 0 && m) atomicMax(maxbits, m);
}

__device__ __forceinline__ int weight_scale_exp(unsigned maxbits) {
    const int E = maxbits ? (int)((maxbits >> 23) & 255u) - 127 : 0;  // subnormal maxima count as 2^-127
    return 12 - max(-100, min(100, E));
}

__global__ __launch_bounds__(256) void k_split_weights(const float *__restrict__ w, ConvGeom g,
                                                       const unsigned *__restrict__ maxbits,
                                                       half8 *__restrict__ whi, half8 *__restrict__ wlo,
                                                       int *__restrict__ koff, float *__restrict__ inv_scale) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t total = (int64_t)g.ntiles * g.ksteps * 64;
    const int e = weight_scale_exp(*maxbits);
    if (i == 0) *inv_scale = ldexpf(1.0f, -e);
    if (i < total) {
        const int lane = (int)(i & 63);
        const int64_t r = i >> 6;
        const int ks = (int)(r % g.ksteps);
        const int nt = (int)(r / g.ksteps);
        const int n = nt * 16 + (lane & 15);
        half8 h, l;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int k = ks * 32 + (lane >> 4) * 8 + j;
            // scaled by 2^(e-1): the spike operand is 2.0, so the products are w * 2^e
            const float v = (n < g.Cout && k < g.Kc) ? ldexpf(w[(int64_t)n * g.Kc + k], e - 1) : 0.0f;
            const _Float16 hv = (_Float16)v;
            const float rest = v - (float)hv;  // exact: hv is within half an fp16 ulp of v
            h[j] = hv;
            l[j] = (_Float16)rest;
        }
        whi[i] = h;
        wlo[i] = l;
    }
    if (i < (int64_t)g.ksteps * 32) {
        const int k = (int)i;
        int off = 0;
        if (k < g.Kc) {
            const int ci = k / (g.K * g.K), rem = k % (g.K * g.K);
            const int ky = rem / g.K, kx = rem % g.K;
            off = (ci * g.Hp + ky) * g.Wp + kx;
        }
        koff[k] = off;
    }
}

// 3. the fused GEMM + fire.  A wave owns MW consecutive 16-position M tiles
// (across the whole batch) and NW 16-feature N tiles, for all time steps,
// processed TB steps at a time.  Lane l feeds A row l%16 / B column l%16
// with the 8 taps 8*(l/16)..+7 and receives C[4*(l/16) + j][l%16], j = 0..3:
// four consecutive positions of one feature.
//
// The four waves of a workgroup share their NW feature tiles, so the weight
// fragments are staged once per workgroup in LDS, KC K-steps at a time; the
// spike-time gathers of K-step ks+1 are in flight while step ks computes.
// Steps past T in the last time block are computed but never stored.
//
// Block order is XCD-aware: hardware hands consecutive workgroups to the 8
// XCDs in turn, so block i is remapped to logical block
// (i % 8) * ceil(nblk / 8) + i / 8.  Each XCD then sweeps a contiguous range
// of positions, and the partial 128-byte lines at the edges of one block's
// output runs are completed by its neighbour in the same L2 before they are
// written back.
constexpr int KC = 8;                 // K-steps of weight fragments per LDS chunk, at most
constexpr size_t LDS_BUDGET = 79872;  // per workgroup: two workgroups fit one CU's 160 KiB

template <int MW>
__device__ __forceinline__ void gather_tp(uint32_t (&tp)[MW][8], int ks, const uint8_t *__restrict__ tpad,
                                          const uint32_t (&abase)[MW], const int *koff_lds, int gq) {
    const int *ko = koff_lds + ks * 32 + gq * 8;
    int o[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = ko[j];
#pragma unroll
    for (int i = 0; i < MW; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) tp[i][j] = tpad[abase[i] + (uint32_t)o[j]];
}

template <int MW, int NW, int TB>
__device__ __forceinline__ void mfma_kstep(const uint32_t (&tp)[MW][8], const uint4 *fr, int lane,
                                           f4 (&acc)[MW][NW][TB], int tb0) {
    half8 bh[NW], bl[NW];
#pragma unroll
    for (int n = 0; n < NW; ++n) {
        bh[n] = __builtin_bit_cast(half8, fr[(2 * n) * 64 + lane]);
        bl[n] = __builtin_bit_cast(half8, fr[(2 * n + 1) * 64 + lane]);
    }
#pragma unroll
    for (int i = 0; i < MW; ++i) {
        // 16-bit lanes: (0x4000 + t - tp) has bit 14 set iff tp <= t (no borrow
        // crosses the halves since 0x4000 > 255); 0x4000 is fp16 2.0
        uint32_t d[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) d[q] = (0x4000u + (uint32_t)tb0) * 0x10001u - (tp[i][2 * q] | (tp[i][2 * q + 1] << 16));
#pragma unroll
        for (int t = 0; t < TB; ++t) {
            u4 a;
            a.x = d[0] & 0x40004000u;
            a.y = d[1] & 0x40004000u;
            a.z = d[2] & 0x40004000u;
            a.w = d[3] & 0x40004000u;
            const half8 ah = __builtin_bit_cast(half8, a);
#pragma unroll
            for (int n = 0; n < NW; ++n)
                acc[i][n][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bh[n], acc[i][n][t], 0, 0, 0);
#pragma unroll
            for (int n = 0; n < NW; ++n)
                acc[i][n][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bl[n], acc[i][n][t], 0, 0, 0);
#pragma unroll
            for (int q = 0; q < 4; ++q) d[q] += 0x10001u;
        }
    }
}

template <int MW, int NW, int TB, bool INF>
__device__ __forceinline__ void conv_tile(float inv_s, const uint8_t *__restrict__ tpad, const uint4 *frl_all,
                                          const int *koff_lds,
                                          const half8 *__restrict__ wfh, const half8 *__restrict__ wfl, uint4 *frl_chunk,
                                          bool resident, int kc, const ConvGeom &g, int ng, int mg, bool active,
                                          int tid, int lane, int gq, int c, float *__restrict__ P,
                                          uint8_t *__restrict__ S, uint8_t *__restrict__ TF, float *__restrict__ VF) {
    uint32_t abase[MW];
    int64_t img[MW];
    int mpos0[MW];
#pragma unroll
    for (int i = 0; i < MW; ++i) {
        const int64_t gm = (int64_t)mg * MW + i;
        const bool v = active && gm < g.total_mtiles;
        const int64_t b = v ? gm / g.mt_per_img : 0;
        const int mt = v ? (int)(gm % g.mt_per_img) : 0;
        const int pos = min(mt * 16 + c, g.HoWo - 1);  // rows past the image are computed, not stored
        const int y = pos / g.Wo, x = pos % g.Wo;
        abase[i] = (uint32_t)(((int64_t)b * g.Cin * g.Hp + y) * g.Wp + x);
        img[i] = v ? b : -1;
        mpos0[i] = mt * 16 + gq * 4;
    }
    // per (tile, feature) store offsets at step 0; a step adds Cout*HoWo
    const int64_t tstride = (int64_t)g.Cout * g.HoWo;
    int64_t obase[MW][NW];
    bool ost[MW][NW];
#pragma unroll
    for (int i = 0; i < MW; ++i)
#pragma unroll
        for (int n = 0; n < NW; ++n) {
            const int f = (ng * NW + n) * 16 + c;
            ost[i][n] = img[i] >= 0 && f < g.Cout && mpos0[i] < g.HoWo;
            obase[i][n] = ost[i][n] ? (img[i] * g.T * tstride + (int64_t)f * g.HoWo + mpos0[i]) : 0;
        }
    const bool full4 = g.vec4 != 0;

    int tfirst[MW][NW][4];
    float vfirst[MW][NW][4];
#pragma unroll
    for (int i = 0; i < MW; ++i)
#pragma unroll
        for (int n = 0; n < NW; ++n)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                tfirst[i][n][j] = g.T;
                vfirst[i][n][j] = 0.0f;
            }

    const int t_begin = INF ? g.T - 1 : 0;
    for (int tb0 = t_begin; tb0 < g.T; tb0 += TB) {
        f4 acc[MW][NW][TB];
#pragma unroll
        for (int i = 0; i < MW; ++i)
#pragma unroll
            for (int n = 0; n < NW; ++n)
#pragma unroll
                for (int t = 0; t < TB; ++t) acc[i][n][t] = f4{0.f, 0.f, 0.f, 0.f};

        for (int k0 = 0; k0 < g.ksteps; k0 += kc) {
            const int nk = min(kc, g.ksteps - k0);
            const uint4 *fr = frl_all + (size_t)k0 * NW * 2 * 64;
            if (!resident) {  // stream this chunk of fragments through LDS (uniform branch)
                __syncthreads();
                for (int idx = tid; idx < nk * NW * 2 * 64; idx += 256) {
                    const int ln = idx & 63, r = idx >> 6;  // r = (ksl*NW + n)*2 + h
                    const int h = r & 1, n = (r >> 1) % NW, ksl = (r >> 1) / NW;
                    const half8 *src = h ? wfl : wfh;
                    frl_chunk[idx] = __builtin_bit_cast(uint4, src[(n * g.ksteps + k0 + ksl) * 64 + ln]);
                }
                __syncthreads();
                fr = frl_chunk;
            }
            if (active) {
                uint32_t ta[MW][8], tb[MW][8];
                gather_tp<MW>(ta, k0, tpad, abase, koff_lds, gq);
                for (int kl = 0; kl < nk; kl += 2) {
                    if (kl + 1 < nk) gather_tp<MW>(tb, k0 + kl + 1, tpad, abase, koff_lds, gq);
                    mfma_kstep<MW, NW, TB>(ta, fr + kl * NW * 2 * 64, lane, acc, tb0);
                    if (kl + 1 >= nk) break;
                    if (kl + 2 < nk) gather_tp<MW>(ta, k0 + kl + 2, tpad, abase, koff_lds, gq);
                    mfma_kstep<MW, NW, TB>(tb, fr + (kl + 1) * NW * 2 * 64, lane, acc, tb0);
                }
            }
        }
        if (!active) continue;

        // epilogue: potentials, spikes and first-spike tracking of this time block
#pragma unroll
        for (int t = 0; t < TB; ++t) {
            const int tt = tb0 + t;
            if (tt >= g.T) break;  // uniform
#pragma unroll
            for (int i = 0; i < MW; ++i)
#pragma unroll
                for (int n = 0; n < NW; ++n) {
                    const f4 v = acc[i][n][t] * inv_s;  // undo the weight scaling (a power of two)
                    uint32_t sp = 0;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const bool s = INF ? (v[j] > 0.0f) : (v[j] >= g.thr);
                        const bool first = s && tfirst[i][n][j] == g.T;
                        tfirst[i][n][j] = first ? tt : tfirst[i][n][j];
                        vfirst[i][n][j] = first ? v[j] : vfirst[i][n][j];
                        sp |= s ? (1u << (8 * j)) : 0u;
                    }
                    if (!ost[i][n]) continue;
                    const int64_t o = obase[i][n] + (int64_t)tt * tstride;
                    if (full4) {
                        if (P) *reinterpret_cast<f4 *>(P + o) = v;
                        if (S) *reinterpret_cast<uint32_t *>(S + o) = sp;
                    } else {
                        const int lim = g.HoWo - mpos0[i];
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            if (j < lim) {
                                if (P) P[o + j] = v[j];
                                if (S) S[o + j] = (uint8_t)(sp >> (8 * j));
                            }
                    }
                }
        }
    }
    if (!active) return;

    // Eq.5 mode: every step before the last holds zero potential and no spike.
    if (INF) {
        for (int tt = 0; tt < g.T - 1; ++tt) {
#pragma unroll
            for (int i = 0; i < MW; ++i)
#pragma unroll
                for (int n = 0; n < NW; ++n) {
                    if (!ost[i][n]) continue;
                    const int64_t o = obase[i][n] + (int64_t)tt * tstride;
                    if (full4) {
                        if (P) *reinterpret_cast<f4 *>(P + o) = f4{0.f, 0.f, 0.f, 0.f};
                        if (S) *reinterpret_cast<uint32_t *>(S + o) = 0u;
                    } else {
                        const int lim = g.HoWo - mpos0[i];
                        for (int j = 0; j < 4 && j < lim; ++j) {
                            if (P) P[o + j] = 0.0f;
                            if (S) S[o + j] = 0;
                        }
                    }
                }
        }
    }

    // first-spike time and the potential there
#pragma unroll
    for (int i = 0; i < MW; ++i)
#pragma unroll
        for (int n = 0; n < NW; ++n) {
            if (!ost[i][n]) continue;
            const int f = (ng * NW + n) * 16 + c;
            const int64_t o = (img[i] * (int64_t)g.Cout + f) * g.HoWo + mpos0[i];
            if (full4) {
                uint32_t tv = 0;
#pragma unroll
                for (int j = 0; j < 4; ++j) tv |= (uint32_t)tfirst[i][n][j] << (8 * j);
                *reinterpret_cast<uint32_t *>(TF + o) = tv;
                *reinterpret_cast<f4 *>(VF + o) = f4{vfirst[i][n][0], vfirst[i][n][1], vfirst[i][n][2], vfirst[i][n][3]};
            } else {
                const int lim = g.HoWo - mpos0[i];
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (j < lim) {
                        TF[o + j] = (uint8_t)tfirst[i][n][j];
                        VF[o + j] = vfirst[i][n][j];
                    }
            }
        }
}

// Persistent workgroups.  Workgroup w runs on XCD x = w % 8; the XCDs split
// the M blocks (4 waves x MW tiles of 16 positions) into 8 contiguous slices.
// Each workgroup serves one feature group: it loads that group's weight
// fragments into LDS once (or streams them in chunks when they do not fit)
// and then takes the next M block of its XCD's slice from a counter shared by
// the workgroups of the same (XCD, feature group).  The workgroups of an XCD
// therefore always work on neighbouring positions, so the 128-byte lines
// shared by neighbouring output runs are completed in that XCD's L2 before
// they are written back.  Every workgroup stops when the slice is exhausted.
template <int MW, int NW, int TB, bool INF>
__global__ __launch_bounds__(256, 2) void k_conv_fire(const uint8_t *__restrict__ tpad,
                                                      const half8 *__restrict__ whi,
                                                      const half8 *__restrict__ wlo,
                                                      const int *__restrict__ koff, ConvGeom g,
                                                      int n_mgroups, int n_mblocks, int n_ngroups, int kc,
                                                      int resident, unsigned *__restrict__ counters,
                                                      const float *__restrict__ inv_scale,
                                                      float *__restrict__ P, uint8_t *__restrict__ S,
                                                      uint8_t *__restrict__ TF, float *__restrict__ VF) {
    extern __shared__ uint4 lds[];
    __shared__ int next_mb;
    const float inv_s = *inv_scale;
    int *koff_lds = reinterpret_cast<int *>(lds);      // ksteps*32 offsets
    uint4 *frl = lds + (g.ksteps * 32 * 4 + 15) / 16;  // fragments: all K-steps, or a chunk of kc
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int gq = lane >> 4, c = lane & 15;
    const int x = blockIdx.x % 8, j = blockIdx.x / 8;
    const int ng = j % n_ngroups;
    const int per_x = (n_mblocks + 7) / 8;
    const int mb_lo = x * per_x, mb_hi = min(n_mblocks, mb_lo + per_x);
    if (mb_lo >= mb_hi) return;  // whole workgroup: this XCD's slice is empty
    unsigned *ctr = counters + x * n_ngroups + ng;

    const half8 *wfh = whi + (int64_t)ng * NW * g.ksteps * 64;
    const half8 *wfl = wlo + (int64_t)ng * NW * g.ksteps * 64;
    for (int i = tid; i < g.ksteps * 32; i += 256) koff_lds[i] = koff[i];
    if (resident) {
        for (int idx = tid; idx < g.ksteps * NW * 2 * 64; idx += 256) {
            const int ln = idx & 63, r = idx >> 6;  // r = (ks*NW + n)*2 + h
            const int h = r & 1, n = (r >> 1) % NW, ks = (r >> 1) / NW;
            const half8 *src = h ? wfl : wfh;
            frl[idx] = __builtin_bit_cast(uint4, src[(n * g.ksteps + ks) * 64 + ln]);
        }
    }
    for (;;) {
        __syncthreads();  // LDS fills are visible; everyone has read the previous next_mb
        if (tid == 0) next_mb = mb_lo + (int)atomicAdd(ctr, 1u);
        __syncthreads();
        const int mb = next_mb;
        if (mb >= mb_hi) break;  // uniform
        const int mg = mb * WAVES + wv;
        conv_tile<MW, NW, TB, INF>(inv_s, tpad, frl, koff_lds, wfh, wfl, frl, resident != 0, resident ? g.ksteps : kc, g,
                                   ng, mg, mg < n_mgroups, tid, lane, gq, c, P, S, TF, VF);
    }
}

__global__ void k_zero_u32(unsigned *p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0u;
}

constexpr int MAX_NGROUPS_COUNT = 8 * 64;  // (XCD, feature group) counters reserved in the workspace

struct ConvPlan {
    ConvGeom g;
    size_t tpad_bytes, frag_count, koff_count;
};

int make_plan(int B, int T, int Cin, int H, int W, int Cout, int K, int pad, ConvPlan &pl) {
    SPK_REQUIRE(B >= 0 && T >= 1 && Cin >= 1 && H >= 1 && W >= 1 && Cout >= 1 && K >= 1 && pad >= 0,
                SPK_E_SHAPE, "spk_conv_fire: bad sizes B=%d T=%d Cin=%d H=%d W=%d Cout=%d K=%d pad=%d",
                B, T, Cin, H, W, Cout, K, pad);
    SPK_REQUIRE(T <= 255, SPK_E_RANGE, "spk_conv_fire: T=%d > 255", T);
    ConvGeom &g = pl.g;
    g.B = B; g.T = T; g.Cin = Cin; g.H = H; g.W = W; g.Cout = Cout; g.K = K; g.pad = pad;
    g.Hp = H + 2 * pad;
    g.Wp = W + 2 * pad;
    g.Ho = g.Hp - K + 1;
    g.Wo = g.Wp - K + 1;
    SPK_REQUIRE(g.Ho >= 1 && g.Wo >= 1, SPK_E_SHAPE, "spk_conv_fire: kernel %d larger than padded input %dx%d",
                K, g.Hp, g.Wp);
    SPK_REQUIRE((int64_t)Cin * K * K <= 16384, SPK_E_RANGE, "spk_conv_fire: Cin*K*K=%lld > 16384",
                (long long)Cin * K * K);
    SPK_REQUIRE(Cout <= 4096, SPK_E_RANGE, "spk_conv_fire: Cout=%d > 4096", Cout);
    SPK_REQUIRE((int64_t)g.Ho * g.Wo < (1LL << 31) && (int64_t)Cin * g.Hp * g.Wp <= 65535LL * 256 &&
                    g.Wp <= PAD_LDS,
                SPK_E_RANGE, "spk_conv_fire: image too large");
    // the MFMA kernel addresses the padded first-spike map with 32-bit offsets
    SPK_REQUIRE((int64_t)B * Cin * g.Hp * g.Wp < (1LL << 32), SPK_E_RANGE,
                "spk_conv_fire: padded input of %lld bytes exceeds 4 GiB", (long long)B * Cin * g.Hp * g.Wp);
    g.HoWo = g.Ho * g.Wo;
    g.Kc = Cin * K * K;
    g.ksteps = (g.Kc + 31) / 32;
    g.ntiles = (int)spk::ceil_div(spk::ceil_div(Cout, 16), NW_MAX) * NW_MAX;
    g.mt_per_img = (g.HoWo + 15) / 16;
    g.total_mtiles = (int64_t)B * g.mt_per_img;
    g.vec4 = (g.HoWo % 4) == 0;
    pl.tpad_bytes = (size_t)B * Cin * g.Hp * g.Wp;
    pl.frag_count = (size_t)g.ntiles * g.ksteps * 64;
    pl.koff_count = (size_t)g.ksteps * 32;
    return SPK_OK;
}

size_t plan_workspace(const ConvPlan &pl) {
    spk::Carver c(nullptr);
    c.take<uint8_t>(pl.tpad_bytes);
    c.take<half8>(pl.frag_count);
    c.take<half8>(pl.frag_count);
    c.take<int>(pl.koff_count);
    c.take<unsigned>(MAX_NGROUPS_COUNT + 2);  // work counters, max|w| bits, 1/scale
    return spk::align_up(c.off, 256);
}

template <int MW, int NW, int TB, bool INF>
void launch_conv(const uint8_t *tpad, const half8 *whi, const half8 *wlo, const int *koff, unsigned *counters,
                 const float *inv_scale, const ConvGeom &g, float *P, uint8_t *S, uint8_t *TF, float *VF,
                 hipStream_t st) {
    const int64_t n_mgroups = spk::ceil_div(g.total_mtiles, MW);
    const int64_t n_mblocks = spk::ceil_div(n_mgroups, WAVES);
    const int n_ngroups = (int)spk::ceil_div(spk::ceil_div(g.Cout, 16), NW);
    const size_t koff_bytes = spk::align_up((size_t)g.ksteps * 32 * sizeof(int), 16);
    const size_t step = (size_t)NW * 2 * 64 * 16;  // one K-step of fragments
    const int resident = koff_bytes + (size_t)g.ksteps * step <= LDS_BUDGET;
    const int kc = resident ? g.ksteps
                            : (int)std::max<size_t>(1, std::min<size_t>(KC, (LDS_BUDGET - koff_bytes) / step));
    const size_t lds = koff_bytes + (size_t)kc * step;
    // about two workgroups per CU (256 CUs, 32 per XCD), a multiple of the feature groups per XCD
    const int64_t want = spk::ceil_div(n_mblocks * n_ngroups, 8);
    const int64_t per_xcd = std::min<int64_t>(spk::ceil_div(std::max<int64_t>(64, n_ngroups), n_ngroups) * n_ngroups,
                                              spk::ceil_div(want, n_ngroups) * n_ngroups);
    // the 8 * n_ngroups counters (<= MAX_NGROUPS_COUNT since Cout <= 4096) were zeroed by the caller
    hipLaunchKernelGGL((k_conv_fire<MW, NW, TB, INF>), dim3((unsigned)(per_xcd * 8)), dim3(256), lds, st, tpad, whi,
                       wlo, koff, g, (int)n_mgroups, (int)n_mblocks, n_ngroups, kc, resident, counters, inv_scale, P,
                       S, TF, VF);
}

}  // namespace

extern "C" size_t spk_conv_fire_workspace_size(int B, int T, int Cin, int H, int W, int Cout, int K, int pad) {
    ConvPlan pl;
    if (make_plan(B, T, Cin, H, W, Cout, K, pad, pl) != SPK_OK) return 0;
    return plan_workspace(pl);
}

extern "C" int spk_conv_fire(const uint8_t *wave, int B, int T, int Cin, int H, int W, const float *weight,
                             int Cout, int K, int pad, float threshold, float *potentials, uint8_t *spikes,
                             uint8_t *t_first, float *v_first, void *workspace, size_t ws_bytes, void *stream) {
    ConvPlan pl;
    int rc = make_plan(B, T, Cin, H, W, Cout, K, pad, pl);
    if (rc != SPK_OK) return rc;
    SPK_REQUIRE(!std::isnan(threshold) && !(std::isinf(threshold) && threshold < 0), SPK_E_ARG,
                "spk_conv_fire: threshold must be a number or +INFINITY");
    if (B == 0) return spk::ok();
    SPK_REQUIRE(wave && weight && t_first && v_first, SPK_E_ARG,
                "spk_conv_fire: wave, weight, t_first and v_first are required");
    const size_t need = plan_workspace(pl);
    SPK_REQUIRE(workspace && ws_bytes >= need, SPK_E_WORKSPACE,
                "spk_conv_fire: workspace of %zu bytes < %zu required", ws_bytes, need);
    ConvGeom g = pl.g;
    g.inf_mode = std::isinf(threshold) ? 1 : 0;
    g.thr = g.inf_mode ? 0.0f : threshold;

    spk::Carver cv(workspace);
    uint8_t *tpad = cv.take<uint8_t>(pl.tpad_bytes);
    half8 *whi = cv.take<half8>(pl.frag_count);
    half8 *wlo = cv.take<half8>(pl.frag_count);
    int *koff = cv.take<int>(pl.koff_count);
    unsigned *counters = cv.take<unsigned>(MAX_NGROUPS_COUNT + 2);
    unsigned *maxbits = counters + MAX_NGROUPS_COUNT;
    float *inv_scale = reinterpret_cast<float *>(counters + MAX_NGROUPS_COUNT + 1);
    hipStream_t st = spk::as_stream(stream);

    const int rows_img = Cin * g.Hp;
    const int rows_per_chunk = std::min(rows_img, PAD_LDS / g.Wp);
    const int words = ((Cin * H * W) & 3) == 0 && ((uintptr_t)wave & 3) == 0;
    hipLaunchKernelGGL(k_pad_first_spike, dim3((unsigned)spk::ceil_div(rows_img, rows_per_chunk),
                                               (unsigned)std::min(B, 65535)),
                       dim3(256), 0, st, wave, g, rows_per_chunk, words, tpad);
    hipLaunchKernelGGL(k_zero_u32, dim3((unsigned)spk::ceil_div(MAX_NGROUPS_COUNT + 2, 256)), dim3(256), 0, st,
                       counters, MAX_NGROUPS_COUNT + 2);
    const int64_t nw = (int64_t)Cout * g.Kc;
    hipLaunchKernelGGL(k_weight_absmax, dim3((unsigned)std::min<int64_t>(256, spk::ceil_div(nw, 256))), dim3(256), 0,
                       st, weight, nw, maxbits);
    const int64_t n2 = std::max<int64_t>((int64_t)pl.frag_count, (int64_t)pl.koff_count);
    hipLaunchKernelGGL(k_split_weights, dim3((unsigned)spk::ceil_div(n2, 256)), dim3(256), 0, st, weight, g, maxbits,
                       whi, wlo, koff, inv_scale);
    // tile shape: one 16-position tile by two or four 16-feature tiles per wave
    // (two when the layer has at most 32 features), 2 waves per SIMD
    const bool wide = (Cout + 15) / 16 > 2;
    if (g.inf_mode) {
        if (wide) launch_conv<2, 4, 1, true>(tpad, whi, wlo, koff, counters, inv_scale, g, potentials, spikes, t_first, v_first, st);
        else launch_conv<2, 2, 1, true>(tpad, whi, wlo, koff, counters, inv_scale, g, potentials, spikes, t_first, v_first, st);
    } else if (wide) {
        launch_conv<1, 4, 8, false>(tpad, whi, wlo, koff, counters, inv_scale, g, potentials, spikes, t_first, v_first, st);
    } else if (T % 15 == 0) {
        launch_conv<1, 2, 15, false>(tpad, whi, wlo, koff, counters, inv_scale, g, potentials, spikes, t_first, v_first, st);
    } else {
        launch_conv<1, 2, 16, false>(tpad, whi, wlo, koff, counters, inv_scale, g, potentials, spikes, t_first, v_first, st);
    }
    return spk::check_launch("spk_conv_fire");
}
