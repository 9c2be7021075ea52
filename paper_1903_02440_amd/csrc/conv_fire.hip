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
// in fp16 (we use the value 2.0 for a spike, a single bit, and halve the
// result), and every fp32 weight is split into hi = fp16(w), lo = fp16(w-hi),
// so each product pair carries 22 significant bits of w; accumulation is fp32.
//
// Pipeline of one call (all on the caller's stream):
//   1. k_pad_first_spike: wave [B,T,Cin,H,W] -> zero-padded first-spike map
//      tpad [B,Cin,H+2p,W+2p] (border = T: padding never spikes).
//   2. k_split_weights: W -> hi/lo fp16 B-operand fragments + the receptive
//      field offset table koff[k] = (ci*Hp + ky)*Wp + kx.
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
constexpr int NW = 2;     // 16-feature N tiles per wave (all kernels)

struct ConvGeom {
    int B, T, Cin, H, W, Cout, K, pad;
    int Hp, Wp, Ho, Wo, HoWo;
    int Kc;          // Cin*K*K
    int ksteps;      // ceil(Kc/32)
    int ntiles;      // ceil(Cout/16) rounded up to a multiple of NW
    int mt_per_img;  // ceil(HoWo/16)
    int64_t total_mtiles;
    float thr;
    int inf_mode;
    int vec4;        // HoWo % 4 == 0: 16-byte potential / 4-byte spike stores
};

// 1. first-spike times of the padded input.
__global__ __launch_bounds__(256) void k_pad_first_spike(const uint8_t *__restrict__ wave, ConvGeom g,
                                                         uint8_t *__restrict__ tpad) {
    const int64_t total = (int64_t)g.B * g.Cin * g.Hp * g.Wp;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total) return;
    const int px = (int)(i % g.Wp);
    int64_t r = i / g.Wp;
    const int py = (int)(r % g.Hp);
    r /= g.Hp;
    const int ci = (int)(r % g.Cin);
    const int64_t b = r / g.Cin;
    const int y = py - g.pad, x = px - g.pad;
    int t = g.T;
    if (y >= 0 && y < g.H && x >= 0 && x < g.W) {
        const int64_t plane = (int64_t)g.Cin * g.H * g.W;
        const uint8_t *p = wave + b * g.T * plane + ((int64_t)ci * g.H + y) * g.W + x;
        int s = 0;
        for (int tt = 0; tt < g.T; ++tt) s += p[tt * plane] != 0;
        t = g.T - s;  // a cumulative wave has exactly T - t_first ones
    }
    tpad[i] = (uint8_t)t;
}

// 2. weight fragments.  Fragment (nt, ks, lane) holds, for feature
// n = nt*16 + lane%16, the 8 taps k = ks*32 + 8*(lane/16) + j.
__global__ __launch_bounds__(256) void k_split_weights(const float *__restrict__ w, ConvGeom g,
                                                       half8 *__restrict__ whi, half8 *__restrict__ wlo,
                                                       int *__restrict__ koff) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t total = (int64_t)g.ntiles * g.ksteps * 64;
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
            const float v = (n < g.Cout && k < g.Kc) ? w[(int64_t)n * g.Kc + k] : 0.0f;
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
// (across the whole batch) and NW 16-feature N tiles, for all time steps.
// Lane l feeds A row l%16 / B column l%16 with the 8 taps 8*(l/16)..+7 and
// receives C[4*(l/16) + j][l%16], j = 0..3: four consecutive positions of
// one feature.
template <int MW, int TB>
__global__ __launch_bounds__(256, 2) void k_conv_fire(const uint8_t *__restrict__ tpad,
                                                   const half8 *__restrict__ whi,
                                                   const half8 *__restrict__ wlo,
                                                   const int *__restrict__ koff, ConvGeom g,
                                                   int n_mgroups, int n_mblocks,
                                                   float *__restrict__ P, uint8_t *__restrict__ S,
                                                   uint8_t *__restrict__ TF, float *__restrict__ VF) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int gq = lane >> 4, c = lane & 15;
    const int ng = blockIdx.x / n_mblocks;
    const int mg = (blockIdx.x % n_mblocks) * WAVES + wv;
    if (mg >= n_mgroups) return;

    int64_t abase[MW], img[MW];
    int mpos0[MW];
#pragma unroll
    for (int i = 0; i < MW; ++i) {
        const int64_t gm = (int64_t)mg * MW + i;
        const bool v = gm < g.total_mtiles;
        const int64_t b = v ? gm / g.mt_per_img : 0;
        const int mt = v ? (int)(gm % g.mt_per_img) : 0;
        const int pos = min(mt * 16 + c, g.HoWo - 1);  // rows past the image are computed, not stored
        const int y = pos / g.Wo, x = pos % g.Wo;
        abase[i] = ((int64_t)b * g.Cin * g.Hp + y) * g.Wp + x;
        img[i] = v ? b : -1;
        mpos0[i] = mt * 16 + gq * 4;
    }

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

    const int4 *ko4 = reinterpret_cast<const int4 *>(koff);
    const int64_t HoWo = g.HoWo;
    const int t_begin = g.inf_mode ? g.T - 1 : 0;

    for (int tb0 = t_begin; tb0 < g.T; tb0 += TB) {
        f4 acc[MW][NW][TB];
#pragma unroll
        for (int i = 0; i < MW; ++i)
#pragma unroll
            for (int n = 0; n < NW; ++n)
#pragma unroll
                for (int t = 0; t < TB; ++t) acc[i][n][t] = f4{0.f, 0.f, 0.f, 0.f};

        for (int ks = 0; ks < g.ksteps; ++ks) {
            const int4 k0 = ko4[ks * 8 + gq * 2], k1 = ko4[ks * 8 + gq * 2 + 1];
            uint32_t tpp[MW][4];
#pragma unroll
            for (int i = 0; i < MW; ++i) {
                const uint8_t *p = tpad + abase[i];
                tpp[i][0] = (uint32_t)p[k0.x] | ((uint32_t)p[k0.y] << 16);
                tpp[i][1] = (uint32_t)p[k0.z] | ((uint32_t)p[k0.w] << 16);
                tpp[i][2] = (uint32_t)p[k1.x] | ((uint32_t)p[k1.y] << 16);
                tpp[i][3] = (uint32_t)p[k1.z] | ((uint32_t)p[k1.w] << 16);
            }
            half8 bh[NW], bl[NW];
#pragma unroll
            for (int n = 0; n < NW; ++n) {
                const int64_t fi = ((int64_t)(ng * NW + n) * g.ksteps + ks) * 64 + lane;
                bh[n] = whi[fi];
                bl[n] = wlo[fi];
            }
#pragma unroll
            for (int t = 0; t < TB; ++t) {
                if (tb0 + t < g.T) {
                    // 16-bit lanes: (0x4000 + t - tp) has bit 14 set iff tp <= t
                    // (no borrow crosses the halves since 0x4000 > 255).
                    const uint32_t cst = (0x4000u + (uint32_t)(tb0 + t)) * 0x10001u;
#pragma unroll
                    for (int i = 0; i < MW; ++i) {
                        u4 a;
                        a.x = (cst - tpp[i][0]) & 0x40004000u;
                        a.y = (cst - tpp[i][1]) & 0x40004000u;
                        a.z = (cst - tpp[i][2]) & 0x40004000u;
                        a.w = (cst - tpp[i][3]) & 0x40004000u;
                        const half8 ah = __builtin_bit_cast(half8, a);
#pragma unroll
                        for (int n = 0; n < NW; ++n) {
                            acc[i][n][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bh[n], acc[i][n][t], 0, 0, 0);
                            acc[i][n][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bl[n], acc[i][n][t], 0, 0, 0);
                        }
                    }
                }
            }
        }

        // epilogue: potentials, spikes, first-spike tracking for this time block
#pragma unroll
        for (int t = 0; t < TB; ++t) {
            const int tt = tb0 + t;
            if (tt >= g.T) continue;
#pragma unroll
            for (int i = 0; i < MW; ++i) {
                if (img[i] < 0) continue;
                const int p0 = mpos0[i];
#pragma unroll
                for (int n = 0; n < NW; ++n) {
                    const int f = (ng * NW + n) * 16 + c;
                    const f4 v = acc[i][n][t] * 0.5f;  // spikes entered as 2.0
                    uint32_t sp = 0;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const bool s = g.inf_mode ? (v[j] > 0.0f) : (v[j] >= g.thr);
                        sp |= (uint32_t)s << (8 * j);
                        if (s && tfirst[i][n][j] == g.T) {
                            tfirst[i][n][j] = tt;
                            vfirst[i][n][j] = v[j];
                        }
                    }
                    if (f >= g.Cout) continue;
                    const int64_t o = ((img[i] * g.T + tt) * (int64_t)g.Cout + f) * HoWo + p0;
                    if (g.vec4) {
                        if (p0 < g.HoWo) {
                            if (P) *reinterpret_cast<f4 *>(P + o) = v;
                            if (S) *reinterpret_cast<uint32_t *>(S + o) = sp;
                        }
                    } else {
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            if (p0 + j < g.HoWo) {
                                if (P) P[o + j] = v[j];
                                if (S) S[o + j] = (uint8_t)(sp >> (8 * j));
                            }
                    }
                }
            }
        }
    }

    // Eq.5 mode: every step before the last holds zero potential and no spike.
    if (g.inf_mode) {
        for (int tt = 0; tt < g.T - 1; ++tt) {
#pragma unroll
            for (int i = 0; i < MW; ++i) {
                if (img[i] < 0) continue;
                const int p0 = mpos0[i];
#pragma unroll
                for (int n = 0; n < NW; ++n) {
                    const int f = (ng * NW + n) * 16 + c;
                    if (f >= g.Cout) continue;
                    const int64_t o = ((img[i] * g.T + tt) * (int64_t)g.Cout + f) * HoWo + p0;
                    if (g.vec4) {
                        if (p0 < g.HoWo) {
                            if (P) *reinterpret_cast<f4 *>(P + o) = f4{0.f, 0.f, 0.f, 0.f};
                            if (S) *reinterpret_cast<uint32_t *>(S + o) = 0u;
                        }
                    } else {
                        for (int j = 0; j < 4; ++j)
                            if (p0 + j < g.HoWo) {
                                if (P) P[o + j] = 0.0f;
                                if (S) S[o + j] = 0;
                            }
                    }
                }
            }
        }
    }

    // first-spike time and the potential there
#pragma unroll
    for (int i = 0; i < MW; ++i) {
        if (img[i] < 0) continue;
        const int p0 = mpos0[i];
#pragma unroll
        for (int n = 0; n < NW; ++n) {
            const int f = (ng * NW + n) * 16 + c;
            if (f >= g.Cout) continue;
            const int64_t o = (img[i] * (int64_t)g.Cout + f) * HoWo + p0;
            if (g.vec4) {
                if (p0 < g.HoWo) {
                    uint32_t tv = 0;
#pragma unroll
                    for (int j = 0; j < 4; ++j) tv |= (uint32_t)tfirst[i][n][j] << (8 * j);
                    *reinterpret_cast<uint32_t *>(TF + o) = tv;
                    *reinterpret_cast<f4 *>(VF + o) =
                        f4{vfirst[i][n][0], vfirst[i][n][1], vfirst[i][n][2], vfirst[i][n][3]};
                }
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (p0 + j < g.HoWo) {
                        TF[o + j] = (uint8_t)tfirst[i][n][j];
                        VF[o + j] = vfirst[i][n][j];
                    }
            }
        }
    }
}

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
    SPK_REQUIRE((int64_t)Cin * K * K <= 65536, SPK_E_RANGE, "spk_conv_fire: Cin*K*K=%lld > 65536",
                (long long)Cin * K * K);
    SPK_REQUIRE((int64_t)g.Ho * g.Wo < (1LL << 31) && (int64_t)Cin * g.Hp * g.Wp < (1LL << 31),
                SPK_E_RANGE, "spk_conv_fire: image too large");
    g.HoWo = g.Ho * g.Wo;
    g.Kc = Cin * K * K;
    g.ksteps = (g.Kc + 31) / 32;
    g.ntiles = (int)spk::ceil_div(spk::ceil_div(Cout, 16), NW) * NW;
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
    return spk::align_up(c.off, 256);
}

template <int MW, int TB>
void launch_conv(const uint8_t *tpad, const half8 *whi, const half8 *wlo, const int *koff, const ConvGeom &g,
                 float *P, uint8_t *S, uint8_t *TF, float *VF, hipStream_t st) {
    const int64_t n_mgroups = spk::ceil_div(g.total_mtiles, MW);
    const int64_t n_mblocks = spk::ceil_div(n_mgroups, WAVES);
    const int64_t n_ngroups = g.ntiles / NW;
    const int64_t grid = n_mblocks * n_ngroups;
    hipLaunchKernelGGL((k_conv_fire<MW, TB>), dim3((unsigned)grid), dim3(256), 0, st, tpad, whi, wlo, koff, g,
                       (int)n_mgroups, (int)n_mblocks, P, S, TF, VF);
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
    hipStream_t st = spk::as_stream(stream);

    const int64_t n1 = (int64_t)pl.tpad_bytes;
    hipLaunchKernelGGL(k_pad_first_spike, dim3((unsigned)spk::ceil_div(n1, 256)), dim3(256), 0, st, wave, g, tpad);
    const int64_t n2 = std::max<int64_t>((int64_t)pl.frag_count, (int64_t)pl.koff_count);
    hipLaunchKernelGGL(k_split_weights, dim3((unsigned)spk::ceil_div(n2, 256)), dim3(256), 0, st, weight, g, whi,
                       wlo, koff);
    if (g.inf_mode)
        launch_conv<4, 1>(tpad, whi, wlo, koff, g, potentials, spikes, t_first, v_first, st);
    else if (spk::ceil_div(T, 16) * 16 - T < spk::ceil_div(T, 15) * 15 - T)
        launch_conv<1, 16>(tpad, whi, wlo, koff, g, potentials, spikes, t_first, v_first, st);
    else
        launch_conv<1, 15>(tpad, whi, wlo, koff, g, potentials, spikes, t_first, v_first, st);
    return spk::check_launch("spk_conv_fire");
}
