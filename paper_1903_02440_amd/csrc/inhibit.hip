// Pointwise inhibition and pooling of potentials (gfx950).
//
// Paper: section "functional Module" (pointwise inhibition: at each location
// only the neuron of the most salient feature -- the earliest spike, then the
// highest potential -- may spike) and section "snn Module" (pooling applied
// to a potentials tensor keeps the largest potential of each window).
#include "common.hpp"

namespace {

constexpr int PW_U = 8;  // features per block of loads in the pointwise inhibition

// One thread per location of one image (VEC: per 4 consecutive locations,
// with 4-byte / 16-byte accesses; the map size is then a multiple of 4): the
// winner over the C features (the kWTA order: earlier spike, then larger
// potential, then lower feature index), then every feature's surviving
// first-spike time and potential, and, when asked, the survivors' Eq.1 wave
// and the masked potentials.  All C features of the locations are read before
// any is written, so the first-spike outputs may alias the inputs.
// Consecutive threads take consecutive locations, so every per-feature
// access of a wave is contiguous.
template <bool VEC>
__global__ __launch_bounds__(256) void k_pointwise(const uint8_t *tf, const float *vf, int64_t B, int T, int C,
                                                   int64_t HW, uint8_t *out_t, float *out_v, uint8_t *wave,
                                                   float *pot) {
    constexpr int L = VEC ? 4 : 1;
    const int64_t per_img = HW / L;
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= B * per_img) return;
    const int64_t b = q / per_img, p = (q - b * per_img) * L;
    const int64_t base = b * C * HW + p;
    int best[L], bt[L];
    float bv[L];
#pragma unroll
    for (int j = 0; j < L; ++j) {
        best[j] = -1;
        bt[j] = T;
        bv[j] = 0.0f;
    }
    // features in blocks of PW_U, every load of a block issued before the
    // first is used (clamped feature indices keep them unconditional), in
    // increasing feature order so that strict comparisons keep the lower index
    for (int c0 = 0; c0 < C; c0 += PW_U) {
        uint32_t tw[PW_U];
        float4 vw[PW_U];
#pragma unroll
        for (int u = 0; u < PW_U; ++u) {
            const int64_t o = base + (int64_t)min(c0 + u, C - 1) * HW;
            if (VEC) {
                tw[u] = *reinterpret_cast<const uint32_t *>(tf + o);
                vw[u] = *reinterpret_cast<const float4 *>(vf + o);
            } else {
                tw[u] = tf[o];
                vw[u].x = vf[o];
            }
        }
#pragma unroll
        for (int u = 0; u < PW_U; ++u) {
            const int c = c0 + u;
            if (c >= C) break;
            int t[L];
            float v[L];
            t[0] = tw[u] & 255u;
            v[0] = vw[u].x;
            if (VEC) {
                t[L > 1 ? 1 : 0] = (tw[u] >> 8) & 255u;
                t[L > 2 ? 2 : 0] = (tw[u] >> 16) & 255u;
                t[L > 3 ? 3 : 0] = tw[u] >> 24;
                v[L > 1 ? 1 : 0] = vw[u].y; v[L > 2 ? 2 : 0] = vw[u].z; v[L > 3 ? 3 : 0] = vw[u].w;
            }
#pragma unroll
            for (int j = 0; j < L; ++j)
                if (t[j] < T && (best[j] < 0 || t[j] < bt[j] || (t[j] == bt[j] && v[j] > bv[j]))) {
                    best[j] = c;
                    bt[j] = t[j];
                    bv[j] = v[j];
                }
        }
    }
    // the surviving first-spike times of feature c, 4 to a word
    auto word = [&](int c) {
        uint32_t w = 0;
#pragma unroll
        for (int j = 0; j < L; ++j) w |= (uint32_t)(c == best[j] ? bt[j] : T) << (8 * j);
        return w;
    };
    for (int c = 0; c < C; ++c) {
        if (VEC) {
            *reinterpret_cast<uint32_t *>(out_t + base + c * HW) = word(c);
            *reinterpret_cast<float4 *>(out_v + base + c * HW) =
                float4{c == best[0] ? bv[0] : 0.0f, c == best[L > 1 ? 1 : 0] ? bv[L > 1 ? 1 : 0] : 0.0f,
                       c == best[L > 2 ? 2 : 0] ? bv[L > 2 ? 2 : 0] : 0.0f,
                       c == best[L > 3 ? 3 : 0] ? bv[L > 3 ? 3 : 0] : 0.0f};
        } else {
            out_t[base + c * HW] = (uint8_t)(c == best[0] ? bt[0] : T);
            out_v[base + c * HW] = c == best[0] ? bv[0] : 0.0f;
        }
    }
    const int64_t plane = (int64_t)C * HW;
    if (wave)  // feature by feature: its surviving times once, then its T steps
        for (int c = 0; c < C; ++c) {
            uint8_t *w = wave + b * T * plane + (int64_t)c * HW + p;
            if (VEC) {
                const uint32_t wc = word(c);
                for (int t = 0; t < T; ++t) *reinterpret_cast<uint32_t *>(w + t * plane) = spk::spikes4(wc, t, T);
            } else {
                const int tc = c == best[0] ? bt[0] : T;
                for (int t = 0; t < T; ++t) w[t * plane] = (uint8_t)(t >= tc);
            }
        }
    if (pot)
        for (int t = 0; t < T; ++t) {
            float *pp = pot + (b * T + t) * plane + p;
            if constexpr (VEC) {
                // blocks of PW_U features: the loads first (clamped), then the masked stores
                for (int c0 = 0; c0 < C; c0 += PW_U) {
                    float4 xw[PW_U];
#pragma unroll
                    for (int u = 0; u < PW_U; ++u)
                        xw[u] = *reinterpret_cast<const float4 *>(pp + (int64_t)min(c0 + u, C - 1) * HW);
#pragma unroll
                    for (int u = 0; u < PW_U; ++u) {
                        const int c = c0 + u;
                        if (c >= C) break;
                        if (c == best[0] && c == best[1] && c == best[2] && c == best[3])
                            continue;  // the feature survives at all four locations
                        float4 x = xw[u];
                        if (c != best[0]) x.x = 0.0f;
                        if (c != best[1]) x.y = 0.0f;
                        if (c != best[2]) x.z = 0.0f;
                        if (c != best[3]) x.w = 0.0f;
                        *reinterpret_cast<float4 *>(pp + (int64_t)c * HW) = x;
                    }
                }
            } else {
                for (int c = 0; c < C; ++c)
                    if (c != best[0]) pp[c * HW] = 0.0f;
            }
        }
}

// One thread per output value: the maximum over the window of the zero-padded
// input, taken in row-major window order keeping the first of equal values.
__global__ __launch_bounds__(256) void k_pool_potentials(const float *__restrict__ pot, int64_t total, int H, int W,
                                                         int P, int R, int D, int Ho, int Wo,
                                                         float *__restrict__ out) {
    const int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (o >= total) return;
    const int64_t pl = o / ((int64_t)Ho * Wo);
    const int r = (int)(o - pl * Ho * Wo), yo = r / Wo, xo = r - yo * Wo;
    const float *src = pot + pl * H * W;
    bool first = true;
    float m = 0.0f;
    for (int dy = 0; dy < P; ++dy)
        for (int dx = 0; dx < P; ++dx) {
            const int iy = yo * R + dy - D, ix = xo * R + dx - D;
            const float v = (iy >= 0 && iy < H && ix >= 0 && ix < W) ? src[(int64_t)iy * W + ix] : 0.0f;
            if (first || v > m) m = v;
            first = false;
        }
    out[o] = m;
}

// 2x2 windows, stride 2, no padding, W a multiple of 4, Wo even, aligned
// tensors: one thread per two adjacent outputs, from one 16-byte load of each
// of the two input rows; the same comparisons in the same window order.
__global__ __launch_bounds__(256) void k_pool_potentials_2x2(const float *__restrict__ pot, uint32_t pairs, int H,
                                                             int W, int Ho, int Wo, float *__restrict__ out) {
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= pairs) return;
    const uint32_t hw2 = (uint32_t)(Ho * Wo) / 2, wo2 = (uint32_t)Wo / 2;
    const uint32_t pl = i / hw2, r = i - pl * hw2, yo = r / wo2, x2 = r - yo * wo2;
    const float *src = pot + (size_t)pl * H * W + (size_t)(2 * yo) * W + 4 * x2;
    const float4 a = *reinterpret_cast<const float4 *>(src), c = *reinterpret_cast<const float4 *>(src + W);
    auto win = [](float v00, float v01, float v10, float v11) {
        float m = v00;
        if (v01 > m) m = v01;
        if (v10 > m) m = v10;
        if (v11 > m) m = v11;
        return m;
    };
    *reinterpret_cast<float2 *>(out + (size_t)pl * Ho * Wo + (size_t)yo * Wo + 2 * x2) =
        float2{win(a.x, a.y, c.x, c.y), win(a.z, a.w, c.z, c.w)};
}

}  // namespace

extern "C" int spk_pointwise_inhibition(const uint8_t *t_first, const float *v_first, int B, int T, int C, int H,
                                        int W, uint8_t *out_t_first, float *out_v_first, uint8_t *out_wave,
                                        float *potentials, void *stream) {
    SPK_REQUIRE(B >= 0 && T >= 1 && C >= 1 && H >= 1 && W >= 1, SPK_E_SHAPE, "spk_pointwise_inhibition: bad sizes");
    SPK_REQUIRE(T <= 255, SPK_E_RANGE, "spk_pointwise_inhibition: T=%d > 255", T);
    if (B == 0) return spk::ok();
    SPK_REQUIRE(t_first && v_first && out_t_first && out_v_first, SPK_E_ARG,
                "spk_pointwise_inhibition: t_first, v_first, out_t_first and out_v_first are required");
    const int64_t HW = (int64_t)H * W, total = (int64_t)B * HW;
    SPK_REQUIRE(spk::ceil_div(total, 256) < (1LL << 31), SPK_E_RANGE, "spk_pointwise_inhibition: too large");
    auto al = [](const void *q, uintptr_t a) { return ((uintptr_t)q & (a - 1)) == 0; };
    const bool vec = HW % 4 == 0 && al(t_first, 4) && al(out_t_first, 4) && al(out_wave, 4) && al(v_first, 16) &&
                     al(out_v_first, 16) && al(potentials, 16);
    hipStream_t st = spk::as_stream(stream);
    if (vec)
        hipLaunchKernelGGL(k_pointwise<true>, dim3((unsigned)spk::ceil_div(total / 4, 256)), dim3(256), 0, st, t_first,
                           v_first, (int64_t)B, T, C, HW, out_t_first, out_v_first, out_wave, potentials);
    else
        hipLaunchKernelGGL(k_pointwise<false>, dim3((unsigned)spk::ceil_div(total, 256)), dim3(256), 0, st, t_first,
                           v_first, (int64_t)B, T, C, HW, out_t_first, out_v_first, out_wave, potentials);
    return spk::check_launch("spk_pointwise_inhibition");
}

extern "C" int spk_pool_potentials(const float *potentials, int B, int T, int C, int H, int W, int kernel, int stride,
                                   int pad, float *out, void *stream) {
    SPK_REQUIRE(B >= 0 && T >= 1 && C >= 1 && H >= 1 && W >= 1, SPK_E_SHAPE, "spk_pool_potentials: bad sizes");
    SPK_REQUIRE(kernel >= 1 && stride >= 1 && pad >= 0, SPK_E_SHAPE,
                "spk_pool_potentials: bad window %d / stride %d / pad %d", kernel, stride, pad);
    SPK_REQUIRE(H + 2 * pad >= kernel && W + 2 * pad >= kernel, SPK_E_SHAPE,
                "spk_pool_potentials: window %d larger than the padded input", kernel);
    const int Ho = (H + 2 * pad - kernel) / stride + 1, Wo = (W + 2 * pad - kernel) / stride + 1;
    if (B == 0) return spk::ok();
    SPK_REQUIRE(potentials && out, SPK_E_ARG, "spk_pool_potentials: potentials and out are required");
    const int64_t total = (int64_t)B * T * C * Ho * Wo;
    SPK_REQUIRE(spk::ceil_div(total, 256) < (1LL << 31), SPK_E_RANGE, "spk_pool_potentials: too large");
    const bool al16 = ((uintptr_t)potentials & 15) == 0 && ((uintptr_t)out & 7) == 0;
    if (kernel == 2 && stride == 2 && pad == 0 && W % 4 == 0 && Wo % 2 == 0 && Ho == H / 2 && al16 &&
        total / 2 < (1LL << 32) && (int64_t)B * T * C * H * W < (1LL << 32)) {
        const int64_t pairs = total / 2;
        hipLaunchKernelGGL(k_pool_potentials_2x2, dim3((unsigned)spk::ceil_div(pairs, 256)), dim3(256), 0,
                           spk::as_stream(stream), potentials, (uint32_t)pairs, H, W, Ho, Wo, out);
        return spk::check_launch("spk_pool_potentials");
    }
    hipLaunchKernelGGL(k_pool_potentials, dim3((unsigned)spk::ceil_div(total, 256)), dim3(256), 0,
                       spk::as_stream(stream), potentials, total, H, W, kernel, stride, pad, Ho, Wo, out);
    return spk::check_launch("spk_pool_potentials");
}
