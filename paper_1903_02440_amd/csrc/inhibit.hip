// Pointwise inhibition and pooling of potentials (gfx950).
//
// Paper: section "functional Module" (pointwise inhibition: at each location
// only the neuron of the most salient feature -- the earliest spike, then the
// highest potential -- may spike) and section "snn Module" (pooling applied
// to a potentials tensor keeps the largest potential of each window).
#include "common.hpp"

namespace {

// One thread per location of one image: the winner over the C features (the
// kWTA order: earlier spike, then larger potential, then lower feature index),
// then every feature's surviving first-spike time and potential, and, when
// asked, the survivors' Eq.1 wave and the masked potentials.  All C features
// of the location are read before any is written, so the first-spike outputs
// may alias the inputs.  Consecutive threads take consecutive locations, so
// every per-feature access of a wave is contiguous.
__global__ __launch_bounds__(256) void k_pointwise(const uint8_t *tf, const float *vf, int64_t B, int T, int C,
                                                   int64_t HW, uint8_t *out_t, float *out_v, uint8_t *wave,
                                                   float *pot) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= B * HW) return;
    const int64_t b = q / HW, p = q - b * HW;
    const int64_t base = b * C * HW + p;
    int best = -1, bt = T;
    float bv = 0.0f;
    for (int c = 0; c < C; ++c) {
        const int t = tf[base + c * HW];
        if (t >= T) continue;
        const float v = vf[base + c * HW];
        if (best < 0 || t < bt || (t == bt && v > bv)) {
            best = c;
            bt = t;
            bv = v;
        }
    }
    for (int c = 0; c < C; ++c) {
        const bool keep = c == best;
        out_t[base + c * HW] = keep ? (uint8_t)bt : (uint8_t)T;
        out_v[base + c * HW] = keep ? bv : 0.0f;
    }
    const int64_t plane = (int64_t)C * HW;
    if (wave)
        for (int t = 0; t < T; ++t) {
            uint8_t *w = wave + (b * T + t) * plane + p;
            for (int c = 0; c < C; ++c) w[c * HW] = (uint8_t)(c == best && t >= bt);
        }
    if (pot)
        for (int t = 0; t < T; ++t) {
            float *pp = pot + (b * T + t) * plane + p;
            for (int c = 0; c < C; ++c)
                if (c != best) pp[c * HW] = 0.0f;
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
    hipLaunchKernelGGL(k_pointwise, dim3((unsigned)spk::ceil_div(total, 256)), dim3(256), 0, spk::as_stream(stream),
                       t_first, v_first, (int64_t)B, T, C, HW, out_t_first, out_v_first, out_wave, potentials);
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
    hipLaunchKernelGGL(k_pool_potentials, dim3((unsigned)spk::ceil_div(total, 256)), dim3(256), 0,
                       spk::as_stream(stream), potentials, total, H, W, kernel, stride, pad, Ho, Wo, out);
    return spk::check_launch("spk_pool_potentials");
}
