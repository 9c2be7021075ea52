// Spike max-pooling (gfx950).
//
// Paper: section "snn Module" (snn.Pooling / sf.pooling on spike waves: the
// output holds the earliest spike of each window; stride defaults to the
// window; zero padding) and Eq.3 for the output size, read as
// floor((H + 2D - P)/R) + 1 (equal to the printed form whenever P == R).
//
// One thread per output neuron (b, c, yo, xo) of the wave form: for every
// step t it ORs the window's bytes of plane t and stores one byte, so a wave
// reads and writes consecutive x positions of one plane; the first-spike map
// is T minus the number of steps at which the pooled neuron is on.
#include <cstdint>

#include "common.hpp"

namespace {

// Grid: (image, chunk of 256 of the image's C*Ho*Wo outputs).
__global__ __launch_bounds__(256) void k_pool(const uint8_t *__restrict__ in, int T, int C, int H, int W, int P, int R,
                                              int D, int Ho, int Wo, uint8_t *__restrict__ out,
                                              uint8_t *__restrict__ out_tf) {
    const int per_img = C * Ho * Wo;
    const int i = blockIdx.y * 256 + threadIdx.x;
    if (i >= per_img) return;
    const int64_t b = blockIdx.x;
    const int hw = Ho * Wo;
    const int c = i / hw, pix = i - c * hw;
    const int yo = pix / Wo, xo = pix - yo * Wo;
    const int y0 = yo * R - D, x0 = xo * R - D;
    const int ya = max(y0, 0), yb = min(y0 + P, H), xa = max(x0, 0), xb = min(x0 + P, W);
    const int64_t in_plane = (int64_t)C * H * W, out_plane = (int64_t)per_img;
    const uint8_t *src = in + b * T * in_plane + (int64_t)c * H * W;
    uint8_t *dst = out + b * T * out_plane + i;
    int on = 0;
    for (int t = 0; t < T; ++t) {
        const uint8_t *pl = src + t * in_plane;
        int m = 0;
        for (int y = ya; y < yb; ++y)
            for (int x = xa; x < xb; ++x) m |= pl[y * W + x];
        m = m != 0;
        dst[t * out_plane] = (uint8_t)m;
        on += m;
    }
    if (out_tf) out_tf[b * per_img + i] = (uint8_t)(T - on);
}

// Pooling of first-spike maps: the minimum over the window, then its T wave
// bytes.  Grid (image, chunk of the image's C*Ho*Wo outputs); with VEC (C*Ho*Wo
// a multiple of 4, 4-byte aligned outputs) each thread makes 4 consecutive
// outputs and stores them as one word per plane, else one output per thread.
// PW > 0 is the window size known at compile time: every window load is then
// issued before any is used.
template <bool VEC, int PW>
__global__ __launch_bounds__(256) void k_pool_first_spike(const uint8_t *__restrict__ tf, int T, int C, int H, int W,
                                                          int P, int R, int D, int Ho, int Wo,
                                                          uint8_t *__restrict__ out, uint8_t *__restrict__ out_tf) {
    constexpr int NQ = VEC ? 4 : 1;
    const int per_img = C * Ho * Wo;
    const int i0 = (blockIdx.y * 256 + threadIdx.x) * NQ;
    if (i0 >= per_img) return;
    const int64_t b = blockIdx.x;
    const int hw = Ho * Wo;
    uint32_t m4 = 0;
    // (c, yo, xo) of the first output, then stepped along x for the others
    int c = i0 / hw, yo = (i0 - c * hw) / Wo, xo = i0 - c * hw - yo * Wo;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        if (q > 0 && ++xo == Wo) {
            xo = 0;
            if (++yo == Ho) {
                yo = 0;
                ++c;
            }
        }
        const int y0 = yo * R - D, x0 = xo * R - D;
        const int ya = max(y0, 0), yb = min(y0 + P, H), xa = max(x0, 0), xb = min(x0 + P, W);
        const uint8_t *src = tf + (b * C + c) * (int64_t)H * W;
        int m = T;
        if (PW > 0) {
#pragma unroll
            for (int dy = 0; dy < PW; ++dy)
#pragma unroll
                for (int dx = 0; dx < PW; ++dx) {
                    const int y = y0 + dy, x = x0 + dx;
                    const bool in = y >= 0 && y < H && x >= 0 && x < W;
                    m = min(m, in ? (int)src[y * W + x] : T);
                }
        } else {
            for (int y = ya; y < yb; ++y)
                for (int x = xa; x < xb; ++x) m = min(m, (int)src[y * W + x]);
        }
        m4 |= (uint32_t)m << (8 * q);
    }
    if (VEC) {
        if (out_tf) *reinterpret_cast<uint32_t *>(out_tf + b * per_img + i0) = m4;
        if (out) {
            uint8_t *dst = out + b * T * (int64_t)per_img + i0;
            for (int t = 0; t < T; ++t)
                *reinterpret_cast<uint32_t *>(dst + (int64_t)t * per_img) = spk::spikes4(m4, t, T);
        }
    } else {
        const int m = (int)m4;
        if (out_tf) out_tf[b * per_img + i0] = (uint8_t)m;
        if (out) {
            uint8_t *dst = out + b * T * (int64_t)per_img + i0;
            for (int t = 0; t < T; ++t) dst[(int64_t)t * per_img] = (uint8_t)(t >= m);
        }
    }
}

// The same pooling with the input staged in LDS: a workgroup takes CB whole
// input planes of one image (contiguous in memory), copies them with
// coalesced loads, and makes their outputs 4 consecutive ones per thread, so
// the window reads hit LDS instead of scattering bytes over many cache lines.
// Needs CB * Ho * Wo % 4 == 0 (quads never straddle blocks) and 4-byte
// aligned outputs.
template <int PW>
__global__ __launch_bounds__(256) void k_pool_first_spike_lds(const uint8_t *__restrict__ tf, int T, int C, int H,
                                                              int W, int P, int R, int D, int Ho, int Wo, int CB,
                                                              uint8_t *__restrict__ out, uint8_t *__restrict__ out_tf) {
    extern __shared__ uint32_t plsm[];
    uint8_t *lt = reinterpret_cast<uint8_t *>(plsm);
    const int64_t b = blockIdx.x;
    const int c0 = blockIdx.y * CB, cb = min(CB, C - c0);
    const int HW = H * W, hw = Ho * Wo;
    const uint8_t *src = tf + (b * C + c0) * (int64_t)HW;
    const int nbytes = cb * HW;
    if ((((uintptr_t)src) & 3) == 0) {
        // a thread issues up to 16 word loads before its first LDS store (clamped
        // indices keep the loads unconditional, so none waits for the one before)
        const int nw = nbytes >> 2;
        const uint32_t *s4 = reinterpret_cast<const uint32_t *>(src);
        for (int i0 = threadIdx.x; i0 < nw; i0 += 16 * 256) {
            uint32_t v[16];
#pragma unroll
            for (int k = 0; k < 16; ++k) v[k] = s4[min(i0 + k * 256, nw - 1)];
#pragma unroll
            for (int k = 0; k < 16; ++k)
                if (i0 + k * 256 < nw) plsm[i0 + k * 256] = v[k];
        }
        for (int i = (nw << 2) + threadIdx.x; i < nbytes; i += 256) lt[i] = src[i];
    } else {
        for (int i = threadIdx.x; i < nbytes; i += 256) lt[i] = src[i];
    }
    __syncthreads();
    const int per_img = C * hw, nq = cb * hw / 4;
    for (int qd = threadIdx.x; qd < nq; qd += 256) {
        const int j0 = qd * 4;  // first output of the quad within the block
        int c = j0 / hw, yo = (j0 - c * hw) / Wo, xo = j0 - c * hw - yo * Wo;
        uint32_t m4 = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (q > 0 && ++xo == Wo) {
                xo = 0;
                if (++yo == Ho) {
                    yo = 0;
                    ++c;
                }
            }
            const int y0 = yo * R - D, x0 = xo * R - D;
            const uint8_t *pl = lt + c * HW;
            int m = T;
            if (PW > 0) {
#pragma unroll
                for (int dy = 0; dy < PW; ++dy)
#pragma unroll
                    for (int dx = 0; dx < PW; ++dx) {
                        const int y = y0 + dy, x = x0 + dx;
                        const bool in = y >= 0 && y < H && x >= 0 && x < W;
                        m = min(m, in ? (int)pl[y * W + x] : T);
                    }
            } else {
                const int ya = max(y0, 0), yb = min(y0 + P, H), xa = max(x0, 0), xb = min(x0 + P, W);
                for (int y = ya; y < yb; ++y)
                    for (int x = xa; x < xb; ++x) m = min(m, (int)pl[y * W + x]);
            }
            m4 |= (uint32_t)m << (8 * q);
        }
        const int64_t i0 = (int64_t)c0 * hw + j0;
        if (out_tf) *reinterpret_cast<uint32_t *>(out_tf + b * per_img + i0) = m4;
        if (out) {
            uint8_t *dst = out + b * T * (int64_t)per_img + i0;
            for (int t = 0; t < T; ++t)
                *reinterpret_cast<uint32_t *>(dst + (int64_t)t * per_img) = spk::spikes4(m4, t, T);
        }
    }
}

}  // namespace

extern "C" int spk_pool_first_spike(const uint8_t *t_first, int B, int T, int C, int H, int W, int kernel,
                                    int stride, int pad, uint8_t *out_wave, uint8_t *out_t_first, void *stream) {
    SPK_REQUIRE(B >= 0 && T >= 1 && C >= 1 && H >= 1 && W >= 1, SPK_E_SHAPE, "spk_pool_first_spike: bad sizes");
    SPK_REQUIRE(T <= 255, SPK_E_RANGE, "spk_pool_first_spike: T=%d > 255", T);
    SPK_REQUIRE(kernel >= 1 && stride >= 1 && pad >= 0, SPK_E_SHAPE,
                "spk_pool_first_spike: bad window %d / stride %d / pad %d", kernel, stride, pad);
    const int Ho = (H + 2 * pad - kernel) / stride + 1, Wo = (W + 2 * pad - kernel) / stride + 1;
    SPK_REQUIRE(H + 2 * pad >= kernel && W + 2 * pad >= kernel && Ho >= 1 && Wo >= 1, SPK_E_SHAPE,
                "spk_pool_first_spike: window %d larger than the padded input", kernel);
    if (B == 0) return spk::ok();
    SPK_REQUIRE(t_first && (out_wave || out_t_first), SPK_E_ARG,
                "spk_pool_first_spike: t_first and an output are required");
    const int64_t per_img = (int64_t)C * Ho * Wo;
    SPK_REQUIRE(per_img <= 65535LL * 256 && (int64_t)C * H * W < (1LL << 31), SPK_E_RANGE,
                "spk_pool_first_spike: image too large");
    const bool vec = per_img % 4 == 0 && ((uintptr_t)out_wave & 3) == 0 && ((uintptr_t)out_t_first & 3) == 0;
    hipStream_t st = spk::as_stream(stream);
    // LDS-staged form: blocks of whole input planes (up to 16 KB), quads within a block
    const int64_t HW = (int64_t)H * W, hw = (int64_t)Ho * Wo;
    if (vec && HW <= 16384) {
        // about 1024 outputs (4 per thread) per workgroup, at most 16 KB of planes
        int CB = (int)std::min<int64_t>(std::min<int64_t>(C, 16384 / HW), std::max<int64_t>(1, (1024 + hw - 1) / hw));
        while (CB > 1 && (CB * hw) % 4 != 0) --CB;
        if ((CB * hw) % 4 == 0 && (C % CB == 0 || ((int64_t)(C % CB) * hw) % 4 == 0)) {
            const dim3 g2((unsigned)B, (unsigned)spk::ceil_div(C, CB));
            const size_t lds = spk::align_up((size_t)CB * HW, 4);
#define SPK_POOL_LDS(PW)                                                                                          \
    hipLaunchKernelGGL((k_pool_first_spike_lds<PW>), g2, dim3(256), lds, st, t_first, T, C, H, W, kernel, stride, pad, \
                       Ho, Wo, CB, out_wave, out_t_first)
            if (kernel == 2) SPK_POOL_LDS(2);
            else if (kernel == 3) SPK_POOL_LDS(3);
            else SPK_POOL_LDS(0);
#undef SPK_POOL_LDS
            return spk::check_launch("spk_pool_first_spike");
        }
    }
    const dim3 grid((unsigned)B, (unsigned)spk::ceil_div(per_img, vec ? 1024 : 256));
#define SPK_POOL(V, PW)                                                                                            \
    hipLaunchKernelGGL((k_pool_first_spike<V, PW>), grid, dim3(256), 0, st, t_first, T, C, H, W, kernel, stride, pad, \
                       Ho, Wo, out_wave, out_t_first)
    if (vec && kernel == 2) SPK_POOL(true, 2);
    else if (vec && kernel == 3) SPK_POOL(true, 3);
    else if (vec) SPK_POOL(true, 0);
    else SPK_POOL(false, 0);
#undef SPK_POOL
    return spk::check_launch("spk_pool_first_spike");
}

extern "C" int spk_pool(const uint8_t *wave, int B, int T, int C, int H, int W, int kernel, int stride, int pad,
                        uint8_t *out_wave, uint8_t *out_t_first, void *stream) {
    SPK_REQUIRE(B >= 0 && T >= 1 && C >= 1 && H >= 1 && W >= 1, SPK_E_SHAPE, "spk_pool: bad sizes");
    SPK_REQUIRE(T <= 255, SPK_E_RANGE, "spk_pool: T=%d > 255", T);
    SPK_REQUIRE(kernel >= 1 && stride >= 1 && pad >= 0, SPK_E_SHAPE,
                "spk_pool: bad window %d / stride %d / pad %d", kernel, stride, pad);
    const int Ho = (H + 2 * pad - kernel) / stride + 1, Wo = (W + 2 * pad - kernel) / stride + 1;
    SPK_REQUIRE(H + 2 * pad >= kernel && W + 2 * pad >= kernel && Ho >= 1 && Wo >= 1, SPK_E_SHAPE,
                "spk_pool: window %d larger than the padded input", kernel);
    if (B == 0) return spk::ok();
    SPK_REQUIRE(wave && out_wave, SPK_E_ARG, "spk_pool: wave and out_wave are required");
    const int64_t per_img = (int64_t)C * Ho * Wo;
    SPK_REQUIRE(per_img <= 65535LL * 256 && (int64_t)C * H * W < (1LL << 31), SPK_E_RANGE, "spk_pool: image too large");
    hipLaunchKernelGGL(k_pool, dim3((unsigned)B, (unsigned)spk::ceil_div(per_img, 256)), dim3(256), 0,
                       spk::as_stream(stream), wave, T, C, H, W, kernel, stride, pad, Ho, Wo, out_wave, out_t_first);
    return spk::check_launch("spk_pool");
}
