// Synaptic-event count of a convolution (gfx950): the number of (spiking
// pre-synaptic neuron, post-synaptic neuron) pairs, each counted once over
// the whole simulation.  With one spike per neuron and cumulative waves, an
// input neuron spikes at some step exactly when its entry at the last step
// is 1, so for output position (b, y, x) the pairs are Cout times the
// number of in-bounds taps of its receptive field (the padded window at
// (y*stride, x*stride)) whose last-step entry is 1.
#include "common.hpp"

namespace {

__global__ __launch_bounds__(256) void k_count_events(const uint8_t *__restrict__ wave, int64_t B, int T, int Cin,
                                                      int H, int W, int Cout, int K, int stride, int pad, int Ho,
                                                      int Wo,
                                                      unsigned long long *__restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    unsigned long long c = 0;
    if (i < B * Ho * Wo) {
        const int x = (int)(i % Wo), y = (int)((i / Wo) % Ho);
        const int64_t b = i / ((int64_t)Ho * Wo);
        const uint8_t *last = wave + (b * T + (T - 1)) * (int64_t)Cin * H * W;
        for (int ci = 0; ci < Cin; ++ci)
            for (int ky = 0; ky < K; ++ky) {
                const int iy = y * stride + ky - pad;
                if (iy < 0 || iy >= H) continue;
                for (int kx = 0; kx < K; ++kx) {
                    const int ix = x * stride + kx - pad;
                    if (ix >= 0 && ix < W) c += last[((int64_t)ci * H + iy) * W + ix] != 0;
                }
            }
    }
    for (int s = 32; s >= 1; s >>= 1) c += __shfl_xor(c, s, 64);
    if ((threadIdx.x & 63) == 0 && c) atomicAdd(out, c * (unsigned long long)Cout);
}

__global__ void k_zero_u64(unsigned long long *p) { *p = 0; }

}  // namespace

namespace {
int count_events(const uint8_t *wave, int B, int T, int Cin, int H, int W, int Cout, int K, int stride, int pad,
                 uint64_t *count, void *stream, const char *name) {
    SPK_REQUIRE(B >= 0 && T >= 1 && Cin >= 1 && H >= 1 && W >= 1 && Cout >= 1 && K >= 1 && pad >= 0 && stride >= 1,
                SPK_E_SHAPE, "%s: bad sizes", name);
    SPK_REQUIRE(T <= 255, SPK_E_RANGE, "%s: T=%d > 255", name, T);
    SPK_REQUIRE(H + 2 * pad >= K && W + 2 * pad >= K, SPK_E_SHAPE, "%s: kernel larger than the padded input", name);
    const int Ho = (H + 2 * pad - K) / stride + 1, Wo = (W + 2 * pad - K) / stride + 1;
    SPK_REQUIRE(count && (wave || B == 0), SPK_E_ARG, "%s: wave and count are required", name);
    hipStream_t st = spk::as_stream(stream);
    auto *out = reinterpret_cast<unsigned long long *>(count);
    hipLaunchKernelGGL(k_zero_u64, dim3(1), dim3(1), 0, st, out);
    const int64_t n = (int64_t)B * Ho * Wo;
    if (n > 0)
        hipLaunchKernelGGL(k_count_events, dim3((unsigned)spk::ceil_div(n, 256)), dim3(256), 0, st, wave, (int64_t)B,
                           T, Cin, H, W, Cout, K, stride, pad, Ho, Wo, out);
    return spk::check_launch(name);
}
}  // namespace

extern "C" int spk_count_events(const uint8_t *wave, int B, int T, int Cin, int H, int W, int Cout, int K, int pad,
                                uint64_t *count, void *stream) {
    return count_events(wave, B, T, Cin, H, W, Cout, K, 1, pad, count, stream, "spk_count_events");
}

extern "C" int spk_count_events_strided(const uint8_t *wave, int B, int T, int Cin, int H, int W, int Cout, int K,
                                        int stride, int pad, uint64_t *count, void *stream) {
    return count_events(wave, B, T, Cin, H, W, Cout, K, stride, pad, count, stream, "spk_count_events_strided");
}
