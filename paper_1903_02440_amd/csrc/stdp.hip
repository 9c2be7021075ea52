// STDP / R-STDP on the winners' receptive-field weights, and the decision /
// reward step (gfx950).
//
// Paper: Eq.4 (multiplicative STDP with the stabilizer (W-LB)(UB-W)),
// section "snn Module" (R-STDP from two STDP objects) and the tutorial
// (anti-STDP negates the learning rates; reward when the decision matches
// the label, punish otherwise, nothing for a silent sample).
//
// Batch semantics (the paper leaves batch plasticity open): frozen forward,
// ordered replay.  One workgroup owns one output feature f, so no two
// workgroups touch the same weight.  It gathers, in image order, the images
// whose winners include f (one image has at most one winner per feature),
// then every thread replays that list on the weights it owns.  The
// pre-synaptic condition T_j <= T_i is one byte of the cumulative input
// wave at step t_i.  The arithmetic is double precision in the order
//     d = (w-lb)*(ub-w); u = a*d; w = w+u; clamp; round to float
// so that every update is the exactly rounded value of that expression.
#include "common.hpp"

namespace {

constexpr int CHUNK = 1024;  // images scanned per pass (4 per thread)

__global__ __launch_bounds__(256) void k_stdp(float *__restrict__ weight, int Cout, int Cin, int K, int pad,
                                              const uint8_t *__restrict__ pre, int B, int T, int H, int W,
                                              const int32_t *__restrict__ winners, const int32_t *__restrict__ n_win,
                                              int k, const int8_t *__restrict__ reward, float a_plus, float a_minus,
                                              float lb, float ub, int stabilizer) {
#pragma clang fp contract(off)
    __shared__ int4 upd[CHUNK];   // (image, t, y, x)
    __shared__ int usg[CHUNK];    // +1 / -1
    __shared__ int scan[256];
    __shared__ int total;
    const int f = blockIdx.x, tid = threadIdx.x;
    const int KK = K * K, Kc = Cin * KK;
    const int64_t plane = (int64_t)Cin * H * W;
    const double dlb = lb, dub = ub, dap = a_plus, dam = a_minus;

    for (int b0 = 0; b0 < B; b0 += CHUNK) {
        int slot[4], sg[4], mine = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            slot[j] = -1;
            sg[j] = 1;
            const int b = b0 + tid * 4 + j;
            if (b >= B) continue;
            if (reward) {
                if (reward[b] == 0) continue;
                sg[j] = reward[b] > 0 ? 1 : -1;
            }
            const int nw = min(n_win[b], k);
            for (int w = 0; w < nw; ++w)
                if (winners[((int64_t)b * k + w) * 4] == f) {
                    const int t = winners[((int64_t)b * k + w) * 4 + 1];
                    if (t >= 0 && t < T) slot[j] = w;
                    break;
                }
            mine += slot[j] >= 0;
        }
        // block exclusive scan of the per-thread counts keeps image order
        scan[tid] = mine;
        __syncthreads();
        for (int s = 1; s < 256; s <<= 1) {
            const int v = tid >= s ? scan[tid - s] : 0;
            __syncthreads();
            scan[tid] += v;
            __syncthreads();
        }
        int off = scan[tid] - mine;
        if (tid == 255) total = scan[255];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (slot[j] >= 0) {
                const int b = b0 + tid * 4 + j;
                const int32_t *o = winners + ((int64_t)b * k + slot[j]) * 4;
                upd[off] = make_int4(b, o[1], o[2], o[3]);
                usg[off] = sg[j];
                ++off;
            }
        __syncthreads();
        const int n = total;
        for (int e = tid; e < Kc && n > 0; e += 256) {
            const int ci = e / KK, ky = (e % KK) / K, kx = e % K;
            float *wp = weight + (int64_t)f * Kc + e;
            float wf = *wp;
            for (int u = 0; u < n; ++u) {
                const int4 q = upd[u];
                const int iy = q.z + ky - pad, ix = q.w + kx - pad;
                bool on = false;
                if (iy >= 0 && iy < H && ix >= 0 && ix < W)
                    on = pre[((int64_t)q.x * T + q.y) * plane + ((int64_t)ci * H + iy) * W + ix] != 0;
                const double a = (double)usg[u] * (on ? dap : dam);
                const double w = (double)wf;
                const double d = stabilizer ? (w - dlb) * (dub - w) : 1.0;
                const double du = a * d;
                double nw = w + du;
                if (nw < dlb) nw = dlb;
                if (nw > dub) nw = dub;
                wf = (float)nw;
            }
            *wp = wf;
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(256) void k_decide(const int32_t *__restrict__ winners, const int32_t *__restrict__ n_win,
                                                int B, int k, const int32_t *__restrict__ labels, int n_classes,
                                                int32_t *__restrict__ decision, int8_t *__restrict__ reward) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    if (n_win[b] <= 0) {
        decision[b] = -1;
        reward[b] = 0;
        return;
    }
    const int d = winners[(int64_t)b * k * 4] % n_classes;
    decision[b] = d;
    reward[b] = (int8_t)(d == labels[b] ? 1 : -1);
}

int stdp_common(float *weight, int Cout, int Cin, int K, int pad, const uint8_t *pre_wave, int B, int T, int H,
                int W, const int32_t *winners, const int32_t *n_winners, int k, const int8_t *reward, float a_plus,
                float a_minus, float lb, float ub, int stabilizer, void *stream, const char *name) {
    SPK_REQUIRE(Cout >= 1 && Cin >= 1 && K >= 1 && pad >= 0 && B >= 0 && T >= 1 && H >= 1 && W >= 1 && k >= 1,
                SPK_E_SHAPE, "%s: bad sizes", name);
    SPK_REQUIRE(T <= 255, SPK_E_RANGE, "%s: T=%d > 255", name, T);
    SPK_REQUIRE((int64_t)Cin * K * K < (1LL << 31), SPK_E_RANGE, "%s: kernel too large", name);
    SPK_REQUIRE(std::isfinite(a_plus) && std::isfinite(a_minus) && std::isfinite(lb) && std::isfinite(ub) && lb <= ub,
                SPK_E_ARG, "%s: rates and bounds must be finite with lb <= ub", name);
    SPK_REQUIRE(stabilizer == 0 || stabilizer == 1, SPK_E_ARG, "%s: stabilizer must be 0 or 1", name);
    if (B == 0) return spk::ok();
    SPK_REQUIRE(weight && pre_wave && winners && n_winners, SPK_E_ARG,
                "%s: weight, pre_wave, winners and n_winners are required", name);
    hipLaunchKernelGGL(k_stdp, dim3(Cout), dim3(256), 0, spk::as_stream(stream), weight, Cout, Cin, K, pad, pre_wave,
                       B, T, H, W, winners, n_winners, k, reward, a_plus, a_minus, lb, ub, stabilizer);
    return spk::check_launch(name);
}

}  // namespace

extern "C" int spk_stdp(float *weight, int Cout, int Cin, int K, int pad, const uint8_t *pre_wave, int B, int T,
                        int H, int W, const int32_t *winners, const int32_t *n_winners, int k, float a_plus,
                        float a_minus, float lb, float ub, int stabilizer, void *stream) {
    return stdp_common(weight, Cout, Cin, K, pad, pre_wave, B, T, H, W, winners, n_winners, k, nullptr, a_plus,
                       a_minus, lb, ub, stabilizer, stream, "spk_stdp");
}

extern "C" int spk_rstdp(float *weight, int Cout, int Cin, int K, int pad, const uint8_t *pre_wave, int B, int T,
                         int H, int W, const int32_t *winners, const int32_t *n_winners, int k, const int8_t *reward,
                         float a_plus, float a_minus, float lb, float ub, int stabilizer, void *stream) {
    SPK_REQUIRE(reward || B == 0, SPK_E_ARG, "spk_rstdp: reward is required");
    return stdp_common(weight, Cout, Cin, K, pad, pre_wave, B, T, H, W, winners, n_winners, k, reward, a_plus,
                       a_minus, lb, ub, stabilizer, stream, "spk_rstdp");
}

extern "C" int spk_decide(const int32_t *winners, const int32_t *n_winners, int B, int k, const int32_t *labels,
                          int n_classes, int32_t *decision, int8_t *reward, void *stream) {
    SPK_REQUIRE(B >= 0 && k >= 1 && n_classes >= 1, SPK_E_SHAPE, "spk_decide: bad sizes");
    if (B == 0) return spk::ok();
    SPK_REQUIRE(winners && n_winners && labels && decision && reward, SPK_E_ARG, "spk_decide: null buffer");
    hipLaunchKernelGGL(k_decide, dim3((unsigned)spk::ceil_div(B, 256)), dim3(256), 0, spk::as_stream(stream),
                       winners, n_winners, B, k, labels, n_classes, decision, reward);
    return spk::check_launch("spk_decide");
}
