// STDP / R-STDP on the winners' receptive-field weights, and the decision /
// reward step (gfx950).
//
// Paper: Eq.4 (multiplicative STDP with the stabilizer (W-LB)(UB-W)),
// section "snn Module" (R-STDP from two STDP objects) and the tutorial
// (anti-STDP negates the learning rates; reward when the decision matches
// the label, punish otherwise, nothing for a silent sample).
//
// Batch semantics (the paper leaves batch plasticity open): frozen forward,
// ordered replay.  A workgroup owns one output feature f and 256 of its
// weights, so no two threads touch the same weight.  It gathers, in image
// order, the images whose winners include f (one image has at most one
// winner per feature).  Every thread then first fetches, with independent
// loads, the pre-synaptic bit of each update for its weight (T_j <= T_i is
// one byte of the cumulative input wave at step t_i) into its column of an
// LDS bit array, and only then replays the chain of updates on its weight.  The arithmetic is double precision in the order
//     d = (w-lb)*(ub-w); u = a*d; w = w+u; clamp; round to float
// so that every update is the exactly rounded value of that expression.
#include "common.hpp"

namespace {

constexpr int CHUNK = 1024;  // images scanned per pass (4 per thread)

struct StdpArgs {
    int Cout, Cin, K, pad, B, T, H, W, k, stabilizer;
    float a_plus, a_minus, lb, ub;
};

// Grid: (feature f, chunk of 256 of its Cin*K*K weights).  Each thread owns
// one weight and replays the feature's update list on it in image order.
__global__ __launch_bounds__(256) void k_stdp(float *__restrict__ weight, const uint8_t *__restrict__ pre,
                                              const int32_t *__restrict__ winners, const int32_t *__restrict__ n_win,
                                              const int8_t *__restrict__ reward, StdpArgs a) {
#pragma clang fp contract(off)
    __shared__ int4 upd[CHUNK];   // (image, t, y, x)
    __shared__ int usg[CHUNK];    // +1 / -1
    __shared__ uint32_t bits[CHUNK / 32][256];  // pre-synaptic bits: word u/32 of thread tid
    __shared__ int scan[256];
    __shared__ int total;
    const int f = blockIdx.x, tid = threadIdx.x;
    const int KK = a.K * a.K, Kc = a.Cin * KK;
    const int e = blockIdx.y * 256 + tid;
    const bool own = e < Kc;
    const int ci = own ? e / KK : 0, ky = own ? (e % KK) / a.K : 0, kx = own ? e % a.K : 0;
    const int64_t plane = (int64_t)a.Cin * a.H * a.W;
    const int64_t cioff = (int64_t)ci * a.H * a.W;
    const double dlb = a.lb, dub = a.ub, dap = a.a_plus, dam = a.a_minus;
    float wf = own ? weight[(int64_t)f * Kc + e] : 0.0f;

    for (int b0 = 0; b0 < a.B; b0 += CHUNK) {
        int slot[4], sg[4], mine = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            slot[j] = -1;
            sg[j] = 1;
            const int b = b0 + tid * 4 + j;
            if (b >= a.B) continue;
            if (reward) {
                if (reward[b] == 0) continue;
                sg[j] = reward[b] > 0 ? 1 : -1;
            }
            const int nw = min(n_win[b], a.k);
            const int32_t *wb = winners + (int64_t)b * a.k * 4;
            // every record is read (no early exit), so the loads overlap
            for (int w = 0; w < a.k; ++w) {
                const int fw = wb[4 * w], t = wb[4 * w + 1];
                if (w < nw && fw == f && slot[j] < 0 && t >= 0 && t < a.T) slot[j] = w;
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
                const int32_t *o = winners + ((int64_t)b * a.k + slot[j]) * 4;
                upd[off] = make_int4(b, o[1], o[2], o[3]);
                usg[off] = sg[j];
                ++off;
            }
        __syncthreads();
        const int n = total;
        if (own && n > 0) {
            // phase 1: the pre-synaptic bit of every update (the input wave at
            // the winner's step, 0 in the padding).  The 32 loads of a word are
            // unconditional (a masked-off one reads the wave's first byte), so
            // they are all in flight before the first is used.
            for (int u0 = 0; u0 < n; u0 += 32) {
                uint8_t v[32];
                uint32_t ok = 0;
#pragma unroll
                for (int q = 0; q < 32; ++q) {
                    const int4 qq = upd[min(u0 + q, n - 1)];
                    const int iy = qq.z + ky - a.pad, ix = qq.w + kx - a.pad;
                    const bool in = u0 + q < n && iy >= 0 && iy < a.H && ix >= 0 && ix < a.W;
                    const int64_t at = ((int64_t)qq.x * a.T + qq.y) * plane + cioff + (int64_t)iy * a.W + ix;
                    v[q] = pre[in ? at : 0];
                    ok |= (uint32_t)in << q;
                }
                uint32_t word = 0;
#pragma unroll
                for (int q = 0; q < 32; ++q) word |= (uint32_t)(v[q] != 0) << q;
                bits[u0 >> 5][tid] = word & ok;
            }
            // phase 2: the ordered chain of updates on this weight
            for (int u0 = 0; u0 < n; u0 += 32) {
                const uint32_t word = bits[u0 >> 5][tid];
                const int cnt = min(32, n - u0);
                for (int q = 0; q < cnt; ++q) {
                    const double r = (double)usg[u0 + q] * (((word >> q) & 1u) ? dap : dam);
                    const double w = (double)wf;
                    const double d = a.stabilizer ? (w - dlb) * (dub - w) : 1.0;
                    const double du = r * d;
                    double nw = w + du;
                    if (nw < dlb) nw = dlb;
                    if (nw > dub) nw = dub;
                    wf = (float)nw;
                }
            }
        }
        __syncthreads();
    }
    if (own) weight[(int64_t)f * Kc + e] = wf;
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
    StdpArgs a{Cout, Cin, K, pad, B, T, H, W, k, stabilizer, a_plus, a_minus, lb, ub};
    const int64_t chunks = spk::ceil_div((int64_t)Cin * K * K, 256);
    SPK_REQUIRE(chunks <= 65535, SPK_E_RANGE, "%s: kernel too large", name);
    hipLaunchKernelGGL(k_stdp, dim3(Cout, (unsigned)chunks), dim3(256), 0, spk::as_stream(stream), weight, pre_wave,
                       winners, n_winners, reward, a);
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
