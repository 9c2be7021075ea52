// STDP / R-STDP on the winners' receptive-field weights, and the decision /
// reward step (gfx950).
//
// Paper: Eq.4 (multiplicative STDP with the stabilizer (W-LB)(UB-W)),
// section "snn Module" (R-STDP from two STDP objects) and the tutorial
// (anti-STDP negates the learning rates; reward when the decision matches
// the label, punish otherwise, nothing for a silent sample).
//
// Batch semantics (the paper leaves batch plasticity open): frozen forward,
// ordered replay.  Each feature f gets the list, in image order, of the
// images whose winners include f (one image has at most one winner per
// feature).  The pre-synaptic bit of every (update, weight) pair (T_j <= T_i
// is one byte of the cumulative input wave at step t_i) is gathered by a
// fully parallel pass and packed 32 updates to a word, so the serial part --
// one thread per weight replaying its feature's chain of updates in image
// order -- only reads coalesced bit words.  A feature that wins many images
// has a long chain, but its chains run on as many threads as it has weights.
// The arithmetic is double precision in the order
//     d = (w-lb)*(ub-w); u = a*d; w = w+u; clamp; round to float
// so that every update is the exactly rounded value of that expression.
#include <algorithm>
#include <cmath>

#include "common.hpp"

namespace {

constexpr int LIST_THREADS = 1024;  // images scanned per pass of the list kernel

struct StdpArgs {
    int Cout, Cin, K, pad, stride, B, T, H, W, k, stabilizer;
    int times;  // pre is the layer input's first-spike map [B][Cin][H][W] instead of its wave
    float a_plus, a_minus, lb, ub;
};

// Workspace of one call (sizes in spk_stdp_workspace_size):
//   count [Cout]           updates of each feature
//   woff  [Cout+1]         first bit row of each feature (exclusive prefix of ceil(count/32))
//   list  [Cout][B] int4   the feature's updates in image order: (image, t, y, x)
//   lsign [Cout][B] i8     +1 / -1 (STDP / anti-STDP)
//   bits  [rows][Kc] u32   bit q of row woff[f]+i, column e: pre-synaptic bit of update 32i+q on weight e
//   sbits [rows] u32       bit q of row woff[f]+i: update 32i+q is an anti-STDP one (negated rates)
struct StdpWork {
    int *count, *woff;
    int4 *list;
    int8_t *lsign;
    uint32_t *bits, *sbits;
    int64_t rows;  // capacity of bits in rows of Kc words
};

int64_t bit_rows(int Cout, int B, int k) { return ((int64_t)B * std::min(k, Cout) + 31) / 32 + Cout; }

StdpWork carve(void *ws, int Cout, int Cin, int K, int B, int k, size_t *bytes) {
    spk::Carver c(ws);
    StdpWork w;
    w.count = c.take<int>(Cout);
    w.woff = c.take<int>(Cout + 1);
    w.list = c.take<int4>((size_t)Cout * B);
    w.lsign = c.take<int8_t>((size_t)Cout * B);
    w.rows = bit_rows(Cout, B, k);
    w.bits = c.take<uint32_t>((size_t)w.rows * Cin * K * K);
    w.sbits = c.take<uint32_t>((size_t)w.rows);
    if (bytes) *bytes = spk::align_up(c.off, 256);
    return w;
}

// 1. Grid: one workgroup per feature f.  For each pass over up to 1024 images
// (one per thread) it finds the image's winner of feature f (one image has at
// most one), then a wave ballot and a scan of the 16 wave counts place the
// updates in image order.
__global__ __launch_bounds__(LIST_THREADS) void k_stdp_list(const int32_t *__restrict__ winners,
                                                            const int32_t *__restrict__ n_win,
                                                            const int8_t *__restrict__ reward, StdpArgs a, StdpWork w) {
    __shared__ int wave_cnt[LIST_THREADS / 64];
    const int f = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    int base = 0;
    for (int b0 = 0; b0 < a.B; b0 += LIST_THREADS) {
        const int b = b0 + tid;
        int slot = -1, sg = 1;
        if (b < a.B && (!reward || reward[b] != 0)) {
            if (reward) sg = reward[b] > 0 ? 1 : -1;
            const int nw = min(n_win[b], a.k);
            const int32_t *wb = winners + (int64_t)b * a.k * 4;
            for (int q = 0; q < a.k; ++q) {  // every record is read, so the loads overlap
                const int fw = wb[4 * q], t = wb[4 * q + 1];
                if (q < nw && fw == f && slot < 0 && t >= 0 && t < a.T) slot = q;
            }
        }
        const uint64_t mask = __ballot(slot >= 0);
        if (lane == 0) wave_cnt[wv] = __popcll(mask);
        __syncthreads();
        int off = base + __popcll(mask & ((1ull << lane) - 1ull)), n = 0;
        for (int q = 0; q < LIST_THREADS / 64; ++q) {
            off += q < wv ? wave_cnt[q] : 0;
            n += wave_cnt[q];
        }
        if (slot >= 0) {
            const int32_t *o = winners + ((int64_t)b * a.k + slot) * 4;
            w.list[(int64_t)f * a.B + off] = make_int4(b, o[1], o[2], o[3]);
            w.lsign[(int64_t)f * a.B + off] = (int8_t)sg;
        }
        base += n;
        __syncthreads();  // wave_cnt is rewritten by the next pass
    }
    if (tid == 0) w.count[f] = base;
}

// 2. One workgroup: woff[f] = sum over f' < f of ceil(count[f'] / 32).
__global__ __launch_bounds__(1024) void k_stdp_offsets(int Cout, StdpWork w) {
    __shared__ int part[1024];
    const int tid = threadIdx.x;
    const int per = (Cout + 1023) / 1024, f0 = tid * per;
    int sum = 0;
    for (int f = f0; f < min(Cout, f0 + per); ++f) sum += (w.count[f] + 31) / 32;
    part[tid] = sum;
    __syncthreads();
    for (int s = 1; s < 1024; s <<= 1) {
        const int v = tid >= s ? part[tid - s] : 0;
        __syncthreads();
        part[tid] += v;
        __syncthreads();
    }
    int run = part[tid] - sum;
    for (int f = f0; f < min(Cout, f0 + per); ++f) {
        w.woff[f] = run;
        run += (w.count[f] + 31) / 32;
    }
    if (tid == 1023) w.woff[Cout] = part[1023];
}

// 3. Grid (chunk of 256 weights, bit row).  Row r belongs to the feature f
// with woff[f] <= r < woff[f+1] (binary search); its thread for weight
// e = (ci, ky, kx) loads the pre-synaptic byte of each of the row's up to 32
// updates -- the layer input at (image, winner step, ci, y*s+ky-pad,
// x*s+kx-pad) for the layer's stride s, 0 in the padding -- with independent
// loads and packs the 32 bits.
__global__ __launch_bounds__(256) void k_stdp_bits(const uint8_t *__restrict__ pre, StdpArgs a, StdpWork w) {
    const int r = blockIdx.y;
    if (r >= w.woff[a.Cout]) return;  // uniform
    int lo = 0, hi = a.Cout - 1;      // the largest f with woff[f] <= r
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (w.woff[mid] <= r) lo = mid;
        else hi = mid - 1;
    }
    const int f = lo, u0 = (r - w.woff[f]) * 32, cnt = min(32, w.count[f] - u0);
    if (blockIdx.x == 0 && threadIdx.x < 64) {  // the row's sign word
        const bool neg = (int)threadIdx.x < cnt && w.lsign[(int64_t)f * a.B + u0 + threadIdx.x] < 0;
        const uint64_t m = __ballot(neg);
        if (threadIdx.x == 0) w.sbits[r] = (uint32_t)m;
    }
    // the row's updates, read once into LDS (entries past the row repeat its last)
    __shared__ int4 s_lst[32];
    if (threadIdx.x < 32) s_lst[threadIdx.x] = w.list[(int64_t)f * a.B + u0 + min((int)threadIdx.x, cnt - 1)];
    __syncthreads();
    const int KK = a.K * a.K, Kc = a.Cin * KK;
    const int e = blockIdx.x * 256 + threadIdx.x;
    if (e >= Kc) return;
    const int ci = e / KK, ky = (e % KK) / a.K, kx = e % a.K;
    const int64_t plane = (int64_t)a.Cin * a.H * a.W, cioff = (int64_t)ci * a.H * a.W;
    // two halves of 16 updates: every byte load of a half is issued before any
    // is used (updates past the row or in the padding load byte 0 of the input
    // and count 0), so that none waits behind a branch
    uint32_t word = 0;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        int64_t off[16];
        int lim[16];
        bool ok[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int q = 16 * h + j;
            const int4 u = s_lst[q];  // (cnt >= 1: the row holds an update)
            const int iy = u.z * a.stride + ky - a.pad, ix = u.w * a.stride + kx - a.pad;
            ok[j] = q < cnt && iy >= 0 && iy < a.H && ix >= 0 && ix < a.W;
            const int64_t img = a.times ? (int64_t)u.x : (int64_t)u.x * a.T + u.y;
            off[j] = ok[j] ? img * plane + cioff + (int64_t)iy * a.W + ix : 0;
            lim[j] = u.y;
        }
        uint8_t v[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) v[j] = pre[off[j]];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            // Eq.1 for a first-spike input: the wave is 1 at step t_i exactly where t_first <= t_i
            const bool bit = ok[j] && (a.times ? (int)v[j] <= lim[j] : v[j] != 0);
            word |= (uint32_t)bit << (16 * h + j);
        }
    }
    w.bits[(int64_t)r * Kc + e] = word;
}

// 4. Grid (chunk of 256 weights, feature): each thread replays its weight's
// chain of updates in image order, 32 per bit word (the next word is loaded
// while the current one is replayed).  The rates of a word's updates come from
// its pre-synaptic and sign bits, off the dependency chain, which is then
//     x = w; d = (x-lb)*(ub-x); u = r*d; w = clamp(x+u); w = float(w)
// With FAST (stabilizer on and max|rate| * (ub-lb) <= 1/2, checked by the
// host) the clamp is applied to the first update of the chain only: from then
// on lb <= x <= ub, so u >= 0 stays below 0.51*(ub-x) and u < 0 above
// -0.51*(x-lb) even after the roundings of d and u, and x+u rounds into
// [lb, ub] without it.  Clamping in double and then rounding, or rounding
// first, give the same float, since lb and ub are floats.
template <bool FAST>
__device__ __forceinline__ float stdp_one(float wf, double r, double dlb, double dub, bool stab, bool clamp) {
#pragma clang fp contract(off)
    const double x = (double)wf;
    const double d = stab ? (x - dlb) * (dub - x) : 1.0;
    const double du = r * d;
    double nw = x + du;
    if (!FAST || clamp) {
        nw = nw < dlb ? dlb : nw;
        nw = nw > dub ? dub : nw;
    }
    return (float)nw;
}

template <bool FAST>
__global__ __launch_bounds__(256) void k_stdp_apply(float *__restrict__ weight, StdpArgs a, StdpWork w) {
#pragma clang fp contract(off)
    const int f = blockIdx.y, tid = threadIdx.x;
    const int n = w.count[f];
    if (n == 0) return;  // uniform
    const int KK = a.K * a.K, Kc = a.Cin * KK;
    const int e = blockIdx.x * 256 + tid;
    const bool own = e < Kc;
    const bool stab = FAST || a.stabilizer;
    const double dlb = a.lb, dub = a.ub, dap = a.a_plus, dam = a.a_minus;
    float *wp = weight + (int64_t)f * Kc + e;
    float wf = own ? *wp : 0.0f;
    const int row0 = w.woff[f];
    const uint32_t *brow = w.bits + (int64_t)row0 * Kc + e;
    const int words = (n + 31) / 32;
    uint32_t nxt = own ? brow[0] : 0u;
    for (int wi = 0; wi < words; ++wi) {
        const uint32_t word = nxt, sw = w.sbits[row0 + wi];
        if (own && wi + 1 < words) nxt = brow[(int64_t)(wi + 1) * Kc];
        const int cnt = min(32, n - 32 * wi);
        if (FAST && wi == 0) {  // the clamped first update
            const double r0 = (word & 1u) ? dap : dam;
            wf = stdp_one<FAST>(wf, (sw & 1u) ? -r0 : r0, dlb, dub, stab, true);
        }
#pragma unroll
        for (int q = 0; q < 32; ++q) {
            if (FAST && q == 0 && wi == 0) continue;
            if (q >= cnt) break;  // uniform
            const double rq = ((word >> q) & 1u) ? dap : dam;
            wf = stdp_one<FAST>(wf, ((sw >> q) & 1u) ? -rq : rq, dlb, dub, stab, false);
        }
    }
    if (own) *wp = wf;
}

// B == 1 (online steps): grid (chunk of 256 weights, winner slot).  Each
// winner updates its feature's weights directly -- the replay's chain of one
// update, with the record rules of k_stdp_list (the first record of a feature
// whose step lies in [0, T); nothing for reward 0) -- without the list,
// offset and bit passes.
template <bool FAST>
__global__ __launch_bounds__(256) void k_stdp_single(float *__restrict__ weight, const uint8_t *__restrict__ pre,
                                                     const int32_t *__restrict__ winners,
                                                     const int32_t *__restrict__ n_win,
                                                     const int8_t *__restrict__ reward, StdpArgs a) {
#pragma clang fp contract(off)
    const int j = blockIdx.y;
    if (j >= min(n_win[0], a.k) || (reward && reward[0] == 0)) return;  // uniform
    auto valid = [&](int q) { return winners[4 * q + 1] >= 0 && winners[4 * q + 1] < a.T; };
    const int f = winners[4 * j], t = winners[4 * j + 1];
    if (f < 0 || f >= a.Cout || !valid(j)) return;
    for (int q = 0; q < j; ++q)
        if (winners[4 * q] == f && valid(q)) return;  // an earlier record of the feature is the one used
    const int KK = a.K * a.K, Kc = a.Cin * KK;
    const int e = blockIdx.x * 256 + threadIdx.x;
    if (e >= Kc) return;
    const int ci = e / KK, ky = (e % KK) / a.K, kx = e % a.K;
    const int iy = winners[4 * j + 2] * a.stride + ky - a.pad, ix = winners[4 * j + 3] * a.stride + kx - a.pad;
    uint8_t v = 0;
    if (iy >= 0 && iy < a.H && ix >= 0 && ix < a.W) {
        if (a.times)
            v = pre[(int64_t)ci * a.H * a.W + (int64_t)iy * a.W + ix] <= t;
        else
            v = pre[((int64_t)t * a.Cin + ci) * a.H * a.W + (int64_t)iy * a.W + ix];
    }
    double r = v != 0 ? (double)a.a_plus : (double)a.a_minus;
    if (reward && reward[0] < 0) r = -r;
    float *wp = weight + (int64_t)f * Kc + e;
    *wp = stdp_one<FAST>(*wp, r, a.lb, a.ub, FAST || a.stabilizer, true);
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

int stdp_common(float *weight, int Cout, int Cin, int K, int stride, int pad, const uint8_t *pre_wave, int B, int T,
                int H, int W, const int32_t *winners, const int32_t *n_winners, int k, const int8_t *reward,
                float a_plus, float a_minus, float lb, float ub, int stabilizer, void *workspace, size_t ws_bytes,
                void *stream, const char *name, bool times = false) {
    SPK_REQUIRE(Cout >= 1 && Cin >= 1 && K >= 1 && pad >= 0 && stride >= 1 && B >= 0 && T >= 1 && H >= 1 &&
                    W >= 1 && k >= 1,
                SPK_E_SHAPE, "%s: bad sizes", name);
    SPK_REQUIRE(stride <= 64, SPK_E_RANGE, "%s: stride=%d > 64", name, stride);
    SPK_REQUIRE(T <= 255, SPK_E_RANGE, "%s: T=%d > 255", name, T);
    SPK_REQUIRE(Cout <= 65535 && (int64_t)Cout * B < (1LL << 31), SPK_E_RANGE, "%s: Cout*B too large", name);
    SPK_REQUIRE((int64_t)Cin * K * K <= 65535LL * 256 && bit_rows(Cout, B, k) <= 65535 &&
                    bit_rows(Cout, B, k) * Cin * K * K < (1LL << 31),
                SPK_E_RANGE, "%s: kernel or batch too large", name);
    SPK_REQUIRE(std::isfinite(a_plus) && std::isfinite(a_minus) && std::isfinite(lb) && std::isfinite(ub) && lb <= ub,
                SPK_E_ARG, "%s: rates and bounds must be finite with lb <= ub", name);
    SPK_REQUIRE(stabilizer == 0 || stabilizer == 1, SPK_E_ARG, "%s: stabilizer must be 0 or 1", name);
    if (B == 0) return spk::ok();
    SPK_REQUIRE(weight && pre_wave && winners && n_winners, SPK_E_ARG,
                "%s: weight, pre_wave, winners and n_winners are required", name);
    size_t need = 0;
    carve(nullptr, Cout, Cin, K, B, k, &need);
    SPK_REQUIRE(workspace && ws_bytes >= need, SPK_E_WORKSPACE, "%s: workspace of %zu bytes < %zu required", name,
                ws_bytes, need);
    StdpWork wk = carve(workspace, Cout, Cin, K, B, k, nullptr);
    StdpArgs a{Cout, Cin, K, pad, stride, B, T, H, W, k, stabilizer, times ? 1 : 0, a_plus, a_minus, lb, ub};
    hipStream_t st = spk::as_stream(stream);
    const unsigned wchunks = (unsigned)spk::ceil_div((int64_t)Cin * K * K, 256);
    // the clamp can be dropped after the first update (see k_stdp_apply)
    const double rmax = std::max(std::fabs((double)a_plus), std::fabs((double)a_minus));
    const bool fast = stabilizer && rmax * ((double)ub - (double)lb) <= 0.5;
    if (B == 1 && k <= 65535) {
        if (fast)
            hipLaunchKernelGGL(k_stdp_single<true>, dim3(wchunks, (unsigned)k), dim3(256), 0, st, weight, pre_wave,
                               winners, n_winners, reward, a);
        else
            hipLaunchKernelGGL(k_stdp_single<false>, dim3(wchunks, (unsigned)k), dim3(256), 0, st, weight, pre_wave,
                               winners, n_winners, reward, a);
        return spk::check_launch(name);
    }
    hipLaunchKernelGGL(k_stdp_list, dim3(Cout), dim3(LIST_THREADS), 0, st, winners, n_winners, reward, a, wk);
    hipLaunchKernelGGL(k_stdp_offsets, dim3(1), dim3(1024), 0, st, Cout, wk);
    hipLaunchKernelGGL(k_stdp_bits, dim3(wchunks, (unsigned)wk.rows), dim3(256), 0, st, pre_wave, a, wk);
    if (fast)
        hipLaunchKernelGGL(k_stdp_apply<true>, dim3(wchunks, Cout), dim3(256), 0, st, weight, a, wk);
    else
        hipLaunchKernelGGL(k_stdp_apply<false>, dim3(wchunks, Cout), dim3(256), 0, st, weight, a, wk);
    return spk::check_launch(name);
}

}  // namespace

extern "C" size_t spk_stdp_workspace_size(int Cout, int Cin, int K, int B, int k) {
    if (Cout < 1 || Cin < 1 || K < 1 || B < 0 || k < 1) return 0;
    size_t need = 0;
    carve(nullptr, Cout, Cin, K, B, k, &need);
    return need;
}

extern "C" int spk_stdp(float *weight, int Cout, int Cin, int K, int pad, const uint8_t *pre_wave, int B, int T,
                        int H, int W, const int32_t *winners, const int32_t *n_winners, int k, float a_plus,
                        float a_minus, float lb, float ub, int stabilizer, void *workspace, size_t ws_bytes,
                        void *stream) {
    return stdp_common(weight, Cout, Cin, K, 1, pad, pre_wave, B, T, H, W, winners, n_winners, k, nullptr, a_plus,
                       a_minus, lb, ub, stabilizer, workspace, ws_bytes, stream, "spk_stdp");
}

extern "C" int spk_rstdp(float *weight, int Cout, int Cin, int K, int pad, const uint8_t *pre_wave, int B, int T,
                         int H, int W, const int32_t *winners, const int32_t *n_winners, int k, const int8_t *reward,
                         float a_plus, float a_minus, float lb, float ub, int stabilizer, void *workspace,
                         size_t ws_bytes, void *stream) {
    SPK_REQUIRE(reward || B == 0, SPK_E_ARG, "spk_rstdp: reward is required");
    return stdp_common(weight, Cout, Cin, K, 1, pad, pre_wave, B, T, H, W, winners, n_winners, k, reward, a_plus,
                       a_minus, lb, ub, stabilizer, workspace, ws_bytes, stream, "spk_rstdp");
}

extern "C" int spk_stdp_first_spike(float *weight, int Cout, int Cin, int K, int pad, const uint8_t *pre_t_first,
                                    int B, int T, int H, int W, const int32_t *winners, const int32_t *n_winners,
                                    int k, float a_plus, float a_minus, float lb, float ub, int stabilizer,
                                    void *workspace, size_t ws_bytes, void *stream) {
    return stdp_common(weight, Cout, Cin, K, 1, pad, pre_t_first, B, T, H, W, winners, n_winners, k, nullptr, a_plus,
                       a_minus, lb, ub, stabilizer, workspace, ws_bytes, stream, "spk_stdp_first_spike", true);
}

extern "C" int spk_rstdp_first_spike(float *weight, int Cout, int Cin, int K, int pad, const uint8_t *pre_t_first,
                                     int B, int T, int H, int W, const int32_t *winners, const int32_t *n_winners,
                                     int k, const int8_t *reward, float a_plus, float a_minus, float lb, float ub,
                                     int stabilizer, void *workspace, size_t ws_bytes, void *stream) {
    SPK_REQUIRE(reward || B == 0, SPK_E_ARG, "spk_rstdp_first_spike: reward is required");
    return stdp_common(weight, Cout, Cin, K, 1, pad, pre_t_first, B, T, H, W, winners, n_winners, k, reward, a_plus,
                       a_minus, lb, ub, stabilizer, workspace, ws_bytes, stream, "spk_rstdp_first_spike", true);
}

extern "C" int spk_stdp_strided(float *weight, int Cout, int Cin, int K, int stride, int pad, const uint8_t *pre_wave,
                                int B, int T, int H, int W, const int32_t *winners, const int32_t *n_winners, int k,
                                float a_plus, float a_minus, float lb, float ub, int stabilizer, void *workspace,
                                size_t ws_bytes, void *stream) {
    return stdp_common(weight, Cout, Cin, K, stride, pad, pre_wave, B, T, H, W, winners, n_winners, k, nullptr,
                       a_plus, a_minus, lb, ub, stabilizer, workspace, ws_bytes, stream, "spk_stdp_strided");
}

extern "C" int spk_rstdp_strided(float *weight, int Cout, int Cin, int K, int stride, int pad,
                                 const uint8_t *pre_wave, int B, int T, int H, int W, const int32_t *winners,
                                 const int32_t *n_winners, int k, const int8_t *reward, float a_plus, float a_minus,
                                 float lb, float ub, int stabilizer, void *workspace, size_t ws_bytes, void *stream) {
    SPK_REQUIRE(reward || B == 0, SPK_E_ARG, "spk_rstdp_strided: reward is required");
    return stdp_common(weight, Cout, Cin, K, stride, pad, pre_wave, B, T, H, W, winners, n_winners, k, reward,
                       a_plus, a_minus, lb, ub, stabilizer, workspace, ws_bytes, stream, "spk_rstdp_strided");
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
