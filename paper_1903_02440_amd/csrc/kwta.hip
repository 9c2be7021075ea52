// k winners-take-all with feature-wise and lateral inhibition (gfx950).
//
// Paper: section "snn Module" (winners chosen first by the earliest spike,
// then by the largest potential; lateral inhibition of the winner's
// surroundings in all feature maps) and "functional Module" (get_k_winners
// returning (feature, row, column) triplets; here with the spike step t).
//
// Every spiking neuron gets a unique 64-bit key whose unsigned order is the
// winner order:
//     bits 63..56  255 - t_first          (earlier spike wins)
//     bits 55..24  v_first, order-mapped  (larger potential wins)
//     bits 23..0   2^24 - 1 - index       (lower linear index wins ties)
// Silent neurons get key 0.  Three paths, by size:
//   * k <= 16 with per-position lists that fit in LDS: the k best keys of every
//     position, then k rounds without global reads ("per-position top-k");
//   * other small maps: tiles of 16 consecutive positions and one 256-thread
//     workgroup per image ("small maps");
//   * large maps cut each feature map into tiles of RB rows:
//   1. k_kwta_tiles: the maximum key of every tile (a group of G lanes per
//      tile, shuffle reduction), written to the workspace.
//   2. k_kwta_select: one workgroup per image keeps its tile keys in LDS and
//      runs the k rounds: block argmax (wave shuffles, then across waves),
//      emit the winner, set the lateral window in an LDS bitmap of inhibited
//      positions, clear the winner's feature tiles, and recompute only the
//      tiles whose current maximum fell inside the window -- every other
//      tile keeps its maximum, since inhibition only removes candidates.
#include <algorithm>

#include "common.hpp"

namespace {

constexpr int SEL_THREADS = 1024;
constexpr int MAX_TILES = 4096;

struct KwtaGeom {
    int B, T, C, H, W, k, r;
    int RB, nbands, ntiles;  // rows per tile, tiles per map, tiles per image
    int G;                   // lanes per tile when computing all tile maxima
    int G2;                  // lanes per tile when recomputing inhibited tiles
};

__device__ __forceinline__ uint64_t kwta_key(int t, float v, uint32_t idx) {
    uint32_t u = __float_as_uint(v);
    u = u == 0x80000000u ? 0u : u;                        // -0 and +0 are equal potentials
    u ^= (uint32_t)((int32_t)u >> 31) | 0x80000000u;     // order-preserving: ~u if negative, else u | sign
    const uint32_t hi = ((uint32_t)(255 - t) << 24) | (u >> 8);
    const uint32_t lo = (u << 24) | (0xFFFFFFu - idx);
    return ((uint64_t)hi << 32) | lo;
}

// Maximum over the wave by DPP lane moves (the value of lane 63 after moves
// within quads, half-rows, rows, then across rows), returned to every lane.
// All 64 lanes must be active.
template <int CTRL, int ROWS>
__device__ __forceinline__ uint64_t max_dpp64(uint64_t v) {
    const int lo = (int)(uint32_t)v, hi = (int)(uint32_t)(v >> 32);
    const uint64_t o = ((uint64_t)(uint32_t)__builtin_amdgcn_update_dpp(hi, hi, CTRL, ROWS, 0xF, false) << 32) |
                       (uint32_t)__builtin_amdgcn_update_dpp(lo, lo, CTRL, ROWS, 0xF, false);
    return o > v ? o : v;
}
__device__ __forceinline__ uint64_t wave_max_u64_dpp(uint64_t v) {
    v = max_dpp64<0xB1, 0xF>(v);   // quad_perm [1,0,3,2]
    v = max_dpp64<0x4E, 0xF>(v);   // quad_perm [2,3,0,1]
    v = max_dpp64<0x141, 0xF>(v);  // row_half_mirror
    v = max_dpp64<0x140, 0xF>(v);  // row_mirror
    v = max_dpp64<0x142, 0xA>(v);  // row_bcast15 into rows 1, 3
    v = max_dpp64<0x143, 0xC>(v);  // row_bcast31 into rows 2, 3
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 63);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t group_max(uint64_t v, int G) {
    for (int s = G >> 1; s >= 1; s >>= 1) {
        const uint64_t o = __shfl_xor(v, s, 64);
        v = o > v ? o : v;
    }
    return v;
}

// Maximum key of one tile over its non-inhibited neurons; all G lanes of the
// group return it.  `inh` is the LDS bitmap of laterally inhibited positions
// (nullptr before any winner exists).
__device__ __forceinline__ uint64_t tile_max(const uint8_t *tf, const float *vf, const KwtaGeom &g, int tile,
                                             int sub, int G, const uint32_t *inh) {
    const int f = tile / g.nbands, band = tile % g.nbands;
    const int y0 = band * g.RB;
    const int rows = min(g.RB, g.H - y0);
    const int nn = rows * g.W;
    const int64_t base = ((int64_t)f * g.H + y0) * g.W;
    uint64_t m = 0;
    for (int j = sub; j < nn; j += G) {
        const int pos = y0 * g.W + j;
        if (inh && ((inh[pos >> 5] >> (pos & 31)) & 1u)) continue;
        const int t = tf[base + j];
        if (t < g.T) {
            const uint64_t key = kwta_key(t, vf[base + j], (uint32_t)(base + j));
            m = key > m ? key : m;
        }
    }
    return group_max(m, G);
}

__global__ __launch_bounds__(256) void k_kwta_tiles(const uint8_t *__restrict__ tf, const float *__restrict__ vf,
                                                    KwtaGeom g, uint64_t *__restrict__ tilekey) {
    const uint32_t gid = (blockIdx.x * blockDim.x + threadIdx.x) / (uint32_t)g.G;  // < 2^31, checked on the host
    const int sub = threadIdx.x % g.G;
    const uint32_t total = (uint32_t)g.B * (uint32_t)g.ntiles;
    const bool live = gid < total;
    const uint32_t b = live ? gid / (uint32_t)g.ntiles : 0;
    const int tile = live ? (int)(gid - b * (uint32_t)g.ntiles) : 0;
    const int64_t N = (int64_t)g.C * g.H * g.W;
    // every lane takes part in the shuffles; lanes past the end read tile 0 of image 0
    const uint64_t m = tile_max(tf + b * N, vf + b * N, g, tile, sub, g.G, nullptr);
    if (live && sub == 0) tilekey[gid] = m;
}

__global__ __launch_bounds__(SEL_THREADS) void k_kwta_select(const uint8_t *__restrict__ tf_all,
                                                             const float *__restrict__ vf_all, KwtaGeom g,
                                                             const uint64_t *__restrict__ tilekey,
                                                             int32_t *__restrict__ winners,
                                                             int32_t *__restrict__ n_winners) {
    extern __shared__ uint64_t smem64[];
    uint64_t *keys = smem64;                                          // ntiles
    int *list = reinterpret_cast<int *>(keys + g.ntiles);             // ntiles
    const int nwords = (g.H * g.W + 31) / 32;
    uint32_t *inh = reinterpret_cast<uint32_t *>(list + g.ntiles);    // nwords
    __shared__ uint64_t red[SEL_THREADS / 64];
    __shared__ int nlist;

    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t N = (int64_t)g.C * g.H * g.W;
    const uint8_t *tf = tf_all + (int64_t)b * N;
    const float *vf = vf_all + (int64_t)b * N;
    int32_t *win = winners + (int64_t)b * g.k * 4;

    for (int i = tid; i < g.ntiles; i += SEL_THREADS) keys[i] = tilekey[(int64_t)b * g.ntiles + i];
    for (int i = tid; i < nwords; i += SEL_THREADS) inh[i] = 0u;
    for (int i = tid; i < 4 * g.k; i += SEL_THREADS) win[i] = -1;
    if (tid == 0) nlist = 0;
    __syncthreads();

    int found = 0;
    for (int round = 0; round < g.k; ++round) {
        uint64_t m = 0;
        for (int i = tid; i < g.ntiles; i += SEL_THREADS) m = keys[i] > m ? keys[i] : m;
        m = spk::wave_max_u64(m);
        if (lane == 0) red[wv] = m;
        __syncthreads();
        uint64_t best = 0;
        for (int w = 0; w < SEL_THREADS / 64; ++w) best = red[w] > best ? red[w] : best;
        if (best == 0) break;  // uniform: every thread read the same red[]
        const int idx = (int)(0xFFFFFFu - (uint32_t)(best & 0xFFFFFFu));
        const int t = 255 - (int)(best >> 56);
        const int f = idx / (g.H * g.W), y = (idx / g.W) % g.H, x = idx % g.W;
        if (tid == 0) {
            win[4 * round + 0] = f;
            win[4 * round + 1] = t;
            win[4 * round + 2] = y;
            win[4 * round + 3] = x;
        }
        ++found;
        // lateral window, clipped at the borders
        const int ya = max(0, y - g.r), yb = min(g.H - 1, y + g.r);
        const int xa = max(0, x - g.r), xb = min(g.W - 1, x + g.r);
        const int wh = yb - ya + 1, ww = xb - xa + 1;
        for (int i = tid; i < wh * ww; i += SEL_THREADS) {
            const int pos = (ya + i / ww) * g.W + xa + i % ww;
            atomicOr(&inh[pos >> 5], 1u << (pos & 31));
        }
        // retire the winner's feature map; list tiles whose maximum is now inhibited
        for (int i = tid; i < g.ntiles; i += SEL_THREADS) {
            const uint64_t kk = keys[i];
            if (kk == 0) continue;
            if (i / g.nbands == f) {
                keys[i] = 0;
                continue;
            }
            const int ti = (int)(0xFFFFFFu - (uint32_t)(kk & 0xFFFFFFu));
            const int ty = (ti / g.W) % g.H, tx = ti % g.W;
            if (ty >= ya && ty <= yb && tx >= xa && tx <= xb) list[atomicAdd(&nlist, 1)] = i;
        }
        __syncthreads();
        const int nl = nlist;
        const int groups = SEL_THREADS / g.G2, grp = tid / g.G2, sub = tid % g.G2;
        const int passes = (nl + groups - 1) / groups;  // identical trip count for all lanes
        for (int p = 0; p < passes; ++p) {
            const int e = p * groups + grp;
            const int tile = e < nl ? list[e] : list[0];
            const uint64_t mm = tile_max(tf, vf, g, tile, sub, g.G2, inh);
            if (e < nl && sub == 0) keys[tile] = mm;
        }
        __syncthreads();
        if (tid == 0) nlist = 0;
        __syncthreads();
    }
    if (tid == 0) n_winners[b] = found;
}

// ------------------------------------------------------------------ small maps
// When every image has at most SMALL_TILES tiles of 16 consecutive positions
// of one feature map, one 256-thread workgroup per image keeps all its tile
// keys in LDS.  Each round's argmax scan also retires the previous winner
// lazily: a tile of its feature is cleared, a tile whose maximum lies in its
// window is listed (ballot compaction) and then recomputed from global memory,
// one listed tile per thread with its loads issued together, against the LDS
// bitmap of all inhibited positions.  Quotients come from magic multipliers
// (q = umulhi(n, ceil(2^32/d)), exact for the sizes the host admits here).
constexpr int SMALL_TILES = 4096;  // keys, list and bitmap stay within 64 KB of LDS
constexpr int SMALL_THREADS = 256;

struct KwtaSmall {
    int B, T, C, HW, W, k, r, tpm, ntiles;  // tpm: 16-position tiles per feature map
    unsigned mHW, mW;                        // magic multipliers for /HW and /W
};

// n / d as umulhi(n, m) with m = ceil(2^32 / d); m == 0 stands for d == 1 (2^32 does not fit)
__device__ __forceinline__ unsigned qdiv(unsigned n, unsigned m) { return m ? __umulhi(n, m) : n; }

// The 16 first-spike times and potentials of one tile: as four 4-byte and four
// 16-byte loads when `vec` (map size a multiple of 4 and aligned bases: then
// every full tile is aligned), else as single loads.
__device__ __forceinline__ void load_tile16(const uint8_t *__restrict__ tf, const float *__restrict__ vf, int64_t base,
                                            int n, int T, int vec, int (&tv)[16], float (&vv)[16]) {
    if (vec && n == 16) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t w = *reinterpret_cast<const uint32_t *>(tf + base + 4 * q);
            const float4 v = *reinterpret_cast<const float4 *>(vf + base + 4 * q);
            tv[4 * q + 0] = w & 0xFF; tv[4 * q + 1] = (w >> 8) & 0xFF;
            tv[4 * q + 2] = (w >> 16) & 0xFF; tv[4 * q + 3] = w >> 24;
            vv[4 * q + 0] = v.x; vv[4 * q + 1] = v.y; vv[4 * q + 2] = v.z; vv[4 * q + 3] = v.w;
        }
    } else {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            tv[j] = j < n ? (int)tf[base + j] : T;
            vv[j] = j < n ? vf[base + j] : 0.0f;
        }
    }
}

// Four lanes per tile, each with 4 consecutive positions, so a wave's loads
// are contiguous; two shuffle steps combine the quarter maxima.  Grid-stride
// over the batch's tiles (the stride is a multiple of 4 lanes), four strides
// per pass with all their loads issued before any is used.
__global__ __launch_bounds__(256) void k_kwta_tiles16(const uint8_t *__restrict__ tf, const float *__restrict__ vf,
                                                      KwtaSmall g, int vec, uint64_t *__restrict__ tilekey) {
    constexpr int U = 4;
    const uint32_t total = (uint32_t)g.B * (uint32_t)g.ntiles * 4u;  // < 2^31, checked on the host
    const uint32_t stride = gridDim.x * 256u;
    for (uint32_t g0 = blockIdx.x * 256u; g0 < total; g0 += U * stride) {  // uniform per workgroup
        int tv[U][4];
        float vv[U][4];
        uint32_t idx0[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t gt = g0 + u * stride + threadIdx.x;
            const uint32_t gid = gt >> 2;
            const int sub = (int)(gt & 3u);
            idx0[u] = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                tv[u][j] = g.T;
                vv[u][j] = 0.0f;
            }
            if (gt < total) {
                const uint32_t b = gid / (uint32_t)g.ntiles;
                const int tile = (int)(gid - b * (uint32_t)g.ntiles);
                const int f = tile / g.tpm, pos0 = (tile - f * g.tpm) * 16 + 4 * sub;
                const int64_t base = (int64_t)b * g.C * g.HW + (int64_t)f * g.HW + pos0;
                idx0[u] = (uint32_t)(f * g.HW + pos0);
                if (vec && pos0 + 4 <= g.HW) {
                    const uint32_t w = *reinterpret_cast<const uint32_t *>(tf + base);
                    const float4 v = *reinterpret_cast<const float4 *>(vf + base);
                    tv[u][0] = w & 0xFF; tv[u][1] = (w >> 8) & 0xFF; tv[u][2] = (w >> 16) & 0xFF; tv[u][3] = w >> 24;
                    vv[u][0] = v.x; vv[u][1] = v.y; vv[u][2] = v.z; vv[u][3] = v.w;
                } else {
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const bool ok = pos0 + j < g.HW;
                        tv[u][j] = ok ? (int)tf[base + j] : g.T;
                        vv[u][j] = ok ? vf[base + j] : 0.0f;
                    }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t gt = g0 + u * stride + threadIdx.x;
            uint64_t m = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (tv[u][j] < g.T) {
                    const uint64_t key = kwta_key(tv[u][j], vv[u][j], idx0[u] + j);
                    m = key > m ? key : m;
                }
            m = group_max(m, 4);
            if (gt < total && (gt & 3u) == 0) tilekey[gt >> 2] = m;
        }
    }
}

__device__ __forceinline__ uint64_t recompute16(const uint8_t *__restrict__ tf, const float *__restrict__ vf,
                                                const KwtaSmall &g, int vec, int tile, const uint32_t *inh) {
    const int f = tile / g.tpm, pos0 = (tile - f * g.tpm) * 16;
    const int base = f * g.HW + pos0;
    int tv[16];
    float vv[16];
    load_tile16(tf, vf, base, min(16, g.HW - pos0), g.T, vec, tv, vv);
    uint64_t m = 0;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        const int pos = pos0 + j;
        if (tv[j] < g.T && !((inh[pos >> 5] >> (pos & 31)) & 1u)) {
            const uint64_t key = kwta_key(tv[j], vv[j], (uint32_t)(base + j));
            m = key > m ? key : m;
        }
    }
    return m;
}

__global__ __launch_bounds__(SMALL_THREADS) void k_kwta_select_small(const uint8_t *__restrict__ tf_all,
                                                                     const float *__restrict__ vf_all, KwtaSmall g,
                                                                     int vec, const uint64_t *__restrict__ tilekey,
                                                                     int32_t *__restrict__ winners,
                                                                     int32_t *__restrict__ n_winners) {
    extern __shared__ uint64_t keys[];  // ntiles keys, the inhibition bitmap, ntiles list entries
    const int nwords = (g.HW + 31) / 32;
    uint32_t *inh = reinterpret_cast<uint32_t *>(keys + g.ntiles);
    uint16_t *list = reinterpret_cast<uint16_t *>(inh + nwords);
    __shared__ uint64_t red[SMALL_THREADS / 64];
    __shared__ int nlist[2];
    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t N = (int64_t)g.C * g.HW;
    const uint8_t *tf = tf_all + (int64_t)b * N;
    const float *vf = vf_all + (int64_t)b * N;
    int32_t *win = winners + (int64_t)b * g.k * 4;
    for (int i = tid; i < g.ntiles; i += SMALL_THREADS) keys[i] = tilekey[(int64_t)b * g.ntiles + i];
    for (int i = tid; i < nwords; i += SMALL_THREADS) inh[i] = 0u;
    for (int i = tid; i < 4 * g.k; i += SMALL_THREADS) win[i] = -1;
    if (tid < 2) nlist[tid] = 0;
    __syncthreads();
    const uint64_t below = (1ULL << lane) - 1ULL;  // lanes under this one
    const int H = g.HW / g.W;
    int fw = -1, yw = 0, xw = 0, found = 0;
    for (int round = 0; round < g.k; ++round) {
        int *cnt = &nlist[round & 1];
        // scan: retire the previous winner's feature, list the tiles whose
        // maximum fell in its window, and take the maximum of the rest
        uint64_t m = 0;
        for (int i0 = 0; i0 < g.ntiles; i0 += SMALL_THREADS) {
            const int i = i0 + tid;
            uint64_t key = i < g.ntiles ? keys[i] : 0;
            bool redo = false;
            if (key != 0 && fw >= 0) {
                const unsigned idx = 0xFFFFFFu - (unsigned)(key & 0xFFFFFFu);
                const unsigned f = qdiv(idx, g.mHW), pos = idx - f * (unsigned)g.HW;
                const int y = (int)qdiv(pos, g.mW), x = (int)pos - y * g.W;
                if ((int)f == fw) {
                    key = 0;
                    keys[i] = 0;
                } else if (abs(y - yw) <= g.r && abs(x - xw) <= g.r) {
                    redo = true;
                    key = 0;
                }
            }
            const uint64_t mask = __ballot(redo);
            if (mask) {
                int at = 0;
                if (lane == 0) at = atomicAdd(cnt, __popcll(mask));
                at = __shfl(at, 0, 64);
                if (redo) list[at + __popcll(mask & below)] = (uint16_t)i;
            }
            m = key > m ? key : m;
        }
        __syncthreads();
        // recompute the listed tiles, one per thread
        const int nl = *cnt;
        for (int e = tid; e < nl; e += SMALL_THREADS) {
            const int tile = list[e];
            const uint64_t key = recompute16(tf, vf, g, vec, tile, inh);
            keys[tile] = key;
            m = key > m ? key : m;
        }
        m = spk::wave_max_u64(m);
        if (lane == 0) red[wv] = m;
        __syncthreads();
        uint64_t best = 0;
#pragma unroll
        for (int w = 0; w < SMALL_THREADS / 64; ++w) best = red[w] > best ? red[w] : best;
        if (tid == 0) nlist[(round + 1) & 1] = 0;  // the other counter: last read before the previous barrier
        if (best == 0) break;  // uniform: every thread read the same red[]
        const int idx = (int)(0xFFFFFFu - (unsigned)(best & 0xFFFFFFu));
        const int t = 255 - (int)(best >> 56);
        fw = (int)qdiv((unsigned)idx, g.mHW);
        const int pos = idx - fw * g.HW;
        yw = (int)qdiv((unsigned)pos, g.mW);
        xw = pos - yw * g.W;
        if (tid == 0) {
            win[4 * round + 0] = fw;
            win[4 * round + 1] = t;
            win[4 * round + 2] = yw;
            win[4 * round + 3] = xw;
        }
        ++found;
        const int ya = max(0, yw - g.r), yb = min(H - 1, yw + g.r);
        const int xa = max(0, xw - g.r), xb = min(g.W - 1, xw + g.r);
        const int wh = yb - ya + 1, ww = xb - xa + 1;
        for (int i = tid; i < wh * ww; i += SMALL_THREADS) {
            const int p = (ya + i / ww) * g.W + xa + i % ww;
            atomicOr(&inh[p >> 5], 1u << (p & 31));
        }
        __syncthreads();
    }
    if (tid == 0) n_winners[b] = found;
}

// ------------------------------------------------------------ per-position top-k
// When k <= 16 and each image's lists fit in LDS, one workgroup per image
// first keeps, for every position, the k largest keys over all feature maps:
// one pass over the image's neurons, with each position owned by one thread
// (on maps of few positions, the feature maps are split among up to
// TOPK_THREADS / HW threads per position, whose lists the owner then merges;
// small batches, which leave most CUs idle, take up to TOPK_THREADS_SMALL_B
// threads per workgroup so that each thread scans fewer feature maps).
// The rounds never read global memory again.  At round j at most j features
// are retired, so a position's best live key is among its first j + 1 list
// entries: the owner skips entries of retired features with a per-position
// cursor, and marks its position inhibited when it falls in a winner's
// window (with at most 4 positions per thread, the cursors and the current
// best keys live in registers).  Only the per-round maximum crosses threads.
constexpr int TOPK_THREADS = 256;       // most threads per workgroup
constexpr int TOPK_THREADS_SMALL_B = 1024;  // most threads per workgroup for batches below TOPK_SMALL_B
constexpr int TOPK_SMALL_B = 256;
constexpr int TOPK_MAX_K = 16;
constexpr size_t TOPK_LDS = 40 * 1024;  // lists and cursors (the stash adds 16 KB)
constexpr int TOPK_U = 8;               // feature maps loaded per block
constexpr int TOPK_STASH_MIN = 64;      // features per split from which the stash pays
constexpr int TOPK_RP = 4;              // positions per thread up to which the rounds keep their keys in registers
// Batches below TOPK_PRE_B images (online steps) leave most CUs idle: the
// lists are then built by a grid of (image, split of the feature maps)
// workgroups into the workspace, and the rounds' workgroup merges them.
constexpr int TOPK_PRE_B = 8;
constexpr int TOPK_PRE_NS = 16;         // feature splits at most
constexpr int TOPK_PRE_HW = 4096;       // positions at most

struct KwtaTopk {
    int B, T, C, HW, W, k, r;
    int S, fps;  // feature splits per position (small maps) and features per split
    int nt;      // threads per workgroup
    unsigned mHW, mW;
    int ns, fps2;  // workgroup feature splits and their features (ns > 1: lists built by k_kwta_lists)
    uint64_t *lg;  // their lists, [B][ns][HW][KM]
};

// Inserts key into the descending list top (keys are unique; the caller has
// checked key > top[KM - 1], so the last entry drops out).
template <int KM>
__device__ __forceinline__ void topk_insert(uint64_t (&top)[KM], uint64_t key) {
    bool gt[KM];  // every comparison first, then the moves
#pragma unroll
    for (int i = 0; i < KM; ++i) gt[i] = key > top[i];
#pragma unroll
    for (int i = KM - 1; i > 0; --i) top[i] = gt[i - 1] ? top[i - 1] : (gt[i] ? key : top[i]);
    top[0] = gt[0] ? key : top[0];
}

// Grid (image, split): the KM best keys of every position over the split's
// feature maps, into g.lg.
template <int KM, int U>
__global__ __launch_bounds__(TOPK_THREADS_SMALL_B) void k_kwta_lists(const uint8_t *__restrict__ tf_all,
                                                             const float *__restrict__ vf_all, KwtaTopk g) {
    const int b = blockIdx.x, sp = blockIdx.y, HW = g.HW;
    const int64_t N = (int64_t)g.C * HW;
    const uint8_t *tf = tf_all + (int64_t)b * N;
    const float *vf = vf_all + (int64_t)b * N;
    const int fa = sp * g.fps2, fb = min(g.C, fa + g.fps2);
    for (int p = threadIdx.x; p < HW; p += blockDim.x) {
        uint64_t top[KM];
#pragma unroll
        for (int i = 0; i < KM; ++i) top[i] = 0;
        for (int f0 = fa; f0 < fb; f0 += U) {
            int tv[U];
            float vv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const bool ok = f0 + u < fb;
                const int o = (f0 + u) * HW + p;
                tv[u] = ok ? (int)tf[o] : g.T;
                vv[u] = ok ? vf[o] : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (tv[u] < g.T) {
                    const uint64_t key = kwta_key(tv[u], vv[u], (uint32_t)((f0 + u) * HW + p));
                    if (key > top[KM - 1]) topk_insert(top, key);
                }
            }
        }
        uint64_t *dst = g.lg + (((int64_t)b * g.ns + sp) * HW + p) * KM;
#pragma unroll
        for (int i = 0; i < KM; ++i) dst[i] = top[i];
    }
}

template <int KM, int U, bool STASH>
__global__ __launch_bounds__(TOPK_THREADS_SMALL_B) void k_kwta_topk(const uint8_t *__restrict__ tf_all,
                                                            const float *__restrict__ vf_all, KwtaTopk g,
                                                            int32_t *__restrict__ winners,
                                                            int32_t *__restrict__ n_winners) {
    extern __shared__ uint64_t lists[];  // [S][HW][KM] keys, then [HW] cursors
    uint8_t *cur = reinterpret_cast<uint8_t *>(lists + (size_t)g.S * g.HW * KM);
    __shared__ uint64_t red[2][TOPK_THREADS_SMALL_B / 64];
    // a block's keys, read back by their own lane (STASH launches have at most TOPK_THREADS threads)
    __shared__ uint64_t stash[STASH ? U : 1][TOPK_THREADS];
    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int NT = blockDim.x, NW = NT >> 6;
    const int HW = g.HW, S = g.S;
    const int64_t N = (int64_t)g.C * HW;
    const uint8_t *tf = tf_all + (int64_t)b * N;
    const float *vf = vf_all + (int64_t)b * N;
    int32_t *win = winners + (int64_t)b * g.k * 4;
    for (int i = tid; i < 4 * g.k; i += NT) win[i] = -1;

    if (g.ns > 1) {  // the lists of the workgroup splits, merged (each is sorted)
        for (int p = tid; p < HW; p += NT) {
            uint64_t top[KM];
#pragma unroll
            for (int i = 0; i < KM; ++i) top[i] = 0;
            for (int sp = 0; sp < g.ns; ++sp) {
                const uint64_t *src = g.lg + (((int64_t)b * g.ns + sp) * HW + p) * KM;
                for (int e = 0; e < KM; ++e) {
                    const uint64_t key = src[e];
                    if (!(key > top[KM - 1])) break;
                    topk_insert(top, key);
                }
            }
#pragma unroll
            for (int i = 0; i < KM; ++i) lists[(size_t)p * KM + i] = top[i];
        }
    }
    // pass over the image: the KM best keys of every (position, feature split)
    for (int pp = tid; pp < (g.ns > 1 ? 0 : HW * S); pp += NT) {
        const int s = (int)qdiv((unsigned)pp, g.mHW), p = pp - s * HW;
        uint64_t top[KM];
#pragma unroll
        for (int i = 0; i < KM; ++i) top[i] = 0;
        const int fa = s * g.fps, fb = min(g.C, fa + g.fps);
        for (int f0 = fa; f0 < fb; f0 += U) {
            int tv[U];
            float vv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const bool ok = f0 + u < fb;
                const int o = (f0 + u) * HW + p;
                tv[u] = ok ? (int)tf[o] : g.T;
                vv[u] = ok ? vf[o] : 0.0f;
            }
            if constexpr (STASH) {
                // the keys that beat the list's last entry are inserted after the
                // block, each lane walking only its own: the wave then loops as
                // often as its busiest lane rather than once per key any lane keeps
                unsigned pass = 0;
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const uint64_t key = tv[u] < g.T ? kwta_key(tv[u], vv[u], (uint32_t)((f0 + u) * HW + p)) : 0;
                    stash[u][tid] = key;
                    pass |= (key > top[KM - 1] ? 1u : 0u) << u;
                }
                while (pass) {
                    const int j = __builtin_ctz(pass);
                    pass &= pass - 1;
                    const uint64_t key = stash[j][tid];
                    if (key > top[KM - 1]) topk_insert(top, key);
                }
            } else {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    if (tv[u] < g.T) {
                        const uint64_t key = kwta_key(tv[u], vv[u], (uint32_t)((f0 + u) * HW + p));
                        if (key > top[KM - 1]) topk_insert(top, key);
                    }
                }
            }
        }
#pragma unroll
        for (int i = 0; i < KM; ++i) lists[(size_t)pp * KM + i] = top[i];
    }
    if (S > 1 && g.ns <= 1) {  // uniform
        __syncthreads();
        // owners fold the other splits' lists into their own
        for (int p = tid; p < HW; p += NT) {
            uint64_t top[KM];
#pragma unroll
            for (int i = 0; i < KM; ++i) top[i] = lists[(size_t)p * KM + i];
            for (int s = 1; s < S; ++s)
                for (int e = 0; e < KM; ++e) {
                    const uint64_t key = lists[((size_t)s * HW + p) * KM + e];
                    if (!(key > top[KM - 1])) break;  // the split's list is sorted
                    topk_insert(top, key);
                }
#pragma unroll
            for (int i = 0; i < KM; ++i) lists[(size_t)p * KM + i] = top[i];
        }
    }
    int deadf[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) deadf[j] = -1;
    int found = 0;
    auto feature = [&](uint64_t key) { return (int)qdiv(0xFFFFFFu - (unsigned)(key & 0xFFFFFFu), g.mHW); };
    auto is_dead = [&](int f) {
        bool dead = false;
#pragma unroll
        for (int j = 0; j < KM; ++j) dead |= deadf[j] == f;
        return dead;
    };
    if (HW <= TOPK_RP * NT) {  // uniform
        // Each thread holds the best live key of each of its positions in
        // registers (0: none, or inhibited).  A round changes it only where the
        // winner's window covers the position, or where the cached key belongs to
        // the winner's feature: then the list is walked on to the next entry of a
        // live feature (the cached key stays the best live one otherwise).
        uint64_t bk[TOPK_RP];
        int cc[TOPK_RP], py[TOPK_RP], px[TOPK_RP];
#pragma unroll
        for (int i = 0; i < TOPK_RP; ++i) {
            const int p = tid + i * NT;
            bk[i] = p < HW ? lists[(size_t)p * KM] : 0;
            cc[i] = 0;
            py[i] = (int)qdiv((unsigned)min(p, HW - 1), g.mW);
            px[i] = min(p, HW - 1) - py[i] * g.W;
        }
        for (int round = 0; round < g.k; ++round) {
            uint64_t m = 0;
#pragma unroll
            for (int i = 0; i < TOPK_RP; ++i) m = bk[i] > m ? bk[i] : m;
            m = wave_max_u64_dpp(m);
            if (lane == 0) red[round & 1][wv] = m;
            __syncthreads();
            uint64_t best = 0;
#pragma unroll
            for (int w = 0; w < NW; ++w) best = red[round & 1][w] > best ? red[round & 1][w] : best;
            if (best == 0) break;  // uniform
            const int idx = (int)(0xFFFFFFu - (unsigned)(best & 0xFFFFFFu));
            const int t = 255 - (int)(best >> 56);
            const int fw = (int)qdiv((unsigned)idx, g.mHW);
            const int pos = idx - fw * HW;
            const int yw = (int)qdiv((unsigned)pos, g.mW);
            const int xw = pos - yw * g.W;
            if (tid == 0) {
                win[4 * round + 0] = fw;
                win[4 * round + 1] = t;
                win[4 * round + 2] = yw;
                win[4 * round + 3] = xw;
            }
#pragma unroll
            for (int j = 0; j < KM; ++j)
                if (j == found) deadf[j] = fw;
            ++found;
#pragma unroll
            for (int i = 0; i < TOPK_RP; ++i) {
                if (bk[i] == 0) continue;
                if (abs(py[i] - yw) <= g.r && abs(px[i] - xw) <= g.r) {
                    bk[i] = 0;
                    continue;
                }
                if (feature(bk[i]) != fw) continue;
                const int p = tid + i * NT;
                uint64_t key = 0;
                for (int c = cc[i] + 1; c < KM; ++c) {
                    const uint64_t e = lists[(size_t)p * KM + c];
                    if (e == 0) break;
                    if (!is_dead(feature(e))) {
                        key = e;
                        cc[i] = c;
                        break;
                    }
                }
                bk[i] = key;
            }
        }
    } else {
        for (int p = tid; p < HW; p += NT) cur[p] = 0;
        for (int round = 0; round < g.k; ++round) {
            uint64_t m = 0;
            for (int p = tid; p < HW; p += NT) {
                int c = cur[p];
                if (c == 0xFF) continue;  // laterally inhibited
                const int c0 = c;
                uint64_t key = 0;
                for (; c < KM; ++c) {
                    key = lists[(size_t)p * KM + c];
                    if (key == 0) break;
                    if (!is_dead(feature(key))) break;
                    key = 0;
                }
                if (c != c0) cur[p] = (uint8_t)c;
                m = key > m ? key : m;
            }
            m = wave_max_u64_dpp(m);
            if (lane == 0) red[round & 1][wv] = m;
            __syncthreads();
            uint64_t best = 0;
#pragma unroll
            for (int w = 0; w < NW; ++w) best = red[round & 1][w] > best ? red[round & 1][w] : best;
            if (best == 0) break;  // uniform
            const int idx = (int)(0xFFFFFFu - (unsigned)(best & 0xFFFFFFu));
            const int t = 255 - (int)(best >> 56);
            const int fw = (int)qdiv((unsigned)idx, g.mHW);
            const int pos = idx - fw * HW;
            const int yw = (int)qdiv((unsigned)pos, g.mW);
            const int xw = pos - yw * g.W;
            if (tid == 0) {
                win[4 * round + 0] = fw;
                win[4 * round + 1] = t;
                win[4 * round + 2] = yw;
                win[4 * round + 3] = xw;
            }
#pragma unroll
            for (int j = 0; j < KM; ++j)
                if (j == found) deadf[j] = fw;
            ++found;
            for (int p = tid; p < HW; p += NT) {
                const int y = (int)qdiv((unsigned)p, g.mW), x = p - y * g.W;
                if (abs(y - yw) <= g.r && abs(x - xw) <= g.r) cur[p] = 0xFF;
            }
        }
    }
    if (tid == 0) n_winners[b] = found;
}

bool kwta_topk(int B, int T, int C, int H, int W, int k, int r, KwtaTopk &s) {
    const int64_t HW = (int64_t)H * W;
    if (k > TOPK_MAX_K || HW > 65536) return false;
    // maps of few positions split the feature maps among up to NT / HW threads per position
    const int NT = B < TOPK_SMALL_B ? TOPK_THREADS_SMALL_B : TOPK_THREADS;
    int S = HW <= NT ? (int)std::min<int64_t>(C, NT / HW) : 1;
    while (S > 1 && (size_t)HW * (S * k * sizeof(uint64_t) + 1) > TOPK_LDS) --S;  // the splits' lists fit
    const int fps = (C + S - 1) / S;
    S = (C + fps - 1) / fps;
    // threads: whole waves covering HW * S in as few passes as NT allows
    const int64_t work = HW * S, passes = (work + NT - 1) / NT;
    const int nt = (int)(((work + passes - 1) / passes + 63) / 64 * 64);
    if ((size_t)HW * (S * k * sizeof(uint64_t) + 1) > TOPK_LDS) return false;
    auto magic = [](int64_t d) {  // 0 for d == 1 (see qdiv)
        return d == 1 ? 0u : (unsigned)(((1ULL << 32) + (uint64_t)d - 1) / (uint64_t)d);
    };
    auto exact = [](int64_t d, int64_t n) {  // umulhi(x, ceil(2^32/d)) == x/d for all x < n
        const uint64_t m = ((1ULL << 32) + (uint64_t)d - 1) / (uint64_t)d;
        const uint64_t e = m * (uint64_t)d - (1ULL << 32);
        return (uint64_t)n * e < (1ULL << 32);
    };
    if (!exact(HW, (int64_t)C * HW) || !exact(W, HW)) return false;
    s = KwtaTopk{B, T, C, (int)HW, W, k, r, S, fps, nt, magic(HW), magic(W), 1, C, nullptr};
    if (B < TOPK_PRE_B && HW <= TOPK_PRE_HW) {  // lists by a grid of workgroups (the rounds' workgroup: S = 1)
        const int ns = (int)std::min<int64_t>(TOPK_PRE_NS, (C + 15) / 16);
        if (ns > 1) {
            s.ns = ns;
            s.fps2 = (C + ns - 1) / ns;
            s.ns = (C + s.fps2 - 1) / s.fps2;
            s.S = 1;
            s.fps = C;
            const int64_t passes = (HW + NT - 1) / NT;
            s.nt = (int)(((HW + passes - 1) / passes + 63) / 64 * 64);
        }
    }
    return true;
}

template <int KM>
void launch_topk(const KwtaTopk &s, const uint8_t *tf, const float *vf, int32_t *winners, int32_t *nw,
                 hipStream_t st) {
    const size_t lds = (size_t)s.HW * (s.S * KM * sizeof(uint64_t) + 1);
    if (s.ns > 1) {
        const int nt = (int)std::min<int64_t>(TOPK_THREADS_SMALL_B, ((int64_t)s.HW + 63) / 64 * 64);
        hipLaunchKernelGGL(HIP_KERNEL_NAME(k_kwta_lists<KM, TOPK_U>), dim3(s.B, s.ns), dim3(nt), 0, st, tf, vf, s);
        hipLaunchKernelGGL(HIP_KERNEL_NAME(k_kwta_topk<KM, TOPK_U, false>), dim3(s.B), dim3(s.nt), lds, st, tf, vf,
                           s, winners, nw);
        return;
    }
    if (s.fps >= TOPK_STASH_MIN && s.nt <= TOPK_THREADS)
        hipLaunchKernelGGL(HIP_KERNEL_NAME(k_kwta_topk<KM, TOPK_U, true>), dim3(s.B), dim3(s.nt), lds, st, tf, vf, s,
                           winners, nw);
    else
        hipLaunchKernelGGL(HIP_KERNEL_NAME(k_kwta_topk<KM, TOPK_U, false>), dim3(s.B), dim3(s.nt), lds, st, tf, vf, s,
                           winners, nw);
}

void dispatch_topk(const KwtaTopk &s, const uint8_t *tf, const float *vf, int32_t *winners, int32_t *nw,
                   hipStream_t st) {
    switch (s.k) {
#define SPK_TOPK(K) \
    case K: launch_topk<K>(s, tf, vf, winners, nw, st); break;
        SPK_TOPK(1) SPK_TOPK(2) SPK_TOPK(3) SPK_TOPK(4) SPK_TOPK(5) SPK_TOPK(6) SPK_TOPK(7) SPK_TOPK(8)
        SPK_TOPK(9) SPK_TOPK(10) SPK_TOPK(11) SPK_TOPK(12) SPK_TOPK(13) SPK_TOPK(14) SPK_TOPK(15) SPK_TOPK(16)
#undef SPK_TOPK
        default: break;
    }
}

bool kwta_small(int B, int T, int C, int H, int W, int k, int r, KwtaSmall &s) {
    const int64_t HW = (int64_t)H * W;
    const int64_t tpm = (HW + 15) / 16;
    if (HW > 65536 || C * tpm > SMALL_TILES) return false;
    auto magic = [](int64_t d) {  // 0 for d == 1 (see qdiv)
        return d == 1 ? 0u : (unsigned)(((1ULL << 32) + (uint64_t)d - 1) / (uint64_t)d);
    };
    auto exact = [](int64_t d, int64_t n) {  // umulhi(x, ceil(2^32/d)) == x/d for all x < n
        const uint64_t m = ((1ULL << 32) + (uint64_t)d - 1) / (uint64_t)d;
        const uint64_t e = m * (uint64_t)d - (1ULL << 32);
        return (uint64_t)n * e < (1ULL << 32);
    };
    if (!exact(HW, (int64_t)C * HW) || !exact(W, HW)) return false;
    if ((int64_t)B * C * tpm * 16 >= (1LL << 31)) return false;
    s = KwtaSmall{B, T, C, (int)HW, W, k, r, (int)tpm, (int)(C * tpm), magic(HW), magic(W)};
    return true;
}

int kwta_geom(int B, int T, int C, int H, int W, int k, int r, KwtaGeom &g) {
    SPK_REQUIRE(B >= 0 && T >= 1 && C >= 1 && H >= 1 && W >= 1, SPK_E_SHAPE, "spk_kwta: bad sizes");
    SPK_REQUIRE(T <= 255, SPK_E_RANGE, "spk_kwta: T=%d > 255", T);
    SPK_REQUIRE((int64_t)C * H * W <= (1LL << 24), SPK_E_RANGE, "spk_kwta: C*H*W > 2^24");
    SPK_REQUIRE((int64_t)H * W <= 65536, SPK_E_RANGE, "spk_kwta: H*W > 65536");
    SPK_REQUIRE(k >= 1 && r >= 0, SPK_E_ARG, "spk_kwta: k=%d must be >= 1 and radius=%d >= 0", k, r);
    g.B = B; g.T = T; g.C = C; g.H = H; g.W = W; g.k = k; g.r = r;
    int RB = 1;
    while (RB < H && (int64_t)C * ((H + RB - 1) / RB) > MAX_TILES) RB *= 2;
    RB = RB > H ? H : RB;
    g.RB = RB;
    g.nbands = (H + RB - 1) / RB;
    SPK_REQUIRE((int64_t)C * g.nbands <= MAX_TILES, SPK_E_RANGE, "spk_kwta: %d feature maps exceed %d tiles", C,
                MAX_TILES);
    g.ntiles = C * g.nbands;
    const int nn = RB * W;
    int G = 1;
    while (G < nn && G < 64) G <<= 1;
    g.G = G;
    // small tiles are recomputed one per thread: their loads then overlap
    // instead of waiting on each other group after group
    g.G2 = nn <= 32 ? 1 : G;
    SPK_REQUIRE((int64_t)B * g.ntiles * G < (1LL << 31), SPK_E_RANGE, "spk_kwta: batch too large");
    return SPK_OK;
}

}  // namespace

extern "C" size_t spk_kwta_workspace_size(int B, int C, int H, int W) {
    KwtaGeom g;
    if (kwta_geom(B, 1, C, H, W, 1, 0, g) != SPK_OK) return 0;
    KwtaSmall sm;
    const int ntiles = kwta_small(B, 1, C, H, W, 1, 0, sm) ? sm.ntiles : g.ntiles;
    size_t need = (size_t)B * ntiles * sizeof(uint64_t);
    if (B < TOPK_PRE_B && (int64_t)H * W <= TOPK_PRE_HW)  // the workgroup splits' lists (any k up to TOPK_MAX_K)
        need = std::max(need, (size_t)B * TOPK_PRE_NS * H * W * TOPK_MAX_K * sizeof(uint64_t));
    return spk::align_up(need, 256);
}

extern "C" int spk_kwta(const uint8_t *t_first, const float *v_first, int B, int T, int C, int H, int W, int k,
                        int radius, int32_t *winners, int32_t *n_winners, void *workspace, size_t ws_bytes,
                        void *stream) {
    KwtaGeom g;
    int rc = kwta_geom(B, T, C, H, W, k, radius, g);
    if (rc != SPK_OK) return rc;
    if (B == 0) return spk::ok();
    SPK_REQUIRE(t_first && v_first && winners && n_winners, SPK_E_ARG,
                "spk_kwta: t_first, v_first, winners and n_winners are required");
    const size_t need = spk_kwta_workspace_size(B, C, H, W);
    SPK_REQUIRE(workspace && ws_bytes >= need, SPK_E_WORKSPACE, "spk_kwta: workspace of %zu bytes < %zu required",
                ws_bytes, need);
    hipStream_t st = spk::as_stream(stream);
    uint64_t *tilekey = static_cast<uint64_t *>(workspace);
    KwtaTopk tk;
    if (kwta_topk(B, T, C, H, W, k, radius, tk)) {
        tk.lg = static_cast<uint64_t *>(workspace);
        dispatch_topk(tk, t_first, v_first, winners, n_winners, st);
        return spk::check_launch("spk_kwta");
    }
    KwtaSmall sm;
    if (kwta_small(B, T, C, H, W, k, radius, sm)) {
        const int64_t threads = (int64_t)B * sm.ntiles * 4;
        const int vec = (sm.HW % 4) == 0 && ((uintptr_t)t_first & 3) == 0 && ((uintptr_t)v_first & 15) == 0;
        hipLaunchKernelGGL(k_kwta_tiles16, dim3((unsigned)std::min<int64_t>(spk::ceil_div(threads, 256), 8192)),
                           dim3(256), 0, st, t_first,
                           v_first, sm, vec, tilekey);
        const size_t lds = (size_t)sm.ntiles * (sizeof(uint64_t) + sizeof(uint16_t)) + (size_t)(sm.HW + 31) / 32 * 4;
        hipLaunchKernelGGL(k_kwta_select_small, dim3(B), dim3(SMALL_THREADS), lds, st, t_first, v_first, sm, vec,
                           tilekey, winners, n_winners);
        return spk::check_launch("spk_kwta");
    }
    const int64_t threads = (int64_t)B * g.ntiles * g.G;
    hipLaunchKernelGGL(k_kwta_tiles, dim3((unsigned)spk::ceil_div(threads, 256)), dim3(256), 0, st, t_first, v_first,
                       g, tilekey);
    const size_t lds = (size_t)g.ntiles * (sizeof(uint64_t) + sizeof(int)) + ((size_t)H * W + 31) / 32 * 4;
    hipLaunchKernelGGL(k_kwta_select, dim3(B), dim3(SEL_THREADS), lds, st, t_first, v_first, g, tilekey, winners,
                       n_winners);
    return spk::check_launch("spk_kwta");
}
