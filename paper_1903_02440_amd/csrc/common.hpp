// Shared host/device helpers of libspyke (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstddef>
#include <cstdint>

#include "libspyke.h"

namespace spk {

// Records a formatted message for spk_last_error() and returns `code`.
int fail(int code, const char *fmt, ...);
// Clears the thread's last error and returns SPK_OK.
int ok();
// Converts the status of the most recent launch into a libspyke status.
int check_launch(const char *what);

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Hands out 256-byte aligned slices of a caller workspace.
struct Carver {
    char *base;
    size_t off = 0;
    explicit Carver(void *p) : base(static_cast<char *>(p)) {}
    template <class T>
    T *take(size_t count) {
        off = align_up(off, 256);
        T *r = reinterpret_cast<T *>(base ? base + off : nullptr);
        off += count * sizeof(T);
        return r;
    }
};

// Wave64 helpers.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) {
        uint64_t o = __shfl_xor(v, s, 64);
        v = o > v ? o : v;
    }
    return v;
}

// Eq.1 for 4 neurons at once: byte j of the result is 1 when step t has
// reached the first-spike time in byte j of t4 (times <= T, t < T).  With
// T <= 127 every byte is below 128, so (t | 0x80) - b keeps bit 7 exactly
// when t >= b and never borrows from the next byte.
__device__ __forceinline__ uint32_t spikes4(uint32_t t4, int t, int T) {
    if (T <= 127) return (((((uint32_t)t * 0x01010101u) | 0x80808080u) - t4) & 0x80808080u) >> 7;
    uint32_t w = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) w |= (uint32_t)(t >= (int)((t4 >> (8 * j)) & 255u)) << (8 * j);
    return w;
}

__device__ __forceinline__ int wave_sum_i32(int v) {
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) v += __shfl_xor(v, s, 64);
    return v;
}

}  // namespace spk

#define SPK_REQUIRE(cond, code, ...)                 \
    do {                                             \
        if (!(cond)) return spk::fail(code, __VA_ARGS__); \
    } while (0)
