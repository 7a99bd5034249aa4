// Device helpers shared by the pricing kernels (gfx950, wave64).
#pragma once

#include "exact_math.h"
#include "heddle_internal.h"

namespace heddle {

// LDS writes of a wavefront become visible to its other lanes
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int rl32(int v, int lane) { return __builtin_amdgcn_readlane(v, lane); }

__device__ __forceinline__ int64_t rl64(int64_t v, int lane)
{
    uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
    uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), lane);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// lane `lane` of a 32- or 64-bit value, as a wave-uniform value
__device__ __forceinline__ uint32_t uni64(uint32_t v, int lane) { return (uint32_t)__builtin_amdgcn_readlane((int)v, lane); }
__device__ __forceinline__ uint64_t uni64(uint64_t v, int lane) { return (uint64_t)rl64((int64_t)v, lane); }

template <class T> __device__ __forceinline__ T wave_min(T v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        T u = __shfl_xor(v, o);
        v = u < v ? u : v;
    }
    return v;
}

template <class T> __device__ __forceinline__ T wave_max(T v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        T u = __shfl_xor(v, o);
        v = u > v ? u : v;
    }
    return v;
}

// lane mask of a condition (the compare feeds the mask directly)
__device__ __forceinline__ uint64_t ballot(bool c) { return __builtin_amdgcn_ballot_w64(c); }

// uniform value into a scalar register
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

// v with lane `lane` (uniform) replaced by the uniform value x
__device__ __forceinline__ int put_lane(int v, int x, int lane) { return (int)__lane_id() == lane ? x : v; }

// DPP lane permutations within rows of 16 lanes (every source lane exists, so
// bound_ctrl never applies); the move folds into the DPP operand of the min
// or max that consumes it
template <int CTRL> __device__ __forceinline__ uint32_t dpp32(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true);
}
template <int CTRL> __device__ __forceinline__ uint64_t dpp64(uint64_t v)
{
    return ((uint64_t)dpp32<CTRL>((uint32_t)(v >> 32)) << 32) | dpp32<CTRL>((uint32_t)v);
}
template <int CTRL> __device__ __forceinline__ uint32_t dpp(uint32_t v) { return dpp32<CTRL>(v); }
template <int CTRL> __device__ __forceinline__ uint64_t dpp(uint64_t v) { return dpp64<CTRL>(v); }

constexpr int kDppXor1 = 0xB1;          // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;          // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;   // lane i <-> 7 - i within 8
constexpr int kDppMirror = 0x140;       // lane i <-> 15 - i within 16
constexpr int kDppWaveShl1 = 0x130;     // lane i <- lane i + 1 across the wavefront (lane 63 keeps the old value)
constexpr int kDppWaveShr1 = 0x138;     // lane i <- lane i - 1 across the wavefront (lane 0 keeps the old value)

// minimum over aligned groups of k lanes (k a power of two, 1 .. 64, uniform);
// every lane of a group receives the group's minimum
template <class T> __device__ __forceinline__ T group_min(T v, int k)
{
    // nested, so that a runtime k stops at the first level that does not apply
    T u;
    if (k >= 2) {
        u = dpp<kDppXor1>(v); v = u < v ? u : v;
        if (k >= 4) {
            u = dpp<kDppXor2>(v); v = u < v ? u : v;
            if (k >= 8) {
                u = dpp<kDppHalfMirror>(v); v = u < v ? u : v;
                if (k >= 16) {
                    u = dpp<kDppMirror>(v); v = u < v ? u : v;
                    if (k >= 32) {                   // rows of 16 combined through scalar reads
                        const int lane = __lane_id();
                        T r0 = (T)rl64((int64_t)v, 0), r1 = (T)rl64((int64_t)v, 16), r2 = (T)rl64((int64_t)v, 32),
                          r3 = (T)rl64((int64_t)v, 48);
                        if (k == 32) {
                            const T lo = r0 < r1 ? r0 : r1, hi = r2 < r3 ? r2 : r3;
                            v = lane < 32 ? lo : hi;
                        } else {
                            const T a = r0 < r1 ? r0 : r1, b = r2 < r3 ? r2 : r3;
                            v = a < b ? a : b;
                        }
                    }
                }
            }
        }
    }
    return v;
}

// inclusive prefix sum over the wavefront: row_shr 1, 2, 4 and 8 within rows
// of 16 (a lane without a source adds 0), then row_bcast 15 carries row 0's
// total into row 1 and row 2's into row 3, and row_bcast 31 carries the total
// of rows 0 and 1 into rows 2 and 3
__device__ __forceinline__ int wave_inclusive_sum(int v)
{
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);
    v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);
    v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);
    return v;
}

// sum over the wavefront, in every lane (pairs across the halves of groups of
// 2, 4, 8, 16 lanes, then the four rows of 16 through scalar reads)
__device__ __forceinline__ uint32_t wave_sum(uint32_t v)
{
    v += dpp32<kDppXor1>(v);
    v += dpp32<kDppXor2>(v);
    v += dpp32<kDppHalfMirror>(v);
    v += dpp32<kDppMirror>(v);
    return (uint32_t)rl32((int)v, 0) + (uint32_t)rl32((int)v, 16) + (uint32_t)rl32((int)v, 32) +
           (uint32_t)rl32((int)v, 48);
}

// Nearest value with at most 24 significant bits (ties to even) of a
// non-negative integer below 2^63: its fp32 rounding, kept as an exact integer.
__device__ __forceinline__ uint64_t rne24(uint64_t x)
{
    if (x < (1ull << 24)) return x;
    const int sh = 40 - __clzll(x);            // bits dropped: top bit lands at position 23
    const uint64_t q = x >> sh, r = x & ((1ull << sh) - 1), half = 1ull << (sh - 1);
    const uint64_t qr = q + ((r > half || (r == half && (q & 1))) ? 1 : 0);
    return qr << sh;
}

// float of an integer with at most 24 significant bits, times 2^e
__device__ __forceinline__ float exact_float(uint64_t x, int e)
{
    if (x == 0) return 0.0f;
    const int sh = x < (1ull << 24) ? 0 : 40 - __clzll(x);
    return ldexpf((float)(uint32_t)(x >> sh), sh + e);
}

// the integer x with x * 2^e == v, for a float v that is such a multiple
__device__ __forceinline__ uint64_t fixed_of_float(float v, int e)
{
    if (v == 0.0f) return 0;
    int ex;
    const float fr = frexpf(v, &ex);                         // v = fr * 2^ex, 0.5 <= fr < 1
    const uint64_t mant = (uint64_t)ldexpf(fr, 24);          // exact 24-bit integer
    const int sh = ex - 24 - e;
    return sh >= 0 ? mant << sh : mant >> (-sh);
}

__device__ __forceinline__ int nibble(uint64_t w, int l) { return (int)((w >> (4 * l)) & 15); }

template <class V> struct Vec2;
template <> struct Vec2<uint32_t> { typedef uint32_t type __attribute__((ext_vector_type(2))); };
template <> struct Vec2<uint64_t> { typedef uint64_t type __attribute__((ext_vector_type(2))); };
template <class V> struct DPInf { static constexpr V value = ~V(0); };

// all-to-all variant of a stage: none (EP = 1), inside one node, across nodes

}  // namespace heddle
