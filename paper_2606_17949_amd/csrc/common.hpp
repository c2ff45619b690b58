// Device helpers shared by the routing kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rb {

constexpr int WAVE = 64;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// Order-preserving map from fp32 to uint32: a < b (as floats, non-NaN) iff
// key(a) < key(b) as unsigned integers. Used so that distances can be compared,
// selected bit by bit and combined with atomicMin as plain integers.
__device__ __forceinline__ uint32_t f2key(float f)
{
    uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key2f(uint32_t k)
{
    uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
    return __uint_as_float(u);
}

constexpr uint32_t KEY_NONE = 0xffffffffu;   // larger than the key of any finite distance
constexpr int32_t IDX_NONE = 0x7fffffff;

__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }

__device__ __forceinline__ int popc(uint64_t m) { return __builtin_popcountll(m); }

// Number of set bits of m below this lane.
__device__ __forceinline__ int mbcnt(uint64_t m)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (WAVE - 1); }

// bf16 bits -> fp32 (exact).
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Lane exchange by DPP: x of the lane that control CTRL names (rows outside
// ROW_MASK keep their own x).
template <int CTRL, int ROW_MASK = 0xf, typename T>
__device__ __forceinline__ T dpp(T x)
{
    static_assert(sizeof(T) == 4, "32-bit values");
    const int xi = __builtin_bit_cast(int, x);
    if constexpr (ROW_MASK == 0xf)   // every lane has a source: no old value needed
        return __builtin_bit_cast(T, __builtin_amdgcn_mov_dpp(xi, CTRL, 0xf, 0xf, true));
    else
        return __builtin_bit_cast(T, __builtin_amdgcn_update_dpp(xi, xi, CTRL, ROW_MASK, 0xf, false));
}

// Butterfly inside each row of 16 lanes (quad permutes, then half-row and row
// mirrors): every lane ends with its row's result.
template <typename T, typename F>
__device__ __forceinline__ T row16_reduce(T v, F op)
{
    v = op(v, dpp<0xb1>(v));    // quad_perm [1,0,3,2]
    v = op(v, dpp<0x4e>(v));    // quad_perm [2,3,0,1]
    v = op(v, dpp<0x141>(v));   // row_half_mirror
    v = op(v, dpp<0x140>(v));   // row_mirror
    return v;
}

// Wave-wide reductions: the row butterfly, then the row_bcast:15 and
// row_bcast:31 steps carry rows 0..2 into row 3; lane 63 ends with the whole
// wave's result, which is broadcast through a scalar register.
template <typename T, typename F>
__device__ __forceinline__ T wave_reduce(T v, F op)
{
    v = row16_reduce(v, op);
    v = op(v, dpp<0x142, 0xa>(v));   // row_bcast:15 into rows 1 and 3
    v = op(v, dpp<0x143, 0xc>(v));   // row_bcast:31 into rows 2 and 3
    return __builtin_bit_cast(T, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// Lexicographic maximum of (hi, lo) pairs: over each row of 16 lanes when
// WIDTH is 16 (every lane ends with its row's pair), over the wave when it is
// 64 (broadcast to every lane).
template <int WIDTH>
__device__ __forceinline__ void reduce_max_pair(uint32_t &hi, uint32_t &lo)
{
    auto step = [&](uint32_t oh, uint32_t ol) {
        // one 64-bit compare, two selects (no branches)
        const bool take = (((uint64_t)oh << 32) | ol) > (((uint64_t)hi << 32) | lo);
        hi = take ? oh : hi;
        lo = take ? ol : lo;
    };
    step(dpp<0xb1>(hi), dpp<0xb1>(lo));
    step(dpp<0x4e>(hi), dpp<0x4e>(lo));
    step(dpp<0x141>(hi), dpp<0x141>(lo));
    step(dpp<0x140>(hi), dpp<0x140>(lo));
    if constexpr (WIDTH == 64) {
        step(dpp<0x142, 0xa>(hi), dpp<0x142, 0xa>(lo));
        step(dpp<0x143, 0xc>(hi), dpp<0x143, 0xc>(lo));
        hi = (uint32_t)__builtin_amdgcn_readlane((int)hi, 63);
        lo = (uint32_t)__builtin_amdgcn_readlane((int)lo, 63);
    }
}

template <typename F>
__device__ __forceinline__ float wave_reduce_f(float v, F op)
{
    return wave_reduce(v, op);
}

template <typename F>
__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t v, F op)
{
    return wave_reduce(v, op);
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v)
{
    return wave_reduce_u32(v, [](uint32_t a, uint32_t b) { return a > b ? a : b; });
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v)
{
    return wave_reduce_u32(v, [](uint32_t a, uint32_t b) { return a < b ? a : b; });
}

__device__ __forceinline__ float wave_max(float v)
{
    return wave_reduce_f(v, [](float a, float b) { return fmaxf(a, b); });
}

__device__ __forceinline__ float wave_sum(float v)
{
    return wave_reduce_f(v, [](float a, float b) { return a + b; });
}

}  // namespace rb
