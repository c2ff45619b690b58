// Helpers and argument blocks shared by the k-NN kernels (gfx950, wave64).
#pragma once

#include <float.h>

#include "common.hpp"
#include "kernels.hpp"

namespace rb {

struct ScanArgs {
    const uint8_t *queries, *bank;
    const float *bank_norms, *qn;
    int B, N, d, k, nks, nksp, n_chunks, n_qt;
    long rows_per_chunk;
    long row_lo, row_hi;      // query-resident scan: rows [row_lo, row_hi) of every chunk;
    int n_lists, list_base;   // its lists: list_base + c*RS + half of n_lists per query
    uint32_t *tau;    // [B] shared bound (distance keys), lowered with atomicMin
    int32_t *ccnt;    // [B][lists] list lengths
    uint32_t *ckey;   // [B][lists][k]
    int32_t *cidx;    // [B][lists][k]
    uint32_t *ovf;    // per wave: [3][ovf_cap] candidates past the LDS staging area
    int ovf_cap;      // 16*RT*16*NG - STAGE_CAP (every (row, query) pair of an iteration)
};

// Byte offsets of the scan's LDS regions for a tile of ng query groups of
// which the first gr are resident for the whole kernel, with a ring of
// `slots` k-steps for the others.
struct ScanLayout {
    uint32_t res, strm, list, qn, gb, lmk, nu, nx, sq, sk, si, bytes;
};

__host__ __device__ inline ScanLayout scan_layout(int ng, int gr, int nksp, int k, int rt, int slots)
{
    ScanLayout L;
    const uint32_t bm = (uint32_t)ng * 16, frag = WAVE * 16;
    uint32_t o = 0;
    L.res = o;     // [nksp][gr][64] fragments of the resident groups, every k-step
    o += (uint32_t)nksp * gr * frag;
    L.strm = o;    // [slots][ng - gr][64] fragments of the other groups, one k-step per
    // slot, and a sink fragment for loads with no destination
    o += gr < ng ? (uint32_t)(slots * (ng - gr) + 1) * frag : 0u;
    L.list = o;    // [bm][k] (key << 32 | index), the workgroup's candidate lists
    o += bm * k * 8;
    L.qn = o;      // [bm] |q|^2
    o += bm * 4;
    L.gb = o;      // [bm] snapshot of the shared bound
    o += bm * 4;
    L.lmk = o;     // [bm] an upper bound of each list's largest key
    o += bm * 4;
    L.nu = o;      // [bm] each query's candidate threshold on the accumulators
    o += bm * 4;
    L.nx = o;      // [waves][2][16*rt] -|x|^2/2 of this and the next iteration's rows
    o += SCAN_WAVES * 2 * rt * 16 * 4;
    L.sq = o;      // [waves][STAGE_CAP] staged candidates: tile query,
    o += SCAN_WAVES * STAGE_CAP * 4;
    L.sk = o;      //   distance key,
    o += SCAN_WAVES * STAGE_CAP * 4;
    L.si = o;      //   bank row
    o += SCAN_WAVES * STAGE_CAP * 4;
    L.bytes = o;
    return L;
}

// Byte offsets of the query-resident scan's LDS regions.
struct RqLayout {
    uint32_t ring, norms, lists, qinfo, bytes;
};

__host__ __device__ inline RqLayout rq_layout(int k, int qw, int kstg, int stages)
{
    RqLayout L;
    uint32_t o = 0;
    L.ring = o;    // [stages][kstg * RQ_ROWS / 16][64] bank fragments
    o += (uint32_t)stages * kstg * (RQ_ROWS / 16) * WAVE * 16;
    L.norms = o;   // [stages][64] |x|^2 of the rows of a block (with its first stage)
    o += (uint32_t)stages * WAVE * 4;
    L.lists = o;   // [waves][16 * qw][k] (key << 32 | index), one list per owned query
    o += (uint32_t)RQ_WAVES * qw * 16 * k * 8;
    L.qinfo = o;   // [waves][16 * qw] |q|^2, then [waves][16 * qw] the shared bound
    o += (uint32_t)RQ_WAVES * qw * 16 * 8;
    L.bytes = o;
    return L;
}

// Byte offsets of the GEMM-structured scan's LDS regions.
struct GemmLayout {
    uint32_t ring, norms, list, qn, gb, lmk, nu, sq, sk, si, bytes;
};

__host__ __device__ inline GemmLayout gemm_layout(int k)
{
    GemmLayout L;
    uint32_t o = 0;
    L.ring = o;    // [GM_SLOTS][2 * GM_ROWS / 8][64] row and request fragments of a stage
    o += (uint32_t)GM_SLOTS * (2 * GM_ROWS / 8) * WAVE * 16;
    L.norms = o;   // [2][GM_ROWS] |x|^2 of a macro tile's rows
    o += 2u * GM_ROWS * 4;
    L.list = o;    // [GM_QRY][k] (key << 32 | index), the workgroup's candidate lists
    o += (uint32_t)GM_QRY * k * 8;
    L.qn = o;      // [GM_QRY] |q|^2
    o += GM_QRY * 4;
    L.gb = o;      // [GM_QRY] snapshot of the shared bound
    o += GM_QRY * 4;
    L.lmk = o;     // [GM_QRY] an upper bound of each list's largest key
    o += GM_QRY * 4;
    L.nu = o;      // [GM_QRY] each request's candidate threshold on the accumulators
    o += GM_QRY * 4;
    L.sq = o;      // [waves][GM_STAGE] staged candidates: tile request,
    o += GM_WAVES * GM_STAGE * 4;
    L.sk = o;      //   distance key,
    o += GM_WAVES * GM_STAGE * 4;
    L.si = o;      //   bank row
    o += GM_WAVES * GM_STAGE * 4;
    L.bytes = o;
    return L;
}

// The bank-scan launchers, one translation unit per element type and
// k-step raggedness (they are the bulk of the compile time), and one per row
// length for the query-resident scan.
hipError_t launch_scan_gemm(const KnnPlan &p, const ScanArgs &a, hipStream_t s);
hipError_t launch_scan_rq(const KnnPlan &p, const ScanArgs &a, hipStream_t s);
hipError_t launch_scan_rq12(const KnnPlan &p, const ScanArgs &a, hipStream_t s);
hipError_t launch_scan_rq16(const KnnPlan &p, const ScanArgs &a, hipStream_t s);
hipError_t launch_scan_rq24(const KnnPlan &p, const ScanArgs &a, hipStream_t s);
hipError_t launch_scan_rq32(const KnnPlan &p, const ScanArgs &a, hipStream_t s);
hipError_t launch_scan_bf16(const KnnPlan &p, const ScanArgs &a, hipStream_t s);
hipError_t launch_scan_bf16_ragged(const KnnPlan &p, const ScanArgs &a, hipStream_t s);
hipError_t launch_scan_f32(const KnnPlan &p, const ScanArgs &a, hipStream_t s);
hipError_t launch_scan_f32_ragged(const KnnPlan &p, const ScanArgs &a, hipStream_t s);

namespace {

template <int DT> struct Elem;
template <> struct Elem<0> { static constexpr int VEC = 4, ESZ = 4; };   // fp32
template <> struct Elem<1> { static constexpr int VEC = 8, ESZ = 2; };   // bf16

constexpr int KSTEP_BYTES = 64;   // bytes of one row in one k-step (4 lanes x 16 bytes)

// Sum of squares of the 16-byte group held in v, added to s in element order.
template <int DT>
__device__ __forceinline__ float sumsq16(const i32x4 &v, float s)
{
    if constexpr (DT == 1) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t w = (uint32_t)v[e];
            const float x0 = bf16lo(w), x1 = bf16hi(w);
            s = fmaf(x0, x0, s);
            s = fmaf(x1, x1, s);
        }
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float x = __int_as_float(v[e]);
            s = fmaf(x, x, s);
        }
    }
    return s;
}

// One 16x16 MFMA tile step over 16 bytes of K per lane, D = A*B + C:
//   bf16: one v_mfma_f32_16x16x32_bf16 (8 elements per lane)
//   fp32: four v_mfma_f32_16x16x4_f32 (element e of every lane in step e)
// A and B hold the same K positions in the same lanes, so the dot products
// come out right whatever order the hardware assigns K within a step.
template <int DT>
__device__ __forceinline__ f32x4 mfma_step(const i32x4 &a, const i32x4 &b, const f32x4 &c)
{
    if constexpr (DT == 1) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    } else {
        f32x4 d = c;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            d = __builtin_amdgcn_mfma_f32_16x16x4f32(__int_as_float(a[e]), __int_as_float(b[e]), d,
                                                     0, 0, 0);
        return d;
    }
}

__device__ __forceinline__ i32x4 load16(const uint8_t *p) { return *(const i32x4 *)p; }

// Raw buffer resource over [base, base + bytes): loads at or past the end
// return zero, which masks rows past a chunk and queries past the batch.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ __forceinline__ i32x4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t voffset)
{
    return __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voffset, 0, 0));
}

constexpr uint32_t OFF_NONE = 0x80000000u;   // a buffer offset past any resource

// Global -> LDS load of 16 bytes per lane through the buffer resource: lane l's
// bytes land at dst + 16*l (dst is the same for the whole wave); a lane whose
// offset falls outside the resource writes zeros. Completion is counted by
// the wave's vector memory counter, like a load into registers.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, i32x4 *dst, uint32_t voffset)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void *)dst, 16,
                                             (int)voffset, 0, 0, 0);
}

// Wait until at most N vector memory operations of this wave are outstanding
// (they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "the counter has six bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

template <int I> struct Int {
    static constexpr int value = I;
};
template <bool V> struct Bool {
    static constexpr bool value = V;
};

// f(Int<I>) for I = B..E-1, unrolled at compile time.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F &&f)
{
    if constexpr (B < E) {
        f(Int<B>{});
        static_for<B + 1, E>(f);
    }
}

// Workgroup barrier that orders LDS only (waits for this wave's LDS traffic),
// leaving global loads in flight across it.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Workgroup barrier once this wave's LDS reads have returned, with no release
// fence (which would also wait for the wave's global-to-LDS loads still in
// flight); the acquire fence keeps later LDS accesses below it.
__device__ __forceinline__ void stream_barrier()
{
    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ uint32_t lds_load_relaxed(const uint32_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ void lds_store_relaxed(uint32_t *p, uint32_t v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ uint64_t pack(uint32_t key, int32_t idx)
{
    return ((uint64_t)key << 32) | (uint32_t)idx;
}

// 64-bit compare-and-swap in LDS; true when *p held `expect` and now holds `v`.
__device__ __forceinline__ bool lds_cas64(uint64_t *p, uint64_t expect, uint64_t v)
{
    return atomicCAS((unsigned long long *)p, (unsigned long long)expect,
                     (unsigned long long)v) == (unsigned long long)expect;
}

__device__ __forceinline__ uint64_t lds_load64(const uint64_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Inclusive prefix sum over the wave.
__device__ __forceinline__ int wave_incl_scan(int v)
{
    const int lane = lane_id();
#pragma unroll
    for (int m = 1; m < WAVE; m <<= 1) {
        const int o = __shfl_up(v, m);
        if (lane >= m)
            v += o;
    }
    return v;
}

__device__ __forceinline__ int wave_sum_int(int v)
{
#pragma unroll
    for (int m = 1; m < WAVE; m <<= 1)
        v += __shfl_xor(v, m);
    return v;
}

}  // namespace

}  // namespace rb
