// Exact k-nearest-neighbour search over the labelled reference bank
// (RouteBalance Sec. 4.2: the KNN lookup of Alg. 1), for gfx950.
//
// Data flow of one call:
//   knn_init_kernel   per query: |q|^2 and the shared distance bound <- +inf
//   scan_kernel       one workgroup per (bank chunk, query tile): bank rows
//                     stream from HBM straight into MFMA A operands, the query
//                     tile sits in LDS as MFMA B fragments; each 128-row
//                     distance tile is filtered against the per-query bound and
//                     survivors are merged into a per-query top-k list in LDS;
//                     the chunk's lists go to the workspace
//   merge_kernel      per query: the k smallest of all chunk lists, sorted,
//                     optionally followed by the label gather and average
//                     (Sec. 4.2: one lookup predicts quality and length for
//                     every model)
// Order everywhere: distance ascending, equal distances by the lower bank index.
#include "common.hpp"
#include "kernels.hpp"

namespace rb {

namespace {

constexpr int KB = 8;   // k-steps whose bank loads are issued together

template <int DT> struct Elem;
template <> struct Elem<0> { static constexpr int VEC = 4, ESZ = 4; };   // fp32
template <> struct Elem<1> { static constexpr int VEC = 8, ESZ = 2; };   // bf16

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

// One 16x16 MFMA tile step over 16 bytes of K per lane:
//   bf16: one v_mfma_f32_16x16x32_bf16 (8 elements per lane)
//   fp32: four v_mfma_f32_16x16x4_f32 (element e of every lane in step e)
// A and B hold the same K positions in the same lanes, so the dot products
// come out right whatever order the hardware assigns K within a step.
template <int DT>
__device__ __forceinline__ void mfma_step(const i32x4 &a, const i32x4 &b, f32x4 &c)
{
    if constexpr (DT == 1) {
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                    __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            c = __builtin_amdgcn_mfma_f32_16x16x4f32(__int_as_float(a[e]), __int_as_float(b[e]), c,
                                                     0, 0, 0);
    }
}

// Squared norms of rows, one wave per row, 16-byte lanes, fixed reduction tree.
template <int DT>
__global__ __launch_bounds__(256) void bank_norms_kernel(const uint8_t *__restrict__ bank, int N,
                                                         int d, float *__restrict__ norms)
{
    const int lane = lane_id();
    const long wave_g = ((long)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const long n_waves = ((long)gridDim.x * blockDim.x) >> 6;
    const int row_bytes = d * Elem<DT>::ESZ;
    for (long n = wave_g; n < N; n += n_waves) {
        const uint8_t *row = bank + n * row_bytes;
        float s = 0.f;
        for (int off = lane * 16; off < row_bytes; off += WAVE * 16)
            s = sumsq16<DT>(*(const i32x4 *)(row + off), s);
        s = wave_sum(s);
        if (lane == 0)
            norms[n] = s;
    }
}

// Per query: |q|^2 (same arithmetic as the bank norms) and the shared bound.
template <int DT>
__global__ __launch_bounds__(256) void knn_init_kernel(const uint8_t *__restrict__ queries, int B,
                                                       int d, float *__restrict__ qn,
                                                       uint32_t *__restrict__ tau)
{
    const int lane = lane_id();
    const int b = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    if (b >= B)
        return;
    const int row_bytes = d * Elem<DT>::ESZ;
    const uint8_t *row = queries + (size_t)b * row_bytes;
    float s = 0.f;
    for (int off = lane * 16; off < row_bytes; off += WAVE * 16)
        s = sumsq16<DT>(*(const i32x4 *)(row + off), s);
    s = wave_sum(s);
    if (lane == 0) {
        qn[b] = s;
        tau[b] = KEY_NONE;
    }
}

struct ScanArgs {
    const uint8_t *queries, *bank;
    const float *bank_norms, *qn;
    int B, N, d, k, nks, n_chunks, n_qt;
    long rows_per_chunk;
    uint32_t *tau;
    uint32_t *pkey;
    int32_t *pidx;
};

// Keys of the k smallest entries of the union of three per-lane slots, under
// (key, index). Returns T, the k-th smallest key, and U: entries with key == T
// are kept iff their index <= U. Needs at least k valid entries. Bitwise
// selection from the most significant bit, counting with ballots; the loop
// bounds and every branch are wave-uniform.
__device__ __forceinline__ void select_k(uint32_t ka, int32_t ia, bool va, uint32_t kb, int32_t ib,
                                         bool vb, uint32_t kc, int32_t ic, bool vc, int k,
                                         uint32_t &T, int32_t &U)
{
    uint32_t prefix = 0;
    for (int bit = 31; bit >= 0; --bit) {
        const uint32_t trial = prefix | (1u << bit);
        const int c = popc(ballot(va && ka < trial)) + popc(ballot(vb && kb < trial)) +
                      popc(ballot(vc && kc < trial));
        if (c < k)
            prefix = trial;
    }
    T = prefix;
    const int c_lt = popc(ballot(va && ka < T)) + popc(ballot(vb && kb < T)) +
                     popc(ballot(vc && kc < T));
    const int c_eq = popc(ballot(va && ka == T)) + popc(ballot(vb && kb == T)) +
                     popc(ballot(vc && kc == T));
    const int r = k - c_lt;
    U = IDX_NONE;
    if (c_eq > r) {
        uint32_t up = 0;
        for (int bit = 30; bit >= 0; --bit) {
            const uint32_t trial = up | (1u << bit);
            const int c = popc(ballot(va && ka == T && (uint32_t)ia < trial)) +
                          popc(ballot(vb && kb == T && (uint32_t)ib < trial)) +
                          popc(ballot(vc && kc == T && (uint32_t)ic < trial));
            if (c < r)
                up = trial;
        }
        U = (int32_t)up;
    }
}

template <int DT, int NG>
__global__ __launch_bounds__(SCAN_THREADS, 1) void scan_kernel(const ScanArgs A)
{
    constexpr int QT = NG * 16;
    constexpr int VEC = Elem<DT>::VEC;
    constexpr int ESZ = Elem<DT>::ESZ;
    extern __shared__ __align__(16) uint8_t smem[];
    const int k = A.k, nks = A.nks;
    i32x4 *qfrag = (i32x4 *)smem;                                  // [nks][NG][64]
    float *qn = (float *)(smem + (size_t)nks * NG * WAVE * 16);    // [QT]
    uint32_t *dtile = (uint32_t *)(qn + QT);                       // [QT][SCAN_DSTRIDE]
    uint32_t *lkey = dtile + QT * SCAN_DSTRIDE;                    // [QT][k]
    int32_t *lidx = (int32_t *)(lkey + QT * k);                    // [QT][k]
    int *lcnt = (int *)(lidx + QT * k);                            // [QT]
    uint32_t *ltau = (uint32_t *)(lcnt + QT);                      // [QT]

    // Workgroup -> (chunk c, query tile t). Workgroups are dispatched to the
    // eight XCDs round robin, so this map puts every query tile of one chunk
    // on the same XCD, where they share that chunk's lines in L2.
    const int per8 = 8 * A.n_qt;
    const int rem = blockIdx.x % per8;
    const int t = rem / 8;
    const int c = (blockIdx.x / per8) * 8 + rem % 8;
    if (c >= A.n_chunks)
        return;
    const int q0 = t * QT;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int jgrp = lane >> 4, col = lane & 15;
    const size_t row_bytes = (size_t)A.d * ESZ;

    // Query tile as B fragments: lane l of fragment (s, g) holds query
    // 16g + l%16, elements [s*4*VEC + (l/16)*VEC, +VEC). Zero past B and d.
    for (int f = tid; f < nks * NG * WAVE; f += SCAN_THREADS) {
        const int l = f & 63, g = (f >> 6) % NG, s = f / (NG * WAVE);
        const int q = q0 + g * 16 + (l & 15);
        const int kk = s * 4 * VEC + (l >> 4) * VEC;
        i32x4 v = {0, 0, 0, 0};
        if (q < A.B && kk < A.d)
            v = *(const i32x4 *)(A.queries + (size_t)q * row_bytes + (size_t)kk * ESZ);
        qfrag[f] = v;
    }
    for (int q = tid; q < QT; q += SCAN_THREADS) {
        qn[q] = (q0 + q < A.B) ? A.qn[q0 + q] : 0.f;
        lcnt[q] = 0;
        ltau[q] = KEY_NONE;
    }
    __syncthreads();

    const long rbeg = (long)c * A.rows_per_chunk;
    const long rend = min((long)A.N, rbeg + A.rows_per_chunk);
    for (long r0 = rbeg; r0 < rend; r0 += SCAN_RT) {
        const long wr0 = r0 + wave * SCAN_WR;
        f32x4 acc0[NG], acc1[NG];
#pragma unroll
        for (int g = 0; g < NG; ++g) {
            acc0[g] = f32x4{0.f, 0.f, 0.f, 0.f};
            acc1[g] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        if (wr0 < rend) {
            // A fragments: lane l holds bank row wr0 (+16) + l%16, the 16 bytes
            // at (l/16)*16 of each 64-byte k-step.
            const long ra = wr0 + col, rb = wr0 + 16 + col;
            const bool va = ra < rend, vb = rb < rend;
            const uint8_t *pa = A.bank + (size_t)(va ? ra : 0) * row_bytes + jgrp * 16;
            const uint8_t *pb = A.bank + (size_t)(vb ? rb : 0) * row_bytes + jgrp * 16;
            for (int s0 = 0; s0 < nks; s0 += KB) {
                i32x4 xa[KB], xb[KB];
#pragma unroll
                for (int u = 0; u < KB; ++u) {
                    const int s = s0 + u;
                    const bool kv = s < nks && s * 4 * VEC + jgrp * VEC < A.d;
                    const i32x4 z = {0, 0, 0, 0};
                    xa[u] = (va && kv) ? *(const i32x4 *)(pa + (size_t)s * 64) : z;
                    xb[u] = (vb && kv) ? *(const i32x4 *)(pb + (size_t)s * 64) : z;
                }
#pragma unroll
                for (int u = 0; u < KB; ++u) {
                    if (s0 + u < nks) {
#pragma unroll
                        for (int g = 0; g < NG; ++g) {
                            const i32x4 bq = qfrag[((s0 + u) * NG + g) * WAVE + lane];
                            mfma_step<DT>(xa[u], bq, acc0[g]);
                            mfma_step<DT>(xb[u], bq, acc1[g]);
                        }
                    }
                }
            }
        }
        // Accumulator layout: lane l, element e is bank row 4*(l/16)+e of the
        // 16-row tile against query 16g + l%16. Distance |q|^2 + |x|^2 - 2<q,x>.
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int rl = wave * SCAN_WR + h * 16 + jgrp * 4;
            float xn[4];
            bool rv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const long row = r0 + rl + e;
                rv[e] = row < rend;
                xn[e] = rv[e] ? A.bank_norms[row] : 0.f;
            }
#pragma unroll
            for (int g = 0; g < NG; ++g) {
                const int q = g * 16 + col;
                const float qq = qn[q];
                const f32x4 ac = h ? acc1[g] : acc0[g];
                i32x4 w;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    w[e] = rv[e] ? (int)f2key(fmaf(-2.f, ac[e], qq + xn[e])) : (int)KEY_NONE;
                *(i32x4 *)(dtile + q * SCAN_DSTRIDE + rl) = w;
            }
        }
        __syncthreads();

        // Selection: wave w owns queries w, w+4, ... A row survives if it beats
        // this chunk's current k-th (strictly: every listed row has a lower
        // index) and does not exceed the bound shared by all chunks (any
        // chunk's k-th smallest distance bounds the global k-th from above).
        for (int q = wave; q < QT; q += SCAN_WAVES) {
            if (q0 + q >= A.B)
                break;
            const uint32_t k0 = dtile[q * SCAN_DSTRIDE + lane];
            const uint32_t k1 = dtile[q * SCAN_DSTRIDE + WAVE + lane];
            const int32_t i0 = (int32_t)(r0 + lane), i1 = (int32_t)(r0 + WAVE + lane);
            const uint32_t lt = ltau[q];
            const uint32_t gt = __hip_atomic_load(A.tau + q0 + q, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
            const bool p0 = k0 < lt && k0 <= gt;
            const bool p1 = k1 < lt && k1 <= gt;
            const uint64_t m0 = ballot(p0), m1 = ballot(p1);
            if ((m0 | m1) == 0)
                continue;
            uint32_t *qk = lkey + q * k;
            int32_t *qi = lidx + q * k;
            const int cnt = lcnt[q];
            const bool pl = lane < cnt;
            const uint32_t kl = pl ? qk[lane] : KEY_NONE;
            const int32_t il = pl ? qi[lane] : IDX_NONE;
            const int n0 = popc(m0), n1 = popc(m1);
            const int total = cnt + n0 + n1;
            if (total < k) {
                if (p0) {
                    const int pos = cnt + mbcnt(m0);
                    qk[pos] = k0;
                    qi[pos] = i0;
                }
                if (p1) {
                    const int pos = cnt + n0 + mbcnt(m1);
                    qk[pos] = k1;
                    qi[pos] = i1;
                }
                if (lane == 0)
                    lcnt[q] = total;
                continue;
            }
            uint32_t T;
            int32_t U;
            select_k(kl, il, pl, k0, i0, p0, k1, i1, p1, k, T, U);
            const bool sl = pl && (kl < T || (kl == T && il <= U));
            const bool s0 = p0 && (k0 < T || (k0 == T && i0 <= U));
            const bool s1 = p1 && (k1 < T || (k1 == T && i1 <= U));
            const uint64_t ml = ballot(sl), ms0 = ballot(s0), ms1 = ballot(s1);
            // the old list is in registers; rewrite the k kept entries compactly
            if (sl) {
                const int pos = mbcnt(ml);
                qk[pos] = kl;
                qi[pos] = il;
            }
            if (s0) {
                const int pos = popc(ml) + mbcnt(ms0);
                qk[pos] = k0;
                qi[pos] = i0;
            }
            if (s1) {
                const int pos = popc(ml) + popc(ms0) + mbcnt(ms1);
                qk[pos] = k1;
                qi[pos] = i1;
            }
            if (lane == 0) {
                lcnt[q] = k;
                ltau[q] = T;
                if (T < gt)
                    atomicMin(A.tau + q0 + q, T);
            }
        }
        __syncthreads();
    }

    // This chunk's lists (unsorted, padded) -> workspace [B][n_chunks][k].
    for (int q = wave; q < QT; q += SCAN_WAVES) {
        if (q0 + q >= A.B)
            break;
        const int cnt = lcnt[q];
        for (int j = lane; j < k; j += WAVE) {
            const size_t o = ((size_t)(q0 + q) * A.n_chunks + c) * k + j;
            A.pkey[o] = j < cnt ? lkey[q * k + j] : KEY_NONE;
            A.pidx[o] = j < cnt ? lidx[q * k + j] : IDX_NONE;
        }
    }
}

struct MergeArgs {
    const uint32_t *pkey;
    const int32_t *pidx;
    const uint32_t *tau;
    int n_chunks, k;
    int32_t *nbr_idx;
    float *nbr_dist;
    const float *qual, *len;
    int N, M;
    float *q_hat, *l_hat;
};

// Block-wide count: one barrier per call (two alternating slots).
__device__ __forceinline__ int block_count(int c, int *red, int &phase)
{
    const float s = wave_sum((float)c);
    int *slot = red + (phase & 1) * 4;
    if (lane_id() == 0)
        slot[threadIdx.x >> 6] = (int)s;
    __syncthreads();
    ++phase;
    return slot[0] + slot[1] + slot[2] + slot[3];
}

// The label gather and average: sum over neighbours j = 0..k-1 in order. A
// neighbour index outside [0, N) makes both averages NaN instead of reading
// out of bounds.
__device__ __forceinline__ void average_labels(const int32_t *nbr, int k, const float *qual,
                                               const float *len, int N, int M, int m,
                                               float *q_out, float *l_out)
{
    float sq = 0.f, sl = 0.f;
    for (int j = 0; j < k; ++j) {
        const int32_t n = nbr[j];
        if (n < 0 || n >= N) {
            sq = sl = __builtin_nanf("");
            break;
        }
        const size_t o = (size_t)n * M + m;
        sq += qual[o];
        sl += len[o];
    }
    *q_out = sq / (float)k;
    *l_out = sl / (float)k;
}

template <int EPT, bool PREDICT>
__global__ __launch_bounds__(MERGE_THREADS) void merge_kernel(const MergeArgs A)
{
    __shared__ int red[8];
    __shared__ uint32_t skey[RB_MAX_K_DEV];
    __shared__ int32_t sidx[RB_MAX_K_DEV];
    __shared__ int32_t sorted_idx[RB_MAX_K_DEV];
    __shared__ int scount;
    const int b = blockIdx.x, tid = threadIdx.x, k = A.k;
    const int E = A.n_chunks * k;
    const uint32_t *pk = A.pkey + (size_t)b * E;
    const int32_t *pi = A.pidx + (size_t)b * E;
    const uint32_t bound = A.tau[b];
    uint32_t key[EPT];
    int32_t idx[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        const int j = e * MERGE_THREADS + tid;
        key[e] = KEY_NONE;
        idx[e] = IDX_NONE;
        if (j < E) {
            const uint32_t kk = pk[j];
            if (kk <= bound) {   // rows above the final bound cannot be among the k nearest
                key[e] = kk;
                idx[e] = pi[j];
            }
        }
    }
    if (tid == 0)
        scount = 0;
    if (tid < k)
        sorted_idx[tid] = IDX_NONE;
    int phase = 0;
    // T = k-th smallest key
    uint32_t prefix = 0;
    for (int bit = 31; bit >= 0; --bit) {
        const uint32_t trial = prefix | (1u << bit);
        int c = 0;
#pragma unroll
        for (int e = 0; e < EPT; ++e)
            c += (idx[e] != IDX_NONE && key[e] < trial);
        if (block_count(c, red, phase) < k)
            prefix = trial;
    }
    const uint32_t T = prefix;
    int c_lt = 0, c_eq = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        c_lt += (idx[e] != IDX_NONE && key[e] < T);
        c_eq += (idx[e] != IDX_NONE && key[e] == T);
    }
    c_lt = block_count(c_lt, red, phase);
    c_eq = block_count(c_eq, red, phase);
    const int r = k - c_lt;
    int32_t U = IDX_NONE;
    if (c_eq > r) {
        uint32_t up = 0;
        for (int bit = 30; bit >= 0; --bit) {
            const uint32_t trial = up | (1u << bit);
            int c = 0;
#pragma unroll
            for (int e = 0; e < EPT; ++e)
                c += (idx[e] != IDX_NONE && key[e] == T && (uint32_t)idx[e] < trial);
            if (block_count(c, red, phase) < r)
                up = trial;
        }
        U = (int32_t)up;
    }
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        if (idx[e] != IDX_NONE && (key[e] < T || (key[e] == T && idx[e] <= U))) {
            const int pos = atomicAdd(&scount, 1);
            skey[pos] = key[e];
            sidx[pos] = idx[e];
        }
    }
    __syncthreads();
    // exactly k entries; order them by (key, index)
    if (tid < k) {
        const uint32_t mk = skey[tid];
        const int32_t mi = sidx[tid];
        int rank = 0;
        for (int j = 0; j < k; ++j)
            rank += (skey[j] < mk || (skey[j] == mk && sidx[j] < mi));
        A.nbr_idx[(size_t)b * k + rank] = mi;
        if (A.nbr_dist)
            A.nbr_dist[(size_t)b * k + rank] = key2f(mk);
        sorted_idx[rank] = mi;
    }
    if constexpr (PREDICT) {
        __syncthreads();
        for (int m = tid; m < A.M; m += MERGE_THREADS)
            average_labels(sorted_idx, k, A.qual, A.len, A.N, A.M, m,
                           A.q_hat + (size_t)b * A.M + m, A.l_hat + (size_t)b * A.M + m);
    }
}

__global__ __launch_bounds__(64) void predict_kernel(const int32_t *__restrict__ nbr_idx, int k,
                                                     const float *__restrict__ qual,
                                                     const float *__restrict__ len, int N, int M,
                                                     float *__restrict__ q_hat,
                                                     float *__restrict__ l_hat)
{
    __shared__ int32_t nbr[RB_MAX_K_DEV];
    const int b = blockIdx.x;
    for (int j = threadIdx.x; j < k; j += blockDim.x)
        nbr[j] = nbr_idx[(size_t)b * k + j];
    __syncthreads();
    for (int m = threadIdx.x; m < M; m += blockDim.x)
        average_labels(nbr, k, qual, len, N, M, m, q_hat + (size_t)b * M + m,
                       l_hat + (size_t)b * M + m);
}

template <int DT, int NG>
hipError_t launch_scan(const ScanArgs &a, size_t lds, int grid, hipStream_t s)
{
    hipError_t e = hipFuncSetAttribute((const void *)scan_kernel<DT, NG>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL((scan_kernel<DT, NG>), dim3(grid), dim3(SCAN_THREADS), lds, s, a);
    return hipGetLastError();
}

template <bool PRED>
hipError_t launch_merge(const MergeArgs &a, int B, int ept, hipStream_t s)
{
    switch (ept) {
    case 4: hipLaunchKernelGGL((merge_kernel<4, PRED>), dim3(B), dim3(MERGE_THREADS), 0, s, a); break;
    case 8: hipLaunchKernelGGL((merge_kernel<8, PRED>), dim3(B), dim3(MERGE_THREADS), 0, s, a); break;
    case 16: hipLaunchKernelGGL((merge_kernel<16, PRED>), dim3(B), dim3(MERGE_THREADS), 0, s, a); break;
    case 32: hipLaunchKernelGGL((merge_kernel<32, PRED>), dim3(B), dim3(MERGE_THREADS), 0, s, a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

thread_local hipEvent_t t_scan_begin = nullptr, t_scan_end = nullptr;

}  // namespace

void set_scan_events(hipEvent_t begin, hipEvent_t end)
{
    t_scan_begin = begin;
    t_scan_end = end;
}

int plan_knn(int B, int N, int d, int dtype, int k, int num_cu, KnnPlan *p)
{
    const int vec = dtype == 1 ? 8 : 4;
    p->dtype = dtype;
    p->B = B;
    p->N = N;
    p->d = d;
    p->k = k;
    p->nks = (d + 4 * vec - 1) / (4 * vec);
    // largest query tile that is useful for B and fits in LDS
    const int b16 = (B + 15) / 16;
    p->ng = 0;
    for (int ng = 4; ng >= 1; ng >>= 1) {
        if (ng > 1 && ng > b16)
            continue;
        const int qt = ng * 16;
        const size_t lds = (size_t)p->nks * ng * WAVE * 16 + (size_t)qt * 4 +
                           (size_t)qt * SCAN_DSTRIDE * 4 + (size_t)qt * k * 8 + (size_t)qt * 8;
        if (lds <= LDS_LIMIT) {
            p->ng = ng;
            p->lds_bytes = lds;
            break;
        }
    }
    if (p->ng == 0)
        return -1;
    const int qt = p->ng * 16;
    p->n_qt = B > 0 ? (B + qt - 1) / qt : 1;
    // one workgroup per compute unit (the LDS use allows no more)
    int chunks = num_cu / p->n_qt;
    if (chunks < 1)
        chunks = 1;
    const int max_by_merge = MERGE_MAX_ENTRIES / k;
    if (chunks > max_by_merge)
        chunks = max_by_merge;
    const int max_by_rows = (N + 31) / 32;   // chunks of at least 32 rows
    if (chunks > max_by_rows)
        chunks = max_by_rows;
    if (chunks < 1)
        chunks = 1;
    p->n_chunks = chunks;
    p->rows_per_chunk = ((long)N + chunks - 1) / chunks;
    size_t off = 0;
    p->off_tau = off;
    off += align256((size_t)B * 4);
    const size_t off_qn = off;
    (void)off_qn;
    off += align256((size_t)B * 4);
    p->off_pkey = off;
    off += align256((size_t)B * chunks * k * 4);
    p->off_pidx = off;
    off += align256((size_t)B * chunks * k * 4);
    p->bytes = off;
    return 0;
}

hipError_t launch_bank_norms(const void *bank, int dtype, int N, int d, float *norms,
                             hipStream_t s)
{
    long waves = N;
    int grid = (int)((waves + 3) / 4);
    if (grid > 65536)
        grid = 65536;
    if (dtype == 1)
        hipLaunchKernelGGL(bank_norms_kernel<1>, dim3(grid), dim3(256), 0, s,
                           (const uint8_t *)bank, N, d, norms);
    else
        hipLaunchKernelGGL(bank_norms_kernel<0>, dim3(grid), dim3(256), 0, s,
                           (const uint8_t *)bank, N, d, norms);
    return hipGetLastError();
}

hipError_t launch_knn(const KnnPlan &p, const void *queries, const void *bank,
                      const float *bank_norms, void *ws, int32_t *nbr_idx, float *nbr_dist,
                      const float *bank_qual, const float *bank_len, int M, float *q_hat,
                      float *l_hat, hipStream_t s)
{
    uint8_t *w = (uint8_t *)ws;
    uint32_t *tau = (uint32_t *)(w + p.off_tau);
    float *qn = (float *)(w + p.off_tau + align256((size_t)p.B * 4));
    uint32_t *pkey = (uint32_t *)(w + p.off_pkey);
    int32_t *pidx = (int32_t *)(w + p.off_pidx);

    const int init_grid = (p.B + 3) / 4;
    if (p.dtype == 1)
        hipLaunchKernelGGL(knn_init_kernel<1>, dim3(init_grid), dim3(256), 0, s,
                           (const uint8_t *)queries, p.B, p.d, qn, tau);
    else
        hipLaunchKernelGGL(knn_init_kernel<0>, dim3(init_grid), dim3(256), 0, s,
                           (const uint8_t *)queries, p.B, p.d, qn, tau);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;

    ScanArgs a;
    a.queries = (const uint8_t *)queries;
    a.bank = (const uint8_t *)bank;
    a.bank_norms = bank_norms;
    a.qn = qn;
    a.B = p.B;
    a.N = p.N;
    a.d = p.d;
    a.k = p.k;
    a.nks = p.nks;
    a.n_chunks = p.n_chunks;
    a.n_qt = p.n_qt;
    a.rows_per_chunk = p.rows_per_chunk;
    a.tau = tau;
    a.pkey = pkey;
    a.pidx = pidx;
    const int grid = ((p.n_chunks + 7) / 8) * 8 * p.n_qt;
    const bool timed = t_scan_begin && t_scan_end;
    if (timed && (e = hipEventRecord(t_scan_begin, s)) != hipSuccess)
        return e;
    if (p.dtype == 1) {
        if (p.ng == 4) e = launch_scan<1, 4>(a, p.lds_bytes, grid, s);
        else if (p.ng == 2) e = launch_scan<1, 2>(a, p.lds_bytes, grid, s);
        else e = launch_scan<1, 1>(a, p.lds_bytes, grid, s);
    } else {
        if (p.ng == 4) e = launch_scan<0, 4>(a, p.lds_bytes, grid, s);
        else if (p.ng == 2) e = launch_scan<0, 2>(a, p.lds_bytes, grid, s);
        else e = launch_scan<0, 1>(a, p.lds_bytes, grid, s);
    }
    if (e != hipSuccess)
        return e;
    if (timed && (e = hipEventRecord(t_scan_end, s)) != hipSuccess)
        return e;

    MergeArgs m;
    m.pkey = pkey;
    m.pidx = pidx;
    m.tau = tau;
    m.n_chunks = p.n_chunks;
    m.k = p.k;
    m.nbr_idx = nbr_idx;
    m.nbr_dist = nbr_dist;
    m.qual = bank_qual;
    m.len = bank_len;
    m.N = p.N;
    m.M = M;
    m.q_hat = q_hat;
    m.l_hat = l_hat;
    const int E = p.n_chunks * p.k;
    int ept = 4;
    while (ept * MERGE_THREADS < E)
        ept *= 2;
    if (ept > MERGE_MAX_EPT)
        return hipErrorInvalidValue;
    return q_hat ? launch_merge<true>(m, p.B, ept, s) : launch_merge<false>(m, p.B, ept, s);
}

hipError_t launch_predict(const int32_t *nbr_idx, int B, int k, const float *bank_qual,
                          const float *bank_len, int N, int M, float *q_hat, float *l_hat,
                          hipStream_t s)
{
    hipLaunchKernelGGL(predict_kernel, dim3(B), dim3(64), 0, s, nbr_idx, k, bank_qual, bank_len,
                       N, M, q_hat, l_hat);
    return hipGetLastError();
}

}  // namespace rb
