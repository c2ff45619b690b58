// Exact k-nearest-neighbour search over the labelled reference bank
// (RouteBalance Sec. 4.2: the KNN lookup of Alg. 1), for gfx950.
//
// Kernels of one call:
//   seed_groups_kernel  distances of every query to S bank rows spread evenly
//                       over the bank; minima over groups of 16 of those rows
//   seed_bound_kernel   per query: |q|^2, and the k-th smallest group minimum
//                       as the starting bound of the k-th nearest distance
//   scan_kernel         the bank once through MFMA: one workgroup per (bank
//                       chunk, tile of up to 256 queries); bank rows go from
//                       HBM straight into MFMA operand registers, the query
//                       tile streams through an LDS double buffer along K; a
//                       register-level test against the per-query bound lets
//                       only candidates reach the per-wave top-k lists
//   merge_kernel        per query: the k nearest of all lists, sorted, then
//                       optionally the label gather and average (Sec. 4.2: one
//                       lookup predicts quality and length for every model)
// Order everywhere: distance ascending, equal distances by the lower bank
// index. Distances are |q|^2 + |x|^2 - 2<q,x> with fp32 products and
// accumulation; the scan accumulates -|x|^2/2 + <q,x> and reports
// |q|^2 - 2*acc.
#include <float.h>

#include "common.hpp"
#include "kernels.hpp"

namespace rb {

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

template <int I> struct Int {
    static constexpr int value = I;
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

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v)
{
#pragma unroll
    for (int m = 1; m < WAVE; m <<= 1) {
        const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, m);
        const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), m);
        const uint64_t o = ((uint64_t)hi << 32) | lo;
        v = o > v ? o : v;
    }
    return v;
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

// ------------------------------------------------------------------ norms

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
            s = sumsq16<DT>(load16(row + off), s);
        s = wave_sum(s);
        if (lane == 0)
            norms[n] = s;
    }
}

// ------------------------------------------------------------------ seed

struct SeedArgs {
    const uint8_t *queries, *bank;
    const float *bank_norms;
    int B, N, d, nks, S, G, n_qg;
    float *gmin;   // [B][G]
};

// Bank row of seed sample j: S rows spread evenly over [0, N).
__device__ __forceinline__ long seed_row(int j, int N, int S)
{
    return (long)j * N / S;
}

// One wave per (query group of 16, block of 64 sample rows): partial distances
// p = |x|^2 - 2<q,x> by MFMA, then each lane's minimum over its 16 rows. The
// 16 waves of a workgroup take 16 query groups of the same sample block, so
// the block's rows are fetched once into the compute unit's caches.
constexpr int SEED_WAVES = 16;

template <int DT>
__global__ __launch_bounds__(SEED_WAVES * WAVE) void seed_groups_kernel(const SeedArgs A)
{
    constexpr int VEC = Elem<DT>::VEC, ESZ = Elem<DT>::ESZ;
    const int lane = lane_id(), col = lane & 15, jg = lane >> 4;
    const int sb = blockIdx.x;
    const int qg = blockIdx.y * SEED_WAVES + (threadIdx.x >> 6);
    if (qg >= A.n_qg)
        return;
    const size_t rowb = (size_t)A.d * ESZ;
    const int q = qg * 16 + col;
    const bool qv = q < A.B;
    const uint8_t *qp = A.queries + (qv ? (size_t)q * rowb : 0) + jg * 16;
    const uint8_t *ap[4];
    f32x4 acc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        ap[t] = A.bank + (size_t)seed_row(sb * 64 + t * 16 + col, A.N, A.S) * rowb + jg * 16;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            acc[t][e] = -0.5f * A.bank_norms[seed_row(sb * 64 + t * 16 + jg * 4 + e, A.N, A.S)];
    }
    for (int s = 0; s < A.nks; ++s) {
        const bool kv = s * 4 * VEC + jg * VEC < A.d;
        const i32x4 z = {0, 0, 0, 0};
        const i32x4 b = kv && qv ? load16(qp + (size_t)s * KSTEP_BYTES) : z;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const i32x4 a = kv ? load16(ap[t] + (size_t)s * KSTEP_BYTES) : z;
            acc[t] = mfma_step<DT>(a, b, acc[t]);
        }
    }
    float m = INFINITY;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e)
            m = fminf(m, -2.f * acc[t][e]);
    if (qv)
        A.gmin[(size_t)q * A.G + sb * 4 + jg] = m;
}

// One wave per query: |q|^2, and the starting bound = |q|^2 + the k-th smallest
// group minimum, widened by a margin far above any fp32 rounding difference
// between this pass and the scan. Without a seed (G < k) the bound is +inf.
template <int DT, int GPL>
__global__ __launch_bounds__(256) void seed_bound_kernel(const uint8_t *__restrict__ queries, int B,
                                                         int d, int k, const float *__restrict__ gmin,
                                                         int G, float *__restrict__ qn,
                                                         uint32_t *__restrict__ tau)
{
    const int lane = lane_id();
    const int b = (int)(((long)blockIdx.x * blockDim.x + threadIdx.x) >> 6);
    if (b >= B)
        return;
    const int row_bytes = d * Elem<DT>::ESZ;
    const uint8_t *row = queries + (size_t)b * row_bytes;
    float s = 0.f;
    for (int off = lane * 16; off < row_bytes; off += WAVE * 16)
        s = sumsq16<DT>(load16(row + off), s);
    s = wave_sum(s);
    uint32_t T = KEY_NONE;
    if (G >= k) {
        uint32_t key[GPL];
#pragma unroll
        for (int u = 0; u < GPL; ++u) {
            const int i = lane + WAVE * u;
            key[u] = i < G ? f2key(gmin[(size_t)b * G + i]) : KEY_NONE;
        }
        uint32_t prefix = 0;
        for (int bit = 31; bit >= 0; --bit) {
            const uint32_t trial = prefix | (1u << bit);
            int c = 0;
#pragma unroll
            for (int u = 0; u < GPL; ++u)
                c += key[u] < trial;
            if ((int)wave_sum((float)c) < k)
                prefix = trial;
        }
        const float pk = key2f(prefix);
        const float t = s + pk;
        const float margin = ldexpf(s + fabsf(pk) + 1.f, -14);
        T = f2key(t + margin);
    }
    if (lane == 0) {
        qn[b] = s;
        tau[b] = T;
    }
}

// ------------------------------------------------------------------ scan

struct ScanArgs {
    const uint8_t *queries, *bank;
    const float *bank_norms, *qn;
    int B, N, d, k, nks, nksp, n_chunks, n_qt, W;
    long rows_per_chunk;
    uint32_t *tau;    // [B] shared bound (distance keys), lowered with atomicMin
    int32_t *ccnt;    // [B][W] list lengths
    uint32_t *ckey;   // [B][W][k]
    int32_t *cidx;    // [B][W][k]
};

template <int DT, int NG, int RT, bool RAGGED>
__global__ __launch_bounds__(SCAN_THREADS, 1) void scan_kernel(const ScanArgs A)
{
    constexpr int BM = NG * 16;
    constexpr int VEC = Elem<DT>::VEC, ESZ = Elem<DT>::ESZ;
    constexpr int KS = 4 * VEC;                    // elements of one k-step
    constexpr int RW = RT * 16;                    // rows per wave per iteration
    constexpr int RWG = SCAN_WAVES * RW;           // rows per workgroup iteration
    constexpr int QITEMS = NG * WAVE;              // 16-byte query items of one k-step
    constexpr int QPT = (QITEMS + SCAN_THREADS - 1) / SCAN_THREADS;
    constexpr int R = SCAN_UNROLL, P = SCAN_PREFETCH;
    static_assert(P < R, "prefetch distance must leave a free ring slot");
    static_assert(RW == WAVE, "one bank-norm load per lane per iteration");

    extern __shared__ __align__(16) uint8_t smem[];
    const int k = A.k;
    i32x4 *qbuf = (i32x4 *)smem;                                    // [2][NG][64]
    float *qn_s = (float *)(qbuf + 2 * QITEMS);                     // [BM]
    uint32_t *gb_s = (uint32_t *)(qn_s + BM);                       // [BM] shared-bound snapshot
    float *nx_all = (float *)(gb_s + BM);                           // [4][2][RW] -|x|^2/2
    uint32_t *lk_all = (uint32_t *)(nx_all + SCAN_WAVES * 2 * RW);  // [4][BM][k]
    int32_t *li_all = (int32_t *)(lk_all + SCAN_WAVES * BM * k);    // [4][BM][k]
    int *lc_all = (int *)(li_all + SCAN_WAVES * BM * k);            // [4][BM]
    uint32_t *lmk_all = (uint32_t *)(lc_all + SCAN_WAVES * BM);     // [4][BM] max key of a full list
    int32_t *lmi_all = (int32_t *)(lmk_all + SCAN_WAVES * BM);      // [4][BM] its index
    int *sq_all = (int *)(lmi_all + SCAN_WAVES * BM);               // [4][STAGE_CAP]
    uint32_t *sk_all = (uint32_t *)(sq_all + SCAN_WAVES * STAGE_CAP);
    int32_t *si_all = (int32_t *)(sk_all + SCAN_WAVES * STAGE_CAP);

    // Workgroup -> (chunk c, query tile t). Workgroups are dispatched to the
    // eight XCDs round robin, so this map puts every query tile of one chunk
    // on the same XCD, where they share that chunk's lines in L2.
    const int per8 = 8 * A.n_qt;
    const int rem = blockIdx.x % per8;
    const int t = rem / 8;
    const int c = (blockIdx.x / per8) * 8 + rem % 8;
    if (c >= A.n_chunks)
        return;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, jg = lane >> 4;
    const int q0 = t * BM;
    const long rbeg = (long)c * A.rows_per_chunk;
    const long rend = min((long)A.N, rbeg + A.rows_per_chunk);
    const int n_it = rend > rbeg ? (int)((rend - rbeg + RWG - 1) / RWG) : 0;
    const int nks = A.nks, nksp = A.nksp;
    const size_t rowb = (size_t)A.d * ESZ;

    float *nx = nx_all + wave * 2 * RW;
    uint32_t *lk = lk_all + wave * BM * k;
    int32_t *li = li_all + wave * BM * k;
    int *lc = lc_all + wave * BM;
    uint32_t *lmk = lmk_all + wave * BM;
    int32_t *lmi = lmi_all + wave * BM;
    int *sq = sq_all + wave * STAGE_CAP;
    uint32_t *sk = sk_all + wave * STAGE_CAP;
    int32_t *si = si_all + wave * STAGE_CAP;

    for (int i = tid; i < BM; i += SCAN_THREADS) {
        const int q = q0 + i;
        qn_s[i] = q < A.B ? A.qn[q] : 0.f;
        gb_s[i] = q < A.B ? A.tau[q] : 0u;
    }
    for (int i = tid; i < SCAN_WAVES * BM; i += SCAN_THREADS)
        lc_all[i] = 0;

    // ---- loads of one k-step through buffer resources whose base moves by one
    // k-step (64 bytes of a row) per step; each lane keeps a fixed offset. Rows
    // past the chunk and queries past the batch fall outside the resource and
    // load zero; so does every lane of a padding k-step (empty resource). The
    // query items run two k-steps ahead of the MFMAs, the bank rows three.
    const uint8_t *bank_c = A.bank + (size_t)rbeg * rowb;
    const uint32_t bank_c_bytes = (uint32_t)((rend - rbeg) * (long)rowb);
    const uint32_t q_bytes = (uint32_t)((size_t)A.B * rowb);
    uint32_t qvo[QPT];   // per item: q*rowb + (l/16)*16, or OFF_NONE
    int qkk[QPT];        // element offset of the item within a k-step
#pragma unroll
    for (int i = 0; i < QPT; ++i) {
        const int item = tid + SCAN_THREADS * i;
        const int f = item >> 6, l = item & 63;
        const int q = q0 + f * 16 + (l & 15);
        qkk[i] = (l >> 4) * VEC;
        qvo[i] = item < QITEMS ? (uint32_t)((size_t)q * rowb + (l >> 4) * 16) : OFF_NONE;
    }
    int pq_s = 0;             // k-step of the next query load (every iteration is the same)
    int pb_it = 0, pb_s = 0;  // k-step of the next bank load
    uint32_t bvo = (uint32_t)((size_t)(wave * RW + col) * rowb + jg * 16);   // tile 0 of pb_it
    auto issue_q = [&](i32x4(&qs)[QPT]) {
        const bool real = pq_s < nks;
        const __amdgpu_buffer_rsrc_t r =
            make_rsrc(A.queries + pq_s * KSTEP_BYTES, real ? q_bytes - pq_s * KSTEP_BYTES : 0u);
#pragma unroll
        for (int i = 0; i < QPT; ++i) {
            uint32_t vo = qvo[i];
            if constexpr (RAGGED)
                vo = pq_s * KS + qkk[i] < A.d ? vo : OFF_NONE;
            qs[i] = buffer_load16(r, vo);
        }
        if (++pq_s == nksp)
            pq_s = 0;
    };
    auto issue_b = [&](i32x4(&a)[RT]) {
        const bool real = pb_it < n_it && pb_s < nks;
        const __amdgpu_buffer_rsrc_t r = make_rsrc(
            bank_c + pb_s * KSTEP_BYTES, real ? bank_c_bytes - pb_s * KSTEP_BYTES : 0u);
        const bool lane_ok = !RAGGED || pb_s * KS + jg * VEC < A.d;
#pragma unroll
        for (int tt = 0; tt < RT; ++tt)
            a[tt] = buffer_load16(r, lane_ok ? bvo + (uint32_t)(tt * 16 * rowb) : OFF_NONE);
        if (++pb_s == nksp) {
            pb_s = 0;
            ++pb_it;
            bvo += (uint32_t)(RWG * rowb);
        }
    };
    auto stage_queries = [&](int slot, const i32x4(&qs)[QPT]) {
#pragma unroll
        for (int i = 0; i < QPT; ++i) {
            const int item = tid + SCAN_THREADS * i;
            if (item < QITEMS)
                qbuf[slot * QITEMS + item] = qs[i];
        }
    };
    // -|x|^2/2 of bank row `lane` of this wave in iteration it (-inf past the chunk)
    auto load_norm = [&](int it) -> float {
        const long row = rbeg + (long)it * RWG + wave * RW + lane;
        const bool v = it < n_it && row < rend;
        const float xn = A.bank_norms[v ? row : 0];
        return v ? -0.5f * xn : -INFINITY;
    };
    // Filter threshold of tile query i: a value is a candidate if acc >= nu (a
    // superset of distance <= the query's bound; the exact test follows on
    // insertion).
    auto nu_of = [&](int i) -> float {
        if (q0 + i >= A.B)
            return INFINITY;
        uint32_t tk = lds_load_relaxed(gb_s + i);
        if (lc[i] == k)
            tk = min(tk, lmk[i]);
        if (tk == KEY_NONE)
            return -FLT_MAX;
        const float qq = qn_s[i], th = key2f(tk);
        const float v = 0.5f * (qq - th);
        return v - ldexpf(fabsf(qq) + fabsf(th) + fabsf(v), -21);
    };
    auto recompute_max = [&](int i) {
        const uint64_t v = lane < k ? pack(lk[i * k + lane], li[i * k + lane]) : 0;
        const uint64_t m = wave_max_u64(v);
        if (lane == 0) {
            lmk[i] = (uint32_t)(m >> 32);
            lmi[i] = (int32_t)(uint32_t)m;
            atomicMin(A.tau + q0 + i, (uint32_t)(m >> 32));
        }
    };
    // Insert (key, idx) into this wave's list of tile query i (wave-uniform call).
    auto insert = [&](int i, uint32_t key, int32_t idx) {
        if (key > lds_load_relaxed(gb_s + i))
            return;
        const int n = lc[i];
        if (n < k) {
            if (lane == 0) {
                lk[i * k + n] = key;
                li[i * k + n] = idx;
                lc[i] = n + 1;
            }
            if (n + 1 == k)
                recompute_max(i);
            return;
        }
        const uint32_t mk = lmk[i];
        const int32_t mi = lmi[i];
        if (!(key < mk || (key == mk && idx < mi)))
            return;
        if (lane < k && lk[i * k + lane] == mk && li[i * k + lane] == mi) {
            lk[i * k + lane] = key;
            li[i * k + lane] = idx;
        }
        recompute_max(i);
    };
    auto flush = [&](int n) {
        for (int s = 0; s < n; ++s) {
            const int i = __builtin_amdgcn_readfirstlane(sq[s]);
            const uint32_t key = (uint32_t)__builtin_amdgcn_readfirstlane((int)sk[s]);
            const int32_t idx = __builtin_amdgcn_readfirstlane(si[s]);
            insert(i, key, idx);
        }
    };

    f32x4 acc[RT][NG];
    i32x4 ring[R][RT];
    i32x4 qst[2][QPT];
    int x = 0;   // global k-step index of the MFMAs
    const int total = n_it * nksp;

    // One block of R k-steps.
    auto block = [&]() {
#pragma unroll
        for (int u = 0; u < R; ++u) {
            if (x > 0)
                lds_barrier();
            if (x + 1 < total)
                stage_queries((u + 1) & 1, qst[(u + 1) & 1]);
            issue_q(qst[u & 1]);
            issue_b(ring[(u + P) % R]);
            const i32x4 *qb = qbuf + (u & 1) * QITEMS;
            i32x4 b = qb[lane];
#pragma unroll
            for (int g = 0; g < NG; ++g) {
                const i32x4 bn = qb[((g + 1) % NG) * WAVE + lane];   // next fragment, in flight
#pragma unroll
                for (int tt = 0; tt < RT; ++tt)
                    acc[tt][g] = mfma_step<DT>(ring[u][tt], b, acc[tt][g]);
                b = bn;
            }
            ++x;
        }
    };

    // ---- pipeline prologue
#pragma unroll
    for (int u = 0; u < P; ++u)
        issue_b(ring[u]);
    issue_q(qst[0]);
    issue_q(qst[1]);
    stage_queries(0, qst[0]);
    nx[lane] = load_norm(0);
    float nx_next = load_norm(1);
    lds_barrier();

    for (int it = 0; it < n_it; ++it) {
        // the accumulators start from -|x|^2/2 of their rows
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
            const f32x4 nxh = *(const f32x4 *)(nx + (it & 1) * RW + tt * 16 + jg * 4);
#pragma unroll
            for (int g = 0; g < NG; ++g)
                acc[tt][g] = nxh;
        }
        for (int s0 = 0; s0 < nksp; s0 += R)
            block();

        // ---- end of iteration `it`: acc = -|x|^2/2 + <q, x>; dist = |q|^2 - 2*acc
        nx[((it + 1) & 1) * RW + lane] = nx_next;
        nx_next = load_norm(it + 2);
        uint64_t any = 0;
        static_for<0, NG>([&](auto G) {
            constexpr int g = decltype(G)::value;
            float m = -INFINITY;
            static_for<0, RT>([&](auto TT) {
                constexpr int tt = decltype(TT)::value;
                m = fmaxf(m, fmaxf(fmaxf(acc[tt][g][0], acc[tt][g][1]),
                                   fmaxf(acc[tt][g][2], acc[tt][g][3])));
            });
            any |= ballot(m >= nu_of(g * 16 + col));
        });
        if (any) {
            const long wr0 = rbeg + (long)it * RWG + wave * RW;
            // Stage the candidates of one (query group, row tile) in LDS; the
            // switch keeps every accumulator access at a compile-time index.
            auto stage = [&](auto G, auto TT) -> int {
                constexpr int g = decltype(G)::value, tt = decltype(TT)::value;
                const int i = g * 16 + col;
                const float nu = nu_of(i);
                const f32x4 a4 = acc[tt][g];
                if (!ballot(fmaxf(fmaxf(a4[0], a4[1]), fmaxf(a4[2], a4[3])) >= nu))
                    return 0;
                const float qq = qn_s[i];
                int nst = 0;
                static_for<0, 4>([&](auto E) {
                    constexpr int e = decltype(E)::value;
                    const bool cnd = a4[e] >= nu;
                    const uint64_t m = ballot(cnd);
                    if (cnd) {
                        const int pos = nst + mbcnt(m);
                        sq[pos] = i;
                        sk[pos] = f2key(fmaf(-2.f, a4[e], qq));
                        si[pos] = (int32_t)(wr0 + tt * 16 + jg * 4 + e);
                    }
                    nst += popc(m);
                });
                return nst;
            };
            for (int gt = 0; gt < NG * RT; ++gt) {
                int nst = 0;
                switch (gt) {
#define RB_STAGE_CASE(GT)                                                                          \
    case GT:                                                                                       \
        if constexpr (GT < NG * RT)                                                                \
            nst = stage(Int<GT / RT>{}, Int<GT % RT>{});                                           \
        break;
                    RB_STAGE_CASE(0) RB_STAGE_CASE(1) RB_STAGE_CASE(2) RB_STAGE_CASE(3)
                    RB_STAGE_CASE(4) RB_STAGE_CASE(5) RB_STAGE_CASE(6) RB_STAGE_CASE(7)
                    RB_STAGE_CASE(8) RB_STAGE_CASE(9) RB_STAGE_CASE(10) RB_STAGE_CASE(11)
                    RB_STAGE_CASE(12) RB_STAGE_CASE(13) RB_STAGE_CASE(14) RB_STAGE_CASE(15)
                    RB_STAGE_CASE(16) RB_STAGE_CASE(17) RB_STAGE_CASE(18) RB_STAGE_CASE(19)
                    RB_STAGE_CASE(20) RB_STAGE_CASE(21) RB_STAGE_CASE(22) RB_STAGE_CASE(23)
                    RB_STAGE_CASE(24) RB_STAGE_CASE(25) RB_STAGE_CASE(26) RB_STAGE_CASE(27)
                    RB_STAGE_CASE(28) RB_STAGE_CASE(29) RB_STAGE_CASE(30) RB_STAGE_CASE(31)
                    RB_STAGE_CASE(32) RB_STAGE_CASE(33) RB_STAGE_CASE(34) RB_STAGE_CASE(35)
                    RB_STAGE_CASE(36) RB_STAGE_CASE(37) RB_STAGE_CASE(38) RB_STAGE_CASE(39)
                    RB_STAGE_CASE(40) RB_STAGE_CASE(41) RB_STAGE_CASE(42) RB_STAGE_CASE(43)
                    RB_STAGE_CASE(44) RB_STAGE_CASE(45) RB_STAGE_CASE(46) RB_STAGE_CASE(47)
                    RB_STAGE_CASE(48) RB_STAGE_CASE(49) RB_STAGE_CASE(50) RB_STAGE_CASE(51)
                    RB_STAGE_CASE(52) RB_STAGE_CASE(53) RB_STAGE_CASE(54) RB_STAGE_CASE(55)
                    RB_STAGE_CASE(56) RB_STAGE_CASE(57) RB_STAGE_CASE(58) RB_STAGE_CASE(59)
                    RB_STAGE_CASE(60) RB_STAGE_CASE(61) RB_STAGE_CASE(62) RB_STAGE_CASE(63)
#undef RB_STAGE_CASE
                }
                if (nst)
                    flush(nst);
            }
        }
        // pick up bounds other workgroups have lowered
        for (int i = tid; i < BM; i += SCAN_THREADS)
            if (q0 + i < A.B)
                lds_store_relaxed(gb_s + i, __hip_atomic_load(A.tau + q0 + i, __ATOMIC_RELAXED,
                                                              __HIP_MEMORY_SCOPE_AGENT));
    }

    // ---- this wave's lists -> workspace [B][W][k]
    const int wl = c * SCAN_WAVES + wave;
    for (int i = 0; i < BM; ++i) {
        const int q = q0 + i;
        if (q >= A.B)
            break;
        const int n = lc[i];
        const size_t o = (size_t)q * A.W + wl;
        if (lane == 0)
            A.ccnt[o] = n;
        if (lane < n) {
            A.ckey[o * k + lane] = lk[i * k + lane];
            A.cidx[o * k + lane] = li[i * k + lane];
        }
    }
}

// ------------------------------------------------------------------ merge

struct MergeArgs {
    const int32_t *ccnt;
    const uint32_t *ckey;
    const int32_t *cidx;
    int W, B, k;
    int32_t *nbr_idx;
    float *nbr_dist;
    const float *qual, *len;
    int N, M;
    float *q_hat, *l_hat;
};

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

// One workgroup per query: gather the non-empty lists' entries into LDS (a
// block-wide prefix sum places them), select the k smallest (key, index) pairs
// bit by bit from the most significant key bit, order them, then gather and
// average the labels. Entries that do not fit in LDS are read from the
// workspace instead (slower, same result).
template <int LPT, bool PREDICT>
__global__ __launch_bounds__(MERGE_THREADS) void merge_kernel(const MergeArgs A)
{
    __shared__ uint32_t ek[MERGE_CAP];
    __shared__ int32_t ei[MERGE_CAP];
    __shared__ int wsum[MERGE_THREADS / WAVE];
    __shared__ int red[2][MERGE_THREADS / WAVE];
    __shared__ uint32_t sk[RB_MAX_K_DEV];
    __shared__ int32_t si[RB_MAX_K_DEV];
    __shared__ int32_t so[RB_MAX_K_DEV];
    __shared__ int ns_s;
    const int tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
    const int b = blockIdx.x;
    const int k = A.k, W = A.W;
    const int32_t *cnt = A.ccnt + (size_t)b * W;
    const size_t base = (size_t)b * W * k;

    // lists w = tid + MERGE_THREADS*u of this thread, their lengths and offsets
    int n[LPT], mine = 0;
#pragma unroll
    for (int u = 0; u < LPT; ++u) {
        const int w = tid + MERGE_THREADS * u;
        n[u] = w < W ? cnt[w] : 0;
        mine += n[u];
    }
    float incl = (float)mine;   // block prefix sum (counts < 2^24, exact in fp32)
#pragma unroll
    for (int m = 1; m < WAVE; m <<= 1) {
        const float o = __shfl_up(incl, m);
        if (lane >= m)
            incl += o;
    }
    if (lane == WAVE - 1)
        wsum[wave] = (int)incl;
    if (tid == 0)
        ns_s = 0;
    __syncthreads();
    int off = (int)incl - mine, total = 0;
    for (int w = 0; w < MERGE_THREADS / WAVE; ++w) {
        off += w < wave ? wsum[w] : 0;
        total += wsum[w];
    }
    const bool in_lds = total <= MERGE_CAP;
    if (in_lds) {
#pragma unroll
        for (int u = 0; u < LPT; ++u) {
            const size_t o = base + (size_t)(tid + MERGE_THREADS * u) * k;
            for (int j = 0; j < n[u]; ++j) {
                ek[off + j] = A.ckey[o + j];
                ei[off + j] = A.cidx[o + j];
            }
            off += n[u];
        }
    }
    __syncthreads();

    int phase = 0;
    auto block_sum = [&](int c) -> int {
        const float sw = wave_sum((float)c);
        int *slot = red[phase & 1];
        if (lane == 0)
            slot[wave] = (int)sw;
        __syncthreads();
        ++phase;
        int t = 0;
#pragma unroll
        for (int w = 0; w < MERGE_THREADS / WAVE; ++w)
            t += slot[w];
        return t;
    };
    auto count_if = [&](auto pred) -> int {
        int c = 0;
        if (in_lds) {
            for (int e = tid; e < total; e += MERGE_THREADS)
                c += pred(ek[e], ei[e]);
        } else {
#pragma unroll
            for (int u = 0; u < LPT; ++u) {
                const size_t o = base + (size_t)(tid + MERGE_THREADS * u) * k;
                for (int j = 0; j < n[u]; ++j)
                    c += pred(A.ckey[o + j], A.cidx[o + j]);
            }
        }
        return block_sum(c);
    };
    uint32_t prefix = 0;
    for (int bit = 31; bit >= 0; --bit) {
        const uint32_t trial = prefix | (1u << bit);
        if (count_if([&](uint32_t kk, int32_t) { return kk < trial; }) < k)
            prefix = trial;
    }
    const uint32_t T = prefix;
    const int c_lt = count_if([&](uint32_t kk, int32_t) { return kk < T; });
    const int c_eq = count_if([&](uint32_t kk, int32_t) { return kk == T; });
    const int r = k - c_lt;
    int32_t U = IDX_NONE;
    if (c_eq > r) {
        uint32_t up = 0;
        for (int bit = 30; bit >= 0; --bit) {
            const uint32_t trial = up | (1u << bit);
            if (count_if([&](uint32_t kk, int32_t ii) { return kk == T && (uint32_t)ii < trial; }) <
                r)
                up = trial;
        }
        U = (int32_t)up;
    }
    // the k selected entries, compacted (their order is fixed below)
    if (tid < k) {
        sk[tid] = KEY_NONE;
        si[tid] = IDX_NONE;
        so[tid] = IDX_NONE;
    }
    __syncthreads();
    auto take = [&](uint32_t kk, int32_t ii) {
        if (kk < T || (kk == T && ii <= U)) {
            const int pos = atomicAdd(&ns_s, 1);
            if (pos < k) {
                sk[pos] = kk;
                si[pos] = ii;
            }
        }
    };
    if (in_lds) {
        for (int e = tid; e < total; e += MERGE_THREADS)
            take(ek[e], ei[e]);
    } else {
#pragma unroll
        for (int u = 0; u < LPT; ++u) {
            const size_t o = base + (size_t)(tid + MERGE_THREADS * u) * k;
            for (int j = 0; j < n[u]; ++j)
                take(A.ckey[o + j], A.cidx[o + j]);
        }
    }
    __syncthreads();
    if (tid < k) {
        const uint32_t mk = sk[tid];
        const int32_t mi = si[tid];
        int rank = 0;
        for (int j = 0; j < k; ++j)
            rank += (sk[j] < mk || (sk[j] == mk && si[j] < mi));
        A.nbr_idx[(size_t)b * k + rank] = mi;
        if (A.nbr_dist)
            A.nbr_dist[(size_t)b * k + rank] = key2f(mk);
        so[rank] = mi;
    }
    if constexpr (PREDICT) {
        __syncthreads();
        for (int m = tid; m < A.M; m += MERGE_THREADS)
            average_labels(so, k, A.qual, A.len, A.N, A.M, m, A.q_hat + (size_t)b * A.M + m,
                           A.l_hat + (size_t)b * A.M + m);
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

// ------------------------------------------------------------------ host side

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t scan_lds_bytes(int ng, int k)
{
    const size_t bm = (size_t)ng * 16;
    return 2 * (size_t)ng * WAVE * 16 +   // query double buffer: 2 x ng fragments of 1 KB
           bm * 8 +                       // |q|^2, bound snapshot
           (size_t)SCAN_WAVES * 2 * SCAN_RT * 16 * 4 +   // bank norms of two iterations
           (size_t)SCAN_WAVES * bm * k * 8 +   // lists
           (size_t)SCAN_WAVES * bm * 12 +      // counts, max key, max index
           (size_t)SCAN_WAVES * STAGE_CAP * 12;
}

thread_local hipEvent_t t_scan_begin = nullptr, t_scan_end = nullptr;

template <int LPT>
hipError_t launch_merge(const MergeArgs &m, int B, bool predict, hipStream_t s)
{
    if (predict)
        hipLaunchKernelGGL((merge_kernel<LPT, true>), dim3(B), dim3(MERGE_THREADS), 0, s, m);
    else
        hipLaunchKernelGGL((merge_kernel<LPT, false>), dim3(B), dim3(MERGE_THREADS), 0, s, m);
    return hipGetLastError();
}

template <int DT, int NG, bool RAGGED>
hipError_t launch_scan(const ScanArgs &a, size_t lds, int grid, hipStream_t s)
{
    auto kern = scan_kernel<DT, NG, SCAN_RT, RAGGED>;
    hipError_t e = hipFuncSetAttribute((const void *)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(SCAN_THREADS), lds, s, a);
    return hipGetLastError();
}

template <int DT, bool RAGGED>
hipError_t launch_scan_r(const KnnPlan &p, const ScanArgs &a, int grid, hipStream_t s)
{
    switch (p.ng) {
    case 16: return launch_scan<DT, 16, RAGGED>(a, p.lds_bytes, grid, s);
    case 8: return launch_scan<DT, 8, RAGGED>(a, p.lds_bytes, grid, s);
    case 4: return launch_scan<DT, 4, RAGGED>(a, p.lds_bytes, grid, s);
    case 2: return launch_scan<DT, 2, RAGGED>(a, p.lds_bytes, grid, s);
    case 1: return launch_scan<DT, 1, RAGGED>(a, p.lds_bytes, grid, s);
    }
    return hipErrorInvalidValue;
}

template <int DT>
hipError_t launch_scan_dt(const KnnPlan &p, const ScanArgs &a, int grid, hipStream_t s)
{
    const bool ragged = p.d % (4 * Elem<DT>::VEC) != 0;
    return ragged ? launch_scan_r<DT, true>(p, a, grid, s) : launch_scan_r<DT, false>(p, a, grid, s);
}

template <int DT>
hipError_t launch_seed_bound(const KnnPlan &p, const void *queries, const float *gmin, float *qn,
                             uint32_t *tau, hipStream_t s)
{
    const int grid = (p.B + 3) / 4;
    const uint8_t *q = (const uint8_t *)queries;
    const int G = p.S ? p.G : 0;
    if (G <= 1024)
        hipLaunchKernelGGL((seed_bound_kernel<DT, 16>), dim3(grid), dim3(256), 0, s, q, p.B, p.d,
                           p.k, gmin, G, qn, tau);
    else
        hipLaunchKernelGGL((seed_bound_kernel<DT, 32>), dim3(grid), dim3(256), 0, s, q, p.B, p.d,
                           p.k, gmin, G, qn, tau);
    return hipGetLastError();
}

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
    p->nksp = (p->nks + SCAN_UNROLL - 1) / SCAN_UNROLL * SCAN_UNROLL;
    // largest query tile that B can fill and that fits in LDS
    int want = 1;
    while (want < 16 && want * 16 < B)
        want *= 2;
    p->ng = 0;
    for (int ng = want; ng >= 1; ng /= 2) {
        const size_t lds = scan_lds_bytes(ng, k);
        if (lds <= LDS_LIMIT) {
            p->ng = ng;
            p->lds_bytes = lds;
            break;
        }
    }
    if (p->ng == 0)
        return -1;
    p->rt = SCAN_RT;
    const int bm = p->ng * 16;
    p->n_qt = B > 0 ? (B + bm - 1) / bm : 1;
    // one workgroup per compute unit (the LDS use allows no more)
    long chunks = num_cu / p->n_qt;
    if (chunks < 1)
        chunks = 1;
    const long max_chunks = ((long)N + 15) / 16;
    if (chunks > max_chunks)
        chunks = max_chunks;
    const long rowb = (long)d * (dtype == 1 ? 2 : 4);
    if ((long)B * rowb >= (1L << 31))
        return -1;   // the query resource is addressed with 32-bit offsets
    long rpc = ((long)N + chunks - 1) / chunks;
    rpc = (rpc + 15) / 16 * 16;
    while (rpc * rowb >= (1L << 31) - (1L << 20)) {   // so is each bank chunk
        chunks *= 2;
        rpc = ((long)N + chunks - 1) / chunks;
        rpc = (rpc + 15) / 16 * 16;
    }
    p->rows_per_chunk = rpc;
    p->n_chunks = (int)(((long)N + rpc - 1) / rpc);
    p->W = p->n_chunks * SCAN_WAVES;
    if (p->W > MERGE_MAX_LISTS)
        return -1;
    // seed sample: about N/32 rows, 2048..32768, a multiple of 64 and at most N
    long S = N / 32;
    if (S < 2048)
        S = 2048;
    if (S > 32768)
        S = 32768;
    if (S > N)
        S = N;
    S = S / 64 * 64;
    if (S / 16 < k)
        S = 0;
    p->S = (int)S;
    p->G = (int)(S / 16);
    size_t off = 0;
    p->off_tau = off;
    off += align256((size_t)B * 4);
    p->off_qn = off;
    off += align256((size_t)B * 4);
    p->off_gmin = off;
    off += align256((size_t)B * (p->G > 0 ? p->G : 1) * 4);
    p->off_ccnt = off;
    off += align256((size_t)B * p->W * 4);
    p->off_ckey = off;
    off += align256((size_t)B * p->W * k * 4);
    p->off_cidx = off;
    off += align256((size_t)B * p->W * k * 4);
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
    float *qn = (float *)(w + p.off_qn);
    float *gmin = (float *)(w + p.off_gmin);
    int32_t *ccnt = (int32_t *)(w + p.off_ccnt);
    uint32_t *ckey = (uint32_t *)(w + p.off_ckey);
    int32_t *cidx = (int32_t *)(w + p.off_cidx);
    hipError_t e;

    if (p.S > 0) {
        SeedArgs sa;
        sa.queries = (const uint8_t *)queries;
        sa.bank = (const uint8_t *)bank;
        sa.bank_norms = bank_norms;
        sa.B = p.B;
        sa.N = p.N;
        sa.d = p.d;
        sa.nks = p.nks;
        sa.S = p.S;
        sa.G = p.G;
        sa.n_qg = (p.B + 15) / 16;
        sa.gmin = gmin;
        const dim3 grid(p.S / 64, (sa.n_qg + SEED_WAVES - 1) / SEED_WAVES);
        if (p.dtype == 1)
            hipLaunchKernelGGL(seed_groups_kernel<1>, grid, dim3(SEED_WAVES * WAVE), 0, s, sa);
        else
            hipLaunchKernelGGL(seed_groups_kernel<0>, grid, dim3(SEED_WAVES * WAVE), 0, s, sa);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }
    e = p.dtype == 1 ? launch_seed_bound<1>(p, queries, gmin, qn, tau, s)
                     : launch_seed_bound<0>(p, queries, gmin, qn, tau, s);
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
    a.nksp = p.nksp;
    a.n_chunks = p.n_chunks;
    a.n_qt = p.n_qt;
    a.W = p.W;
    a.rows_per_chunk = p.rows_per_chunk;
    a.tau = tau;
    a.ccnt = ccnt;
    a.ckey = ckey;
    a.cidx = cidx;
    const int grid = ((p.n_chunks + 7) / 8) * 8 * p.n_qt;
    const bool timed = t_scan_begin && t_scan_end;
    if (timed && (e = hipEventRecord(t_scan_begin, s)) != hipSuccess)
        return e;
    e = p.dtype == 1 ? launch_scan_dt<1>(p, a, grid, s) : launch_scan_dt<0>(p, a, grid, s);
    if (e != hipSuccess)
        return e;
    if (timed && (e = hipEventRecord(t_scan_end, s)) != hipSuccess)
        return e;

    MergeArgs m;
    m.ccnt = ccnt;
    m.ckey = ckey;
    m.cidx = cidx;
    m.W = p.W;
    m.B = p.B;
    m.k = p.k;
    m.nbr_idx = nbr_idx;
    m.nbr_dist = nbr_dist;
    m.qual = bank_qual;
    m.len = bank_len;
    m.N = p.N;
    m.M = M;
    m.q_hat = q_hat;
    m.l_hat = l_hat;
    const int lpt = (p.W + MERGE_THREADS - 1) / MERGE_THREADS;
    const bool pred = q_hat != nullptr;
    if (lpt <= 1)
        return launch_merge<1>(m, p.B, pred, s);
    if (lpt <= 2)
        return launch_merge<2>(m, p.B, pred, s);
    if (lpt <= 4)
        return launch_merge<4>(m, p.B, pred, s);
    if (lpt <= 8)
        return launch_merge<8>(m, p.B, pred, s);
    if (lpt <= 16)
        return launch_merge<16>(m, p.B, pred, s);
    return hipErrorInvalidValue;
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
