// Exact k-nearest-neighbour search over the labelled reference bank
// (RouteBalance Sec. 4.2: the KNN lookup of Alg. 1), for gfx950.
//
// Kernels of one call:
//   seed_groups_kernel  distances of every query to S bank rows spread evenly
//                       over the bank; minima over groups of 16 of those rows
//   seed_bound_kernel   per query: |q|^2, and the k-th smallest group minimum
//                       as the starting bound of the k-th nearest distance
//   scan_kernel         the bank once through MFMA (scan.hpp): one workgroup
//                       per (bank chunk, tile of up to 256 queries); bank rows
//                       go from HBM straight into MFMA operand registers, the
//                       query tile sits in LDS (part resident, part streamed
//                       along K); a register-level test against the per-query
//                       bound lets only candidates reach the workgroup's
//                       shared top-k lists
//   merge_kernel        per query: the k nearest of all lists, sorted, then
//                       optionally the label gather and average (Sec. 4.2: one
//                       lookup predicts quality and length for every model)
// Order everywhere: distance ascending, equal distances by the lower bank
// index. Distances are |q|^2 + |x|^2 - 2<q,x> with fp32 products and
// accumulation; the scan accumulates -|x|^2/2 + <q,x> and reports
// |q|^2 - 2*acc.
#include "knn_common.hpp"

namespace rb {

namespace {

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

// One workgroup of SEED_WAVES waves per SEED_WAVES groups of 16 sample rows
// and QG query groups of 16 (blockIdx.y): wave w owns group 8*blockIdx.x + w.
// Its bank fragments (row lane%16 of the group, 16-byte quarter lane/16 of
// each 64-byte k-step) come straight from global memory, three k-steps ahead;
// the workgroup stages the k-step's query fragments once in an LDS double
// buffer, so every query is loaded once per workgroup and every sample row
// once. p = |x|^2 - 2<q,x> by MFMA (the accumulators start at -|x|^2/2); each
// query keeps the minimum over the group's 16 rows.
constexpr int SEED_WAVES = 8;
constexpr int SEED_RING = 4;   // k-steps of loads in flight (even: LDS buffer = slot parity)

template <int DT, int QG>
__global__ __launch_bounds__(SEED_WAVES * WAVE) void seed_groups_kernel(const SeedArgs A)
{
    constexpr int VEC = Elem<DT>::VEC, ESZ = Elem<DT>::ESZ;
    constexpr int NT = SEED_WAVES * WAVE;
    constexpr int QPT = (QG * WAVE + NT - 1) / NT;   // query fragments each thread stages
    __shared__ i32x4 qs[2][QG][WAVE];
    const int tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
    const int col = lane & 15, jg = lane >> 4;
    const int grp = blockIdx.x * SEED_WAVES + wave;
    const bool gv = grp < A.G;
    const int qg0 = blockIdx.y * QG;
    const size_t rowb = (size_t)A.d * ESZ;
    const i32x4 z = {0, 0, 0, 0};
    const uint8_t *ap =
        A.bank + (gv ? (size_t)seed_row(grp * 16 + col, A.N, A.S) * rowb : 0) + jg * 16;
    auto a_load = [&](int s) -> i32x4 {
        return gv && s < A.nks && s * 4 * VEC + jg * VEC < A.d ? load16(ap + (size_t)s * KSTEP_BYTES)
                                                               : z;
    };
    // staged fragment f = tid + NT*u is lane f%64 of query group f/64
    const uint8_t *qp[QPT];
    bool qv[QPT];
    int qj[QPT];
#pragma unroll
    for (int u = 0; u < QPT; ++u) {
        const int f = tid + NT * u;
        const int q = (qg0 + (f >> 6)) * 16 + (f & 15);
        qv[u] = f < QG * WAVE && q < A.B;
        qj[u] = (f >> 4) & 3;
        qp[u] = A.queries + (qv[u] ? (size_t)q * rowb : 0) + qj[u] * 16;
    }
    auto q_load = [&](int u, int s) -> i32x4 {
        return qv[u] && s * 4 * VEC + qj[u] * VEC < A.d ? load16(qp[u] + (size_t)s * KSTEP_BYTES)
                                                        : z;
    };
    auto q_store = [&](int buf, int u, const i32x4 &v) {
        const int f = tid + NT * u;
        if (f < QG * WAVE)
            qs[buf][f >> 6][f & 63] = v;
    };
    f32x4 acc[QG];
    {
        f32x4 h;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            h[e] = gv ? -0.5f * A.bank_norms[seed_row(grp * 16 + jg * 4 + e, A.N, A.S)] : 0.f;
#pragma unroll
        for (int g = 0; g < QG; ++g)
            acc[g] = h;
    }
    // register rings: the loads of k-step s + SEED_RING - 1 are issued at step
    // s; step s's fragment sits in slot s % SEED_RING (the loop is unrolled by
    // the ring size, so every slot index is a constant)
    i32x4 ar[SEED_RING], qr[SEED_RING][QPT];
    static_for<0, SEED_RING - 1>([&](auto J) {
        ar[J.value] = a_load(J.value);
#pragma unroll
        for (int u = 0; u < QPT; ++u)
            qr[J.value][u] = q_load(u, J.value);
    });
#pragma unroll
    for (int u = 0; u < QPT; ++u)
        q_store(0, u, qr[0][u]);
    __syncthreads();
    for (int s0 = 0; s0 < A.nks; s0 += SEED_RING) {
        static_for<0, SEED_RING>([&](auto R) {
            constexpr int r = R.value, nx = (r + SEED_RING - 1) % SEED_RING;
            const int s = s0 + r;
            if (s >= A.nks)
                return;
            ar[nx] = a_load(s + SEED_RING - 1);
#pragma unroll
            for (int u = 0; u < QPT; ++u)
                qr[nx][u] = q_load(u, s + SEED_RING - 1);
#pragma unroll
            for (int g = 0; g < QG; ++g)
                acc[g] = mfma_step<DT>(ar[r], qs[r & 1][g][lane], acc[g]);
            if (s + 1 < A.nks) {
#pragma unroll
                for (int u = 0; u < QPT; ++u)
                    q_store((r + 1) & 1, u, qr[(r + 1) % SEED_RING][u]);
            }
            __syncthreads();
        });
    }
#pragma unroll
    for (int g = 0; g < QG; ++g) {
        // p = -2 * acc for this lane's four rows of the group
        float m = fminf(fminf(-2.f * acc[g][0], -2.f * acc[g][1]),
                        fminf(-2.f * acc[g][2], -2.f * acc[g][3]));
        // lanes col, col+16, col+32, col+48 hold the four row quarters
        m = fminf(m, __shfl_xor(m, 16));
        m = fminf(m, __shfl_xor(m, 32));
        const int q = (qg0 + g) * 16 + col;
        if (gv && jg == 0 && q < A.B)
            A.gmin[(size_t)q * A.G + grp] = m;
    }
}

// One wave per query: |q|^2, and the starting bound = |q|^2 + the k-th
// smallest of the wave's 128 lane values (each lane's two smallest group
// minima; lane l holds groups l, l + 64, ...), widened by a margin far above
// any fp32 rounding difference between this pass and the scan. The values
// belong to distinct groups, so the k smallest are distances of k distinct
// sample rows and bound the k-th nearest distance from above; they are the
// k smallest group minima unless three of those share a lane. The k-th
// smallest is found bit by bit from the top, two ballots per bit. Without a
// seed (G < k) the bound is +inf.
template <int DT, int GPL>
__global__ __launch_bounds__(WAVE) void seed_bound_kernel(const uint8_t *__restrict__ queries,
                                                          int B, int d, int k,
                                                          const float *__restrict__ gmin, int G,
                                                          float *__restrict__ qn,
                                                          uint32_t *__restrict__ tau)
{
    static_assert(GPL * WAVE >= SEED_MAX_GROUPS, "every group has a slot");
    const int lane = lane_id();
    const int b = blockIdx.x;
    // every load in flight at once: slots past G read the last group and
    // discard it
    uint32_t m1 = KEY_NONE, m2 = KEY_NONE;   // the lane's smallest and second smallest
    if (G >= k) {
        uint32_t key[GPL];
#pragma unroll
        for (int u = 0; u < GPL; ++u) {
            const int i = u * WAVE + lane;
            const float v = gmin[(size_t)b * G + (i < G ? i : G - 1)];
            key[u] = f2key(v) | (i < G ? 0u : KEY_NONE);   // uses v unconditionally
        }
#pragma unroll
        for (int u = 0; u < GPL; ++u) {
            m2 = min(m2, max(m1, key[u]));
            m1 = min(m1, key[u]);
        }
    }
    const int row_bytes = d * Elem<DT>::ESZ;
    const uint8_t *row = queries + (size_t)b * row_bytes;
    float s = 0.f;
    for (int off = lane * 16; off < row_bytes; off += WAVE * 16)
        s = sumsq16<DT>(load16(row + off), s);
    s = wave_sum(s);
    uint32_t T = KEY_NONE;
    if (G >= k) {
        // the largest prefix with fewer than k lane values below it is the
        // k-th smallest lane value (the lanes hold min(G, 128) >= k groups)
        uint32_t prefix = 0;
        for (int bit = 31; bit >= 0; --bit) {
            const uint32_t trial = prefix | (1u << bit);
            if (popc(ballot(m1 < trial)) + popc(ballot(m2 < trial)) < k)
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

// ------------------------------------------------------------------ list bound

// The shared bound after a first pass over part of every chunk: per query,
// the k-th smallest key among the entries of its first nl lists (of W),
// when there are at least k. Any k of the entries are distances of k
// distinct bank rows, so each lane keeps only its LB_KEEP smallest, and the
// k-th smallest of those kept, an upper bound of the k-th nearest distance
// (the exact k-th smallest unless more than LB_KEEP of the k smallest are one
// lane's), lowers the bound. One wave per query: k rounds each take the
// wave's smallest kept key out of its lane.
constexpr int LB_KEEP = 16;
__global__ __launch_bounds__(WAVE) void list_bound_kernel(const int32_t *__restrict__ ccnt,
                                                         const uint32_t *__restrict__ ckey,
                                                         int W, int nl, int k,
                                                         uint32_t *__restrict__ tau)
{
    const int b = blockIdx.x, lane = lane_id();
    const int32_t *cnt = ccnt + (size_t)b * W;
    const uint32_t *key = ckey + (size_t)b * W * k;
    uint32_t v[LB_KEEP];   // ascending; KEY_NONE: empty
#pragma unroll
    for (int i = 0; i < LB_KEEP; ++i)
        v[i] = KEY_NONE;
    // four lists per lane at a time: their lengths, then their entries
    for (int w0 = 0; w0 < nl; w0 += 4 * WAVE) {
        int m[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int w = w0 + u * WAVE + lane;
            m[u] = w < nl ? cnt[w] : 0;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const uint32_t *kw = key + (size_t)(w0 + u * WAVE + lane) * k;
            for (int j = 0; j < m[u]; ++j) {
                uint32_t x = kw[j];
#pragma unroll
                for (int i = 0; i < LB_KEEP; ++i) {
                    const uint32_t lo = min(v[i], x);
                    x = max(v[i], x);
                    v[i] = lo;
                }
            }
        }
    }
    uint32_t kth = KEY_NONE;
    for (int r = 0; r < k; ++r) {
        uint32_t mn = v[0];
#pragma unroll
        for (int o = 1; o < WAVE; o <<= 1)
            mn = min(mn, (uint32_t)__shfl_xor((int)mn, o));
        if (mn == KEY_NONE)
            return;   // fewer than k keys (keys are below KEY_NONE)
        if (lane == __builtin_ctzll(ballot(v[0] == mn))) {
#pragma unroll
            for (int i = 0; i + 1 < LB_KEEP; ++i)
                v[i] = v[i + 1];
            v[LB_KEEP - 1] = KEY_NONE;
        }
        kth = mn;
    }
    if (lane == 0 && kth < tau[b])
        tau[b] = kth;
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
    bool inv_dist;
};

// Weight of a neighbour at squared distance d2 in the distance-weighted
// average: the inverse of its Euclidean distance, finite at distance 0 (a
// negative d2 from fp32 cancellation counts as 0).
__device__ __forceinline__ float inv_dist_weight(float d2)
{
    return 1.f / (sqrtf(fmaxf(d2, 0.f)) + 1e-6f);
}

// The label gather and average: sum over neighbours j = 0..k-1 in order,
// divided by k, or (wts non-null) weighted by wts[j] and divided by the sum
// of the weights. A neighbour index outside [0, N) makes both averages NaN
// instead of reading out of bounds (the check does not end the loop, so the
// k loads can all be in flight together).
__device__ __forceinline__ void average_labels(const int32_t *nbr, const float *wts, int k,
                                               const float *qual, const float *len, int N, int M,
                                               int m, float *q_out, float *l_out)
{
    float sq = 0.f, sl = 0.f, sw = 0.f;
    bool bad = false;
    if (wts) {
#pragma unroll 8
        for (int j = 0; j < k; ++j) {
            const int32_t n = nbr[j];
            const bool ok = n >= 0 && n < N;
            bad |= !ok;
            const size_t o = (size_t)(ok ? n : 0) * M + m;
            const float w = wts[j];
            sq = fmaf(w, qual[o], sq);
            sl = fmaf(w, len[o], sl);
            sw += w;
        }
    } else {
#pragma unroll 8
        for (int j = 0; j < k; ++j) {
            const int32_t n = nbr[j];
            const bool ok = n >= 0 && n < N;
            bad |= !ok;
            const size_t o = (size_t)(ok ? n : 0) * M + m;
            sq += qual[o];
            sl += len[o];
        }
        sw = (float)k;
    }
    *q_out = bad ? __builtin_nanf("") : sq / sw;
    *l_out = bad ? __builtin_nanf("") : sl / sw;
}

// One wave per query (MERGE_WAVES queries per workgroup, no workgroup
// barrier): the wave's lanes take the lists w = lane + 64*u, a wave prefix
// sum places their entries as packed (key << 32 | index) values in LDS, then
// k rounds each pick the smallest entry above the previous pick (one pass
// over the entries and one 64-bit wave minimum; entries are distinct, so the
// picks are the k smallest in order). Lane r ends with pick r. Entries that do
// not fit in LDS are read from the workspace in every round instead (slower,
// same result). Then, optionally, the label gather and average.
template <int LPL, bool PREDICT>
__global__ __launch_bounds__(MERGE_WAVES * WAVE) void merge_kernel(const MergeArgs A)
{
    __shared__ uint64_t ent_all[MERGE_WAVES][MERGE_CAP];
    const int lane = lane_id(), wave = threadIdx.x >> 6;
    const int b = blockIdx.x * MERGE_WAVES + wave;
    if (b >= A.B)
        return;
    uint64_t *ent = ent_all[wave];
    const int k = A.k, W = A.W;
    const int32_t *cnt = A.ccnt + (size_t)b * W;
    const size_t base = (size_t)b * W * k;
    // the first GE entries of every list of this lane are loaded with the
    // list lengths, whatever the lengths (lists are short once the bound is
    // tight; a lane past the last list reads the last list); longer lists
    // finish after
    constexpr int GE = LPL <= 8 ? 4 : 1;
    uint32_t kk[LPL][GE];
    int32_t ii[LPL][GE];
    int n[LPL], mine = 0;
#pragma unroll
    for (int u = 0; u < LPL; ++u) {
        const int w = lane + WAVE * u;
        n[u] = w < W ? cnt[w] : 0;
        const size_t o = base + (size_t)min(w, W - 1) * k;
#pragma unroll
        for (int j = 0; j < GE; ++j) {
            kk[u][j] = j < k ? A.ckey[o + j] : 0u;
            ii[u][j] = j < k ? A.cidx[o + j] : 0;
        }
    }
#pragma unroll
    for (int u = 0; u < LPL; ++u)
        mine += n[u];
    const int incl = wave_incl_scan(mine);
    const int total = __builtin_amdgcn_readlane(incl, WAVE - 1);
    const bool in_lds = total <= MERGE_CAP;
    if (in_lds) {
        int off = incl - mine;
#pragma unroll
        for (int u = 0; u < LPL; ++u) {
            const size_t o = base + (size_t)(lane + WAVE * u) * k;
#pragma unroll
            for (int j = 0; j < GE; ++j)
                if (j < n[u])
                    ent[off + j] = pack(kk[u][j], ii[u][j]);
            for (int j = GE; j < n[u]; ++j)
                ent[off + j] = pack(A.ckey[o + j], A.cidx[o + j]);
            off += n[u];
        }
    }
    uint64_t prev = 0, pick = ~0ull;
    for (int r = 0; r < k; ++r) {
        uint64_t m = ~0ull;
        auto see = [&](uint64_t v) {
            if (v > prev && v < m)
                m = v;
        };
        if (in_lds) {
            for (int e = lane; e < total; e += WAVE)
                see(ent[e]);
        } else {
#pragma unroll
            for (int u = 0; u < LPL; ++u) {
                const size_t o = base + (size_t)(lane + WAVE * u) * k;
                for (int j = 0; j < n[u]; ++j)
                    see(pack(A.ckey[o + j], A.cidx[o + j]));
            }
        }
        // wave minimum: the largest complement
        uint32_t hi = ~(uint32_t)(m >> 32), lo = ~(uint32_t)m;
        reduce_max_pair<WAVE>(hi, lo);
        m = ((uint64_t)~hi << 32) | ~lo;
        if (lane == r)
            pick = m;
        prev = m;
    }
    const int32_t pidx = (int32_t)(uint32_t)pick;
    if (lane < k) {
        A.nbr_idx[(size_t)b * k + lane] = pidx;
        if (A.nbr_dist)
            A.nbr_dist[(size_t)b * k + lane] = key2f((uint32_t)(pick >> 32));
    }
    if constexpr (PREDICT) {
        __shared__ int32_t nbr_all[MERGE_WAVES][RB_MAX_K_DEV];
        __shared__ float wts_all[MERGE_WAVES][RB_MAX_K_DEV];
        int32_t *nbr = nbr_all[wave];
        float *wts = wts_all[wave];
        if (lane < k) {
            nbr[lane] = pidx;
            wts[lane] = inv_dist_weight(key2f((uint32_t)(pick >> 32)));
        }
        const int M = A.M;
        if (k * M <= WAVE) {
            // every (neighbour, model) label in flight at once: lane j*M + m
            // loads neighbour j's labels for model m; lane m then adds them
            // up in neighbour order exactly as average_labels does
            const int jl = lane / M, ml = lane - jl * M;
            const bool own = lane < k * M;
            const int32_t nj = __shfl(pidx, own ? jl : 0);
            const bool ok = nj >= 0 && nj < A.N;
            const size_t o = (size_t)(ok ? nj : 0) * M + (own ? ml : 0);
            const float qv = A.qual[o], lv = A.len[o];
            const int mm = lane < M ? lane : 0;
            float sq = 0.f, sl = 0.f, sw = 0.f;
            bool bad = false;
            for (int j = 0; j < k; ++j) {
                const int src = j * M + mm;
                const float q = __shfl(qv, src), l = __shfl(lv, src);
                bad |= __shfl((int)ok, src) == 0;
                if (A.inv_dist) {
                    const float w = wts[j];
                    sq = fmaf(w, q, sq);
                    sl = fmaf(w, l, sl);
                    sw += w;
                } else {
                    sq += q;
                    sl += l;
                }
            }
            if (!A.inv_dist)
                sw = (float)k;
            if (lane < M) {
                A.q_hat[(size_t)b * M + lane] = bad ? __builtin_nanf("") : sq / sw;
                A.l_hat[(size_t)b * M + lane] = bad ? __builtin_nanf("") : sl / sw;
            }
        } else {
            for (int m = lane; m < M; m += WAVE)
                average_labels(nbr, A.inv_dist ? wts : nullptr, k, A.qual, A.len, A.N, M, m,
                               A.q_hat + (size_t)b * M + m, A.l_hat + (size_t)b * M + m);
        }
    }
}

// One workgroup per request; nbr_dist is read only for the weighted average.
__global__ __launch_bounds__(64) void predict_kernel(const int32_t *__restrict__ nbr_idx,
                                                     const float *__restrict__ nbr_dist, int k,
                                                     const float *__restrict__ qual,
                                                     const float *__restrict__ len, int N, int M,
                                                     float *__restrict__ q_hat,
                                                     float *__restrict__ l_hat)
{
    __shared__ int32_t nbr[RB_MAX_K_DEV];
    __shared__ float wts[RB_MAX_K_DEV];
    const int b = blockIdx.x;
    for (int j = threadIdx.x; j < k; j += blockDim.x) {
        nbr[j] = nbr_idx[(size_t)b * k + j];
        if (nbr_dist)
            wts[j] = inv_dist_weight(nbr_dist[(size_t)b * k + j]);
    }
    __syncthreads();
    for (int m = threadIdx.x; m < M; m += blockDim.x)
        average_labels(nbr, nbr_dist ? wts : nullptr, k, qual, len, N, M, m,
                       q_hat + (size_t)b * M + m, l_hat + (size_t)b * M + m);
}

// ------------------------------------------------------------------ host side

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

thread_local hipEvent_t t_scan_begin = nullptr, t_scan_end = nullptr;

template <int LPL>
hipError_t launch_merge(const MergeArgs &m, int B, bool predict, hipStream_t s)
{
    const dim3 grid((B + MERGE_WAVES - 1) / MERGE_WAVES), block(MERGE_WAVES * WAVE);
    if (predict)
        hipLaunchKernelGGL((merge_kernel<LPL, true>), grid, block, 0, s, m);
    else
        hipLaunchKernelGGL((merge_kernel<LPL, false>), grid, block, 0, s, m);
    return hipGetLastError();
}

template <int DT>
hipError_t launch_seed_bound(const KnnPlan &p, const void *queries, const float *gmin, float *qn,
                             uint32_t *tau, hipStream_t s)
{
    const uint8_t *q = (const uint8_t *)queries;
    const int G = p.S ? p.G : 0;
    constexpr int GPL = SEED_MAX_GROUPS / WAVE;
    hipLaunchKernelGGL((seed_bound_kernel<DT, GPL>), dim3(p.B), dim3(WAVE), 0, s,
                       q, p.B, p.d, p.k, gmin, G, qn, tau);
    return hipGetLastError();
}

}  // namespace

void set_scan_events(hipEvent_t begin, hipEvent_t end)
{
    t_scan_begin = begin;
    t_scan_end = end;
}

int plan_knn(int B, int N, int d, int dtype, int k, int num_cu, KnnPlan *p, int reserve)
{
    const int vec = dtype == 1 ? 8 : 4;
    p->dtype = dtype;
    p->B = B;
    p->N = N;
    p->d = d;
    p->k = k;
    p->nks = (d + 4 * vec - 1) / (4 * vec);
    p->nksp = (p->nks + SCAN_KPAD - 1) / SCAN_KPAD * SCAN_KPAD;
    const bool ragged = d % (4 * vec) != 0;
    // The query-resident scan takes bf16 rows of 12, 16, 24 or 32 full
    // k-steps (d = 384, 512, 768, 1024) when the batch fits the registers of
    // one workgroup: the first (query groups per wave, row halves) of the
    // row length's list, in order of capacity, that holds B queries, with
    // the first ring whose LDS (ring, lists, query data) fits: four slots of
    // half blocks (whole blocks for d = 384), which keep three stages of
    // loads in flight, else two slots of whole or of half blocks. A wave
    // holds qw * nks * 4 registers of query fragments, at most 192. A batch
    // of up to 64 queries takes it only over a bank of at least
    // RQ_SMALL_B_MIN_ROWS rows per compute unit: over fewer, its per-workgroup
    // start (every wave loading its queries, the ring filling) costs more than
    // the tile scan's, whose query tile stays in LDS (measured: 100,000 rows
    // of 768 at 64 queries, 49.9 against 43.6 us cold; 1,000,000 rows, 264
    // against 286 us).
    p->kind = 0;
    p->qw = p->rs = p->spb = p->stages = 0;
    const bool rq_small_ok = (long)N >= (long)RQ_SMALL_B_MIN_ROWS * num_cu;
    if (dtype == 1 && !ragged && B >= 1 && (B > 64 || rq_small_ok)) {
        static const int tab12[][2] = {{1, 2}, {2, 2}, {4, 2}, {4, 1}};
        static const int tab16[][2] = {{1, 2}, {2, 2}, {2, 1}};
        static const int tab32[][2] = {{1, 2}, {1, 1}};
        const int(*tab)[2] = nullptr;
        int n_tab = 0;
        if (p->nks == 12) {
            tab = tab12;
            n_tab = 4;
        } else if (p->nks == 16 || p->nks == 24) {
            tab = tab16;
            n_tab = 3;
        } else if (p->nks == 32) {
            tab = tab32;
            n_tab = 2;
        }
        for (int t = 0; t < n_tab && p->kind == 0; ++t) {
            const int qw = tab[t][0], rs = tab[t][1];
            if ((RQ_WAVES / rs) * qw * 16 < B)
                continue;
            // (stages per block, slots)
            static const int ring12[][2] = {{1, 4}, {1, 2}};
            static const int ring16[][2] = {{2, 4}, {1, 2}, {2, 2}};
            static const int ring32[][2] = {{2, 4}, {2, 2}};
            const int(*ring)[2] = p->nks == 12 ? ring12 : p->nks == 32 ? ring32 : ring16;
            const int n_ring = p->nks == 16 || p->nks == 24 ? 3 : 2;
            for (int u = 0; u < n_ring; ++u) {
                const int spb = ring[u][0], stages = ring[u][1];
                if (rq_layout(k, qw, p->nks / spb, stages).bytes <= LDS_LIMIT) {
                    p->kind = 1;
                    p->qw = qw;
                    p->rs = rs;
                    p->spb = spb;
                    p->stages = stages;
                    break;
                }
            }
        }
    }
    // The GEMM-structured scan takes batches of more than 256 bf16 requests
    // that the query-resident scan cannot hold, whose rows are a whole
    // number of its 64-element stages (at least two) and whose lists fit its
    // LDS beside the stage ring. (With one tile of requests per chunk it
    // would fetch every bank row from HBM with a single stage of lead, so
    // smaller batches stay on the other scans.)
    if (dtype == 1 && B > 256 && p->kind != 1 && d % GM_KST == 0 && d >= 2 * GM_KST &&
        gemm_layout(k).bytes <= LDS_LIMIT) {
        p->kind = 2;
        p->qw = p->rs = p->spb = p->stages = 0;
    }
    // tile scan: largest query tile that B can fill and whose lists fit in
    // LDS; then as many of its query groups resident in LDS as the rest of
    // the space holds
    int want = 1;
    while (want < 16 && want * 16 < B)
        want *= 2;
    p->ng = 0;
    for (int ng = want; ng >= 1; ng /= 2) {
        const int slots = scan_ring(dtype, ng, 0, ragged);
        if (scan_layout(ng, 0, p->nksp, k, SCAN_RT, slots).bytes <= LDS_LIMIT) {
            p->ng = ng;
            break;
        }
    }
    if (p->ng == 0)
        return -1;
    // resident query groups: all, half, a quarter, an eighth or none of the
    // tile (the counts the scan is compiled for), the most that fit
    const int gr_opts[5] = {p->ng, p->ng / 2, p->ng / 4, p->ng / 8, 0};
    p->gr = 0;
    for (int gr : gr_opts) {
        const int slots = scan_ring(dtype, p->ng, gr, ragged);
        if (scan_layout(p->ng, gr, p->nksp, k, SCAN_RT, slots).bytes <= LDS_LIMIT) {
            p->gr = gr;
            break;
        }
    }
    p->lds_bytes = scan_layout(p->ng, p->gr, p->nksp, k, SCAN_RT,
                               scan_ring(dtype, p->ng, p->gr, ragged))
                       .bytes;
    p->rt = SCAN_RT;
    const int bm = p->ng * 16;
    p->n_qt = B > 0 ? (B + bm - 1) / bm : 1;
    if (p->kind == 1) {
        p->n_qt = 1;
        p->lds_bytes = rq_layout(k, p->qw, p->nks / p->spb, p->stages).bytes;
    } else if (p->kind == 2) {
        p->n_qt = (B + GM_QRY - 1) / GM_QRY;
        p->lds_bytes = gemm_layout(k).bytes;
    }
    // one workgroup per compute unit (the LDS use allows no more); with
    // `reserve`, that many units of each XCD stay free: workgroups go to the
    // XCDs round robin and the tiles of a chunk share its XCD, so a whole
    // number of chunks per XCD is kept below the XCD's unit count. The GEMM
    // scan also fills the units that this leaves over (up to n_qt - 1 per
    // XCD): its last n_chunks % 8 chunks are spread over neighbouring XCDs,
    // at most two per chunk for four request tiles (measured at B = 1,024,
    // d = 1,024: 248 workgroups 1,821 us per launch against 1,942 us for 224)
    long chunks = num_cu / p->n_qt;
    if (reserve > 0) {
        const long per_xcd = (num_cu / 8 - reserve) / p->n_qt;
        if (per_xcd >= 1)
            chunks = per_xcd * 8;
        if (p->kind == 2)
            chunks = (num_cu - 8L * reserve) / p->n_qt;
    }
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
    // The query-resident scan goes in two passes when the seed covers less
    // than 1/32 of a long bank (N / 32 above the largest seed, 32,768 rows)
    // and the batch exceeds 128 requests: the first pass takes the first eighth of every chunk, the
    // k-th smallest entry of its lists then bounds the second, over the rest,
    // which leaves a second set of lists. The bank is still read once and the
    // second pass runs under the bound of a sample of an eighth of the bank.
    // (Measured, one pass against two: B = 512, N = 4,000,000, d = 384
    // 1,656 against 1,497 us; B = 256, N = 1,000,000, d = 768, where the seed
    // already covers N/32, 446-450 against 437-444; B <= 128 10-13 % slower
    // in two passes: the second launch's start outweighs the fewer
    // candidates.)
    p->rq_split = 0;
    if (p->kind == 1 && B > 128 && (long)N / 32 > 16L * SEED_MAX_GROUPS &&
        p->rows_per_chunk >= RQ_SPLIT_MIN_ROWS)
        p->rq_split = (int)(p->rows_per_chunk / 8 / RQ_ROWS * RQ_ROWS);
    p->W = p->n_chunks * (p->kind == 1 ? p->rs : 1) * (p->rq_split > 0 ? 2 : 1);
    if (p->W > MERGE_MAX_LISTS)
        return -1;
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
    // candidate overflow: per scan wave, every (row, query) pair of one
    // iteration beyond the LDS staging area
    // (the GEMM-structured scan: per wave, its 64 x 128 values of a macro
    // tile beyond its LDS staging area)
    const long pairs = (long)SCAN_RT * 16 * p->ng * 16;
    p->ovf_cap = p->kind == 0 && pairs > STAGE_CAP ? (int)(pairs - STAGE_CAP)
                 : p->kind == 2                    ? 64 * 128 - GM_STAGE
                                                   : 0;
    p->grid = p->kind == 1 ? p->n_chunks : ((p->n_chunks + 7) / 8) * 8 * p->n_qt;
    const int waves_per_wg = p->kind == 2 ? GM_WAVES : SCAN_WAVES;
    p->off_ovf = off;
    off += align256((size_t)p->grid * waves_per_wg * 3 * (p->ovf_cap > 0 ? p->ovf_cap : 1) * 4);
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
                      float *l_hat, bool inv_dist, hipStream_t s, int phases)
{
    uint8_t *w = (uint8_t *)ws;
    uint32_t *tau = (uint32_t *)(w + p.off_tau);
    float *qn = (float *)(w + p.off_qn);
    float *gmin = (float *)(w + p.off_gmin);
    int32_t *ccnt = (int32_t *)(w + p.off_ccnt);
    uint32_t *ckey = (uint32_t *)(w + p.off_ckey);
    int32_t *cidx = (int32_t *)(w + p.off_cidx);
    hipError_t e;

    if (phases & KNN_LISTS) {
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
            // 16 query groups per workgroup, or 4 for a batch of at most 64
            const int qg = sa.n_qg <= 4 ? 4 : 16;
            const dim3 grid((p.G + SEED_WAVES - 1) / SEED_WAVES, (sa.n_qg + qg - 1) / qg);
            const dim3 block(SEED_WAVES * WAVE);
            if (p.dtype == 1) {
                if (qg == 4)
                    hipLaunchKernelGGL((seed_groups_kernel<1, 4>), grid, block, 0, s, sa);
                else
                    hipLaunchKernelGGL((seed_groups_kernel<1, 16>), grid, block, 0, s, sa);
            } else {
                if (qg == 4)
                    hipLaunchKernelGGL((seed_groups_kernel<0, 4>), grid, block, 0, s, sa);
                else
                    hipLaunchKernelGGL((seed_groups_kernel<0, 16>), grid, block, 0, s, sa);
            }
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
        a.rows_per_chunk = p.rows_per_chunk;
        a.row_lo = 0;
        a.row_hi = p.rows_per_chunk;
        a.n_lists = p.W;
        a.list_base = 0;
        a.tau = tau;
        a.ccnt = ccnt;
        a.ckey = ckey;
        a.cidx = cidx;
        a.ovf = (uint32_t *)(w + p.off_ovf);
        a.ovf_cap = p.ovf_cap;
        const bool timed = t_scan_begin && t_scan_end;
        if (timed && (e = hipEventRecord(t_scan_begin, s)) != hipSuccess)
            return e;
        const bool ragged = p.d % (p.dtype == 1 ? 32 : 16) != 0;
        if (p.kind == 2)
            e = launch_scan_gemm(p, a, s);
        else if (p.kind == 1 && p.rq_split > 0) {
            a.row_hi = p.rq_split;
            e = launch_scan_rq(p, a, s);
            if (e == hipSuccess) {
                hipLaunchKernelGGL(list_bound_kernel, dim3(p.B), dim3(WAVE), 0, s, ccnt, ckey,
                                   p.W, p.W / 2, p.k, tau);
                e = hipGetLastError();
            }
            a.row_lo = p.rq_split;
            a.row_hi = p.rows_per_chunk;
            a.list_base = p.W / 2;
            if (e == hipSuccess)
                e = launch_scan_rq(p, a, s);
        } else if (p.kind == 1)
            e = launch_scan_rq(p, a, s);
        else
            e = p.dtype == 1
                    ? (ragged ? launch_scan_bf16_ragged(p, a, s) : launch_scan_bf16(p, a, s))
                    : (ragged ? launch_scan_f32_ragged(p, a, s) : launch_scan_f32(p, a, s));
        if (e != hipSuccess)
            return e;
        if (timed && (e = hipEventRecord(t_scan_end, s)) != hipSuccess)
            return e;
    }
    if (!(phases & KNN_MERGE))
        return hipSuccess;

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
    m.inv_dist = inv_dist;
    const int lpl = (p.W + WAVE - 1) / WAVE;
    const bool pred = q_hat != nullptr;
    if (lpl <= 1)
        return launch_merge<1>(m, p.B, pred, s);
    if (lpl <= 2)
        return launch_merge<2>(m, p.B, pred, s);
    if (lpl <= 4)
        return launch_merge<4>(m, p.B, pred, s);
    if (lpl <= 8)
        return launch_merge<8>(m, p.B, pred, s);
    if (lpl <= 16)
        return launch_merge<16>(m, p.B, pred, s);
    if (lpl <= 32)
        return launch_merge<32>(m, p.B, pred, s);
    if (lpl <= 64)
        return launch_merge<64>(m, p.B, pred, s);
    return hipErrorInvalidValue;
}

hipError_t launch_predict(const int32_t *nbr_idx, const float *nbr_dist, int B, int k,
                          bool inv_dist, const float *bank_qual, const float *bank_len, int N,
                          int M, float *q_hat, float *l_hat, hipStream_t s)
{
    hipLaunchKernelGGL(predict_kernel, dim3(B), dim3(64), 0, s, nbr_idx,
                       inv_dist ? nbr_dist : nullptr, k, bank_qual, bank_len, N, M, q_hat, l_hat);
    return hipGetLastError();
}

}  // namespace rb
