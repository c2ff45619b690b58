// The bank scan of the exact k-nearest-neighbour search (RouteBalance Sec. 4.2:
// the KNN lookup of Alg. 1) for a batch whose whole query tile fits in the
// registers of one workgroup: bf16 rows of NKS full k-steps, at most
// RQ_WAVES * QW * 16 queries.
#pragma once

#include "knn_common.hpp"

namespace rb {

namespace {

// Global -> LDS load of 4 bytes per lane (lane l's bytes land at dst + 4*l).
__device__ __forceinline__ void dma4(__amdgpu_buffer_rsrc_t r, float *dst, uint32_t voffset)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void *)dst, 4,
                                             (int)voffset, 0, 0, 0);
}

// One workgroup per bank chunk; RQ_WAVES waves, two per SIMD. Wave w owns
// queries [16*QW*w, 16*QW*(w+1)) and
// holds their fragments for every k-step in registers for the whole kernel,
// so no query byte is loaded twice. The chunk goes by in blocks of RQ_ROWS
// rows; each block's k-steps are cut into
// stages of RQ_KSTG k-steps, which global-to-LDS loads bring into a ring of
// RQ_STAGES slots, RQ_STAGES - 1 stages ahead of the MFMAs, so that every
// bank byte crosses from L2 into the compute unit once and serves all the
// waves. Each wave keeps, per owned query, its own list of the k best
// candidates of the chunk (no other wave touches it) and its own candidate
// threshold; the lists start from the shared bound the seed pass computed.
template <int NKS, int QW>
__global__ __launch_bounds__(RQ_WAVES * WAVE, 1) void rq_scan_kernel(const ScanArgs A)
{
    constexpr int TT = RQ_ROWS / 16, KSTG = RQ_KSTG, S = RQ_STAGES;
    constexpr int F = KSTG * TT;                // fragments of one stage
    constexpr int FPW = F / RQ_WAVES;           // of them, loaded by each wave
    constexpr int SPB = NKS / KSTG;             // stages of one block
    constexpr int QPW = QW * 16;                // queries of one wave
    static_assert(NKS % KSTG == 0 && F % RQ_WAVES == 0, "whole stages, equal shares");
    static_assert(RQ_ROWS <= WAVE, "one norm per lane");

    extern __shared__ __align__(16) uint8_t smem[];
    const RqLayout L = rq_layout(A.k, QW);
    i32x4 *ring = (i32x4 *)(smem + L.ring);              // [S][F][64] fragments
    float *nslot = (float *)(smem + L.norms);            // [S][64] |x|^2 of a block's rows
    uint64_t *lists = (uint64_t *)(smem + L.lists);      // [waves][QPW][k]
    float *qn_l = (float *)(smem + L.qinfo);             // [waves][QPW] |q|^2
    uint32_t *tau_l = (uint32_t *)(smem + L.qinfo) + RQ_WAVES * QPW;   // [waves][QPW] bound

    const int c = blockIdx.x;
    if (c >= A.n_chunks)
        return;
    const int tid = threadIdx.x, lane = tid & 63;
    __builtin_assume(tid < RQ_WAVES * WAVE);
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane & 15, jg = lane >> 4;
    const int k = A.k;
    const uint32_t rowb = (uint32_t)A.d * 2;
    const long rbeg = (long)c * A.rows_per_chunk;
    const long rend = min((long)A.N, rbeg + A.rows_per_chunk);
    const int nrows = rend > rbeg ? (int)(rend - rbeg) : 0;
    const int n_blk = (nrows + RQ_ROWS - 1) / RQ_ROWS;
    const int n_stg = n_blk * SPB;
    const int qw0 = wave * QPW;
    const bool active = qw0 < A.B;   // (a wave past the batch only loads its share)

    // ---- the wave's queries: fragments of every k-step (zero past the batch)
    const __amdgpu_buffer_rsrc_t rq = make_rsrc(A.queries, (uint32_t)A.B * rowb);
    i32x4 qf[QW][NKS];
#pragma unroll
    for (int g = 0; g < QW; ++g) {
        const int q = qw0 + g * 16 + col;
        const uint32_t base = q < A.B ? (uint32_t)q * rowb + jg * 16 : OFF_NONE;
#pragma unroll
        for (int s = 0; s < NKS; ++s)
            qf[g][s] = buffer_load16(rq, base + s * KSTEP_BYTES);
    }
    // |q|^2 and the shared bound from the seed pass of the wave's queries, in
    // LDS (they are needed only for candidates)
    float *qn_w = qn_l + wave * QPW;
    uint32_t *tau_w = tau_l + wave * QPW;
    if (lane < QPW) {
        const int q = qw0 + lane;
        qn_w[lane] = q < A.B ? A.qn[q] : 0.f;
        tau_w[lane] = q < A.B ? A.tau[q] : KEY_NONE;
    }
    // Filter threshold on the accumulators for bound key tk: a value is a
    // candidate if acc >= nu (a superset of distance <= the bound).
    auto nu_of = [](uint32_t tk, float qn, bool valid) -> float {
        const float th = key2f(tk);
        const float v = 0.5f * (qn - th);
        const float nu = v - ldexpf(fabsf(qn) + fabsf(th) + fabsf(v), -21);
        return !valid ? INFINITY : tk == KEY_NONE ? -FLT_MAX : nu;
    };
    // the threshold of the lane's query of each group
    auto nu_q = [&](int i, uint32_t listmax) -> float {
        return nu_of(min(tau_w[i], listmax), qn_w[i], qw0 + i < A.B);
    };
    float nu[QW];
#pragma unroll
    for (int g = 0; g < QW; ++g)
        nu[g] = nu_q(g * 16 + col, KEY_NONE);
    // the wave's lists; empty slots hold distinct sentinels above every entry
    uint64_t *wl = lists + (size_t)wave * QPW * k;
    for (int e = lane; e < QPW * k; e += WAVE)
        wl[e] = pack(KEY_NONE, IDX_NONE - e % k);

    // ---- stage z (block z / SPB, its k-steps from (z % SPB) * KSTG) into
    // slot z % S: this wave's FPW fragments and, with a block's first stage,
    // the last wave loads the block's row norms. Every stage issues the same
    // fragment loads whether or not it fetches anything (past the last block
    // the resource is empty and the slot gets zeros).
    const __amdgpu_buffer_rsrc_t rbk =
        make_rsrc(A.bank + (size_t)rbeg * rowb, (uint32_t)nrows * rowb);
    const __amdgpu_buffer_rsrc_t rnm = make_rsrc(A.bank_norms + rbeg, (uint32_t)nrows * 4u);
    const __amdgpu_buffer_rsrc_t rnone = make_rsrc(A.bank, 0u);
    auto issue = [&](int z) {
        const int slot = z % S, bz = z / SPB, st = z - bz * SPB;
        const bool real = z < n_stg;
        const __amdgpu_buffer_rsrc_t r = real ? rbk : rnone;
#pragma unroll
        for (int j = 0; j < FPW; ++j) {
            const int f = wave + RQ_WAVES * j;
            const int t = f % TT, ks = st * KSTG + f / TT;
            const uint32_t vo =
                (uint32_t)(bz * RQ_ROWS + t * 16 + col) * rowb + ks * KSTEP_BYTES + jg * 16;
            dma16(r, ring + (slot * F + f) * WAVE, vo);
        }
        if (st == 0 && wave == RQ_WAVES - 1)
            dma4(real ? rnm : rnone, nslot + slot * WAVE,
                 lane < RQ_ROWS ? (uint32_t)(bz * RQ_ROWS + lane) * 4u : OFF_NONE);
    };

    // Insert (ckey, cidx) into the list of the wave's query g*16 + cq (a wave
    // call; the list keeps the k smallest pairs inserted so far) and lower
    // that query's threshold to the list's new largest key.
    auto insert = [&](int g, int cq, uint32_t ckey, int32_t cidx) {
        uint64_t *li = wl + (g * 16 + cq) * k;
        const uint64_t cand = pack(ckey, cidx);
        uint64_t v = lane < k ? li[lane] : 0ull;
        uint32_t hi = (uint32_t)(v >> 32), lo = (uint32_t)v;
        reduce_max_pair<WAVE>(hi, lo);
        const uint64_t mx = pack(hi, (int32_t)lo);
        if (cand >= mx)
            return;
        const int pos = __builtin_ctzll(ballot(lane < k && v == mx));
        if (lane == pos) {
            li[lane] = cand;
            v = cand;
        }
        hi = (uint32_t)(v >> 32);
        lo = (uint32_t)v;
        reduce_max_pair<WAVE>(hi, lo);   // hi: an upper bound of the list's largest key
#pragma unroll
        for (int gg = 0; gg < QW; ++gg)
            if (gg == g && col == cq)
                nu[gg] = nu_q(gg * 16 + col, hi);
    };

    // ---- pipeline prologue: stages 0 .. S-2
#pragma unroll
    for (int z = 0; z < S - 1; ++z) {
        __builtin_amdgcn_sched_barrier(0);
        issue(z);
        __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();

    int z = 0;   // the stage being consumed
    for (int b = 0; b < n_blk; ++b) {
        f32x4 acc[TT][QW];
        static_for<0, SPB>([&](auto ST) {
            constexpr int st = decltype(ST)::value;
            // this wave's part of stage z has landed once at most FPW*(S-2)
            // loads are outstanding (the fragment loads of the S-2 stages
            // issued after it); the barrier then tells that every wave's
            // part has and that every wave is done with stage z - 1, whose
            // slot the next load reuses
            __builtin_amdgcn_sched_barrier(0);
            wait_vmcnt<FPW * (S - 2)>();
            stream_barrier();
            issue(z + S - 1);
            __builtin_amdgcn_sched_barrier(0);
            const int slot = z % S;
            if constexpr (st == 0) {
                // the accumulators start from -|x|^2/2 of their rows (-inf
                // for rows past the chunk)
#pragma unroll
                for (int t = 0; t < TT; ++t) {
                    const f32x4 xn = *(const f32x4 *)(nslot + slot * WAVE + t * 16 + jg * 4);
                    f32x4 h;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        h[e] = b * RQ_ROWS + t * 16 + jg * 4 + e < nrows ? -0.5f * xn[e]
                                                                        : -INFINITY;
#pragma unroll
                    for (int g = 0; g < QW; ++g)
                        acc[t][g] = h;
                }
            }
            if (active) {
                const i32x4 *fr = ring + slot * F * WAVE + lane;
                static_for<0, KSTG>([&](auto J) {
                    constexpr int j = decltype(J)::value, s = st * KSTG + j;
                    i32x4 a[TT];
#pragma unroll
                    for (int t = 0; t < TT; ++t)
                        a[t] = fr[(j * TT + t) * WAVE];
#pragma unroll
                    for (int t = 0; t < TT; ++t)
#pragma unroll
                        for (int g = 0; g < QW; ++g)
                            acc[t][g] = mfma_step<1>(a[t], qf[g][s], acc[t][g]);
                });
                // two k-steps of fragment reads in flight: the reads of k-steps
                // 0 and 1, then per k-step its MFMAs and the reads two ahead
                __builtin_amdgcn_sched_group_barrier(0x100, 2 * TT, 0);
                static_for<0, KSTG>([&](auto J) {
                    __builtin_amdgcn_sched_group_barrier(0x008, TT * QW, 0);
                    if constexpr (decltype(J)::value + 2 < KSTG)
                        __builtin_amdgcn_sched_group_barrier(0x100, TT, 0);
                });
            }
            ++z;
        });
        if (!active)
            continue;
        // ---- candidates of the block: acc = -|x|^2/2 + <q, x>, distance
        // |q|^2 - 2*acc; a value passes if acc >= nu of its query
        static_for<0, QW>([&](auto G) {
            constexpr int g = decltype(G)::value;
            float m = -INFINITY;
#pragma unroll
            for (int t = 0; t < TT; ++t)
                m = fmaxf(m, fmaxf(fmaxf(acc[t][g][0], acc[t][g][1]),
                                   fmaxf(acc[t][g][2], acc[t][g][3])));
            if (!ballot(m >= nu[g]))
                return;
            const float qg = qn_w[g * 16 + col];
#pragma unroll
            for (int t = 0; t < TT; ++t)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float a = acc[t][g][e];
                    uint64_t mk = ballot(a >= nu[g]);
                    const uint32_t key = f2key(fmaf(-2.f, a, qg));
                    const int32_t idx = (int32_t)(rbeg + b * RQ_ROWS + t * 16 + jg * 4 + e);
                    while (mk) {
                        const int src = __builtin_ctzll(mk);
                        mk &= mk - 1;
                        insert(g, src & 15, (uint32_t)__builtin_amdgcn_readlane((int)key, src),
                               __builtin_amdgcn_readlane(idx, src));
                    }
                }
        });
    }

    // ---- the wave's lists -> workspace [B][n_chunks][k], valid entries first
    // (no global-to-LDS load may still be in flight when the workgroup ends)
    wait_vmcnt<0>();
    if (!active)
        return;
    for (int i = 0; i < QPW; ++i) {
        const int q = qw0 + i;
        if (q >= A.B)
            break;
        const uint64_t v = lane < k ? wl[i * k + lane] : pack(KEY_NONE, 0);
        const uint32_t key = (uint32_t)(v >> 32);
        const bool valid = key != KEY_NONE;
        const uint64_t m = ballot(valid);
        const size_t o = (size_t)q * A.n_chunks + c;
        if (valid) {
            const int pos = mbcnt(m);
            A.ckey[o * k + pos] = key;
            A.cidx[o * k + pos] = (int32_t)(uint32_t)v;
        }
        if (lane == 0)
            A.ccnt[o] = popc(m);
    }
}

template <int NKS, int QW>
hipError_t launch_rq_scan(const ScanArgs &a, size_t lds, int grid, hipStream_t s)
{
    auto kern = rq_scan_kernel<NKS, QW>;
    hipError_t e = hipFuncSetAttribute((const void *)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(RQ_WAVES * WAVE), lds, s, a);
    return hipGetLastError();
}

}  // namespace

}  // namespace rb
