// The bank scan of the exact k-nearest-neighbour search (RouteBalance Sec. 4.2:
// the KNN lookup of Alg. 1) for a batch whose whole query tile fits in the
// registers of one workgroup: bf16 rows of NKS full k-steps, at most
// (RQ_WAVES / RS) * QW * 16 queries.
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

// Bank fragments travel from HBM to LDS in whole 128-byte lines: one
// global-to-LDS load brings 8 rows x 128 bytes (two k-steps of each row,
// eight 16-byte chunks of one line per group of 8 lanes), so every line is
// fetched by one instruction. In LDS, load f of a stage (row group
// rg = f % 4 of the block, k-step pair f / 4) holds row rg*8 + ri's chunk c
// (quarter c % 4 of k-step 2*(f/4) + c/4) at position
// 8*ri + (c ^ rq_perm(ri) ^ 2*(rg & 1)), rq_perm taking the row pairs of a
// group to 0, 1, 4, 5. The MFMA A-fragment read (lane (col, jg): row col,
// quarter jg of one k-step) then puts the sixteen lanes that LDS serves
// together (lanes 8p..8p+7 and 32+8p..32+8p+7: eight rows at quarters jg
// and jg + 2) on distinct bank groups, as it does the sixteen rows of one
// quarter: no bank conflicts (a plain XOR with the row, which spreads only
// the latter, costs four conflict cycles per read).
__device__ __forceinline__ int rq_perm(int ri)
{
    return ((ri >> 1) & 1) | ((ri >> 2) << 2);
}
__device__ __forceinline__ uint32_t rq_chunk(int ri, int rg, int c)
{
    return (uint32_t)(8 * ri + (c ^ rq_perm(ri) ^ (2 * (rg & 1))));
}

// One workgroup per bank chunk; RQ_WAVES waves, two per SIMD, in RS row
// halves of RQ_WAVES / RS query slots. Wave w owns the queries of slot
// w % (RQ_WAVES / RS), [16*QW*slot, 16*QW*(slot+1)), and holds their
// fragments for every k-step in registers for the whole kernel, so no query
// byte is loaded twice. The chunk goes by in blocks of RQ_ROWS rows (two
// 16-row MFMA tiles); with RS = 1 every wave takes both tiles of a block,
// with RS = 2 the waves of row half h take tile h (so a batch of up to 64
// requests still keeps all eight waves busy). Each block's k-steps are cut
// into SPB stages, which global-to-LDS loads bring in whole 128-byte lines
// into a ring of S slots, S - 1 stages ahead of the MFMAs, so
// that every bank byte crosses from L2 into the compute unit once and serves
// all the waves. Each wave keeps, per owned query, its own list of the k
// best candidates of its rows of the chunk (no other wave touches it) and its
// own candidate threshold; the lists start from the shared bound the seed
// pass computed. A chunk therefore leaves RS lists per query (per pass, when
// the scan takes the rows of every chunk in two launches).
template <int NKS, int QW, int RS, int SPB, int S>
__global__ __launch_bounds__(RQ_WAVES * WAVE, 1) void rq_scan_kernel(const ScanArgs A)
{
    constexpr int TT = RQ_ROWS / 16;
    constexpr int KSTG = NKS / SPB;             // k-steps of one stage
    constexpr int F = KSTG * TT;                // fragments of one stage
    constexpr int FPW = F / RQ_WAVES;           // of them, loaded by each wave
    constexpr int QPW = QW * 16;                // queries of one wave
    constexpr int NQS = RQ_WAVES / RS;          // query slots
    constexpr int TW = TT / RS;                 // tiles of a block each wave takes
    static_assert(NKS % SPB == 0 && F % RQ_WAVES == 0, "whole stages, equal shares");
    static_assert(KSTG % 2 == 0 && TT == 2, "stages of whole k-step pairs, 32-row blocks");
    // With four query groups a wave holds 192 registers of query fragments;
    // both tiles' accumulators would not fit beside them, so such a wave
    // takes the tiles of a block one after the other (one stage per block)
    constexpr bool TSEQ = QW >= 4 && TW == 2;
    constexpr int TA = TSEQ ? 1 : TW;           // tiles whose accumulators are live together
    static_assert(!TSEQ || SPB == 1, "tiles one after the other within one stage");
    static_assert(RS == 1 || RS == 2, "one or two row halves");
    static_assert(RQ_ROWS <= WAVE, "one norm per lane");

    extern __shared__ __align__(16) uint8_t smem[];
    const RqLayout L = rq_layout(A.k, QW, KSTG, S);
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
    const int slot_q = wave % NQS, half = wave / NQS;   // query slot, row half
    const int col = lane & 15, jg = lane >> 4;
    const int k = A.k;
    const uint32_t rowb = (uint32_t)A.d * 2;
    // rows [row_lo, row_hi) of chunk c
    const long cbeg = (long)c * A.rows_per_chunk;
    const long rbeg = cbeg + A.row_lo;
    const long rend = min((long)A.N, cbeg + min(A.rows_per_chunk, A.row_hi));
    const int nrows = rend > rbeg ? (int)(rend - rbeg) : 0;
    const int n_blk = (nrows + RQ_ROWS - 1) / RQ_ROWS;
    const int n_stg = n_blk * SPB;
    const int qw0 = slot_q * QPW;
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
    for (int i = lane; i < QPW; i += WAVE) {
        const int q = qw0 + i;
        qn_w[i] = q < A.B ? A.qn[q] : 0.f;
        tau_w[i] = q < A.B ? A.tau[q] : KEY_NONE;
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
    // this lane's place in a load: row ri of the row group, the chunk of the
    // 128-byte line that lands at its position (rq_chunk inverted)
    const int dri = lane >> 3;
    auto dma_chunk = [&](int rg) { return (lane & 7) ^ rq_perm(dri) ^ (2 * (rg & 1)); };
    auto issue = [&](int z) {
        const int slot = z % S, bz = z / SPB, st = z - bz * SPB;
        const bool real = z < n_stg;
        const __amdgpu_buffer_rsrc_t r = real ? rbk : rnone;
#pragma unroll
        for (int j = 0; j < FPW; ++j) {
            const int f = wave + RQ_WAVES * j;
            const int rg = f % 4, pair = st * (KSTG / 2) + f / 4;
            const uint32_t vo = (uint32_t)(bz * RQ_ROWS + rg * 8 + dri) * rowb +
                                pair * (2 * KSTEP_BYTES) + dma_chunk(rg) * 16;
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

    // the block tile of wave tile t
    auto tile_of = [&](int t) { return RS == 2 ? half : t; };
    // accumulators of wave tiles t0 .. t0+TA-1 from -|x|^2/2 of their rows
    // (-inf for rows past the chunk), the norms of block b in norm slot `slot`
    auto init_acc = [&](f32x4(&ac)[TA][QW], int slot, int b, int t0) {
#pragma unroll
        for (int t = 0; t < TA; ++t) {
            const int tt = tile_of(t0 + t);
            const f32x4 xn = *(const f32x4 *)(nslot + slot * WAVE + tt * 16 + jg * 4);
            f32x4 h;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                h[e] = b * RQ_ROWS + tt * 16 + jg * 4 + e < nrows ? -0.5f * xn[e] : -INFINITY;
#pragma unroll
            for (int g = 0; g < QW; ++g)
                ac[t][g] = h;
        }
    };
    // the MFMAs of stage ST (in slot `slot`) for wave tiles t0 .. t0+TA-1
    auto mfma_tiles = [&](auto ST, f32x4(&ac)[TA][QW], int slot, int t0) {
        constexpr int st = decltype(ST)::value;
        // the lane's A fragment of tile tt, k-step j of the stage: row col of
        // the tile, quarter jg, at load (j/2)*4 + rg
        const i32x4 *fr = ring + slot * F * WAVE;
        uint32_t fbase[TA][2];
#pragma unroll
        for (int t = 0; t < TA; ++t) {
            const int tt = tile_of(t0 + t);
            const int ri = col & 7, rg = tt * 2 + (col >> 3);
#pragma unroll
            for (int h = 0; h < 2; ++h)
                fbase[t][h] = (uint32_t)rg * WAVE + rq_chunk(ri, rg, 4 * h + jg);
        }
        static_for<0, KSTG>([&](auto J) {
            constexpr int j = decltype(J)::value, s = st * KSTG + j;
            i32x4 a[TA];
#pragma unroll
            for (int t = 0; t < TA; ++t)
                a[t] = fr[(j / 2) * 4 * WAVE + fbase[t][j & 1]];
#pragma unroll
            for (int t = 0; t < TA; ++t)
#pragma unroll
                for (int g = 0; g < QW; ++g)
                    ac[t][g] = mfma_step<1>(a[t], qf[g][s], ac[t][g]);
        });
        // two k-steps of fragment reads in flight: the reads of k-steps 0 and
        // 1, then per k-step its MFMAs and the reads two ahead
        __builtin_amdgcn_sched_group_barrier(0x100, 2 * TA, 0);
        static_for<0, KSTG>([&](auto J) {
            __builtin_amdgcn_sched_group_barrier(0x008, TA * QW, 0);
            if constexpr (decltype(J)::value + 2 < KSTG)
                __builtin_amdgcn_sched_group_barrier(0x100, TA, 0);
        });
    };
    // candidates of wave tiles t0 .. t0+TA-1 of block b: acc = -|x|^2/2 +
    // <q, x>, distance |q|^2 - 2*acc; a value passes if acc >= nu of its query
    auto test_tiles = [&](f32x4(&ac)[TA][QW], int b, int t0) {
        static_for<0, QW>([&](auto G) {
            constexpr int g = decltype(G)::value;
            float m = -INFINITY;
#pragma unroll
            for (int t = 0; t < TA; ++t)
                m = fmaxf(m, fmaxf(fmaxf(ac[t][g][0], ac[t][g][1]),
                                   fmaxf(ac[t][g][2], ac[t][g][3])));
            if (!ballot(m >= nu[g]))
                return;
            const float qg = qn_w[g * 16 + col];
#pragma unroll
            for (int t = 0; t < TA; ++t) {
                const int tt = tile_of(t0 + t);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float a = ac[t][g][e];
                    uint64_t mk = ballot(a >= nu[g]);
                    const uint32_t key = f2key(fmaf(-2.f, a, qg));
                    const int32_t idx = (int32_t)(rbeg + b * RQ_ROWS + tt * 16 + jg * 4 + e);
                    while (mk) {
                        const int src = __builtin_ctzll(mk);
                        mk &= mk - 1;
                        insert(g, src & 15, (uint32_t)__builtin_amdgcn_readlane((int)key, src),
                               __builtin_amdgcn_readlane(idx, src));
                    }
                }
            }
        });
    };
    // this wave's part of stage z has landed once at most FPW*(S-2) loads are
    // outstanding (the fragment loads of the S-2 stages issued after it); the
    // barrier then tells that every wave's part has and that every wave is
    // done with stage z - 1, whose slot the next load reuses
    auto next_stage = [&](int z) {
        __builtin_amdgcn_sched_barrier(0);
        wait_vmcnt<FPW * (S - 2)>();
        stream_barrier();
        issue(z + S - 1);
        __builtin_amdgcn_sched_barrier(0);
    };

    int z = 0;   // the stage being consumed
    for (int b = 0; b < n_blk; ++b) {
        if constexpr (TSEQ) {
            // one stage per block; its tiles one after the other, each with
            // its candidate test
            next_stage(z);
            const int slot = z % S;
            if (active) {
                static_for<0, TW>([&](auto T) {
                    f32x4 acc[TA][QW];
                    init_acc(acc, slot, b, T.value);
                    mfma_tiles(Int<0>{}, acc, slot, T.value);
                    test_tiles(acc, b, T.value);
                });
            }
            ++z;
        } else {
            f32x4 acc[TW][QW];
            static_for<0, SPB>([&](auto ST) {
                constexpr int st = decltype(ST)::value;
                next_stage(z);
                const int slot = z % S;
                if constexpr (st == 0) {
                    // the accumulators start from -|x|^2/2 of their rows (-inf
                    // for rows past the chunk)
#pragma unroll
                    for (int t = 0; t < TW; ++t) {
                        const int tt = RS == 2 ? half : t;
                        const f32x4 xn =
                            *(const f32x4 *)(nslot + slot * WAVE + tt * 16 + jg * 4);
                        f32x4 h;
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            h[e] = b * RQ_ROWS + tt * 16 + jg * 4 + e < nrows ? -0.5f * xn[e]
                                                                             : -INFINITY;
#pragma unroll
                        for (int g = 0; g < QW; ++g)
                            acc[t][g] = h;
                    }
                }
                if (active) {
                    // the lane's A fragment of tile tt, k-step j of the stage:
                    // row col of the tile, quarter jg, at load (j/2)*4 + rg
                    const i32x4 *fr = ring + slot * F * WAVE;
                    uint32_t fbase[TW][2];
#pragma unroll
                    for (int t = 0; t < TW; ++t) {
                        const int tt = RS == 2 ? half : t;
                        const int ri = col & 7, rg = tt * 2 + (col >> 3);
#pragma unroll
                        for (int h = 0; h < 2; ++h)
                            fbase[t][h] = (uint32_t)rg * WAVE + rq_chunk(ri, rg, 4 * h + jg);
                    }
                    static_for<0, KSTG>([&](auto J) {
                        constexpr int j = decltype(J)::value, s = st * KSTG + j;
                        i32x4 a[TW];
#pragma unroll
                        for (int t = 0; t < TW; ++t)
                            a[t] = fr[(j / 2) * 4 * WAVE + fbase[t][j & 1]];
#pragma unroll
                        for (int t = 0; t < TW; ++t)
#pragma unroll
                            for (int g = 0; g < QW; ++g)
                                acc[t][g] = mfma_step<1>(a[t], qf[g][s], acc[t][g]);
                    });
                    // two k-steps of fragment reads in flight: the reads of
                    // k-steps 0 and 1, then per k-step its MFMAs and the
                    // reads two ahead
                    __builtin_amdgcn_sched_group_barrier(0x100, 2 * TW, 0);
                    static_for<0, KSTG>([&](auto J) {
                        __builtin_amdgcn_sched_group_barrier(0x008, TW * QW, 0);
                        if constexpr (decltype(J)::value + 2 < KSTG)
                            __builtin_amdgcn_sched_group_barrier(0x100, TW, 0);
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
                for (int t = 0; t < TW; ++t)
                    m = fmaxf(m, fmaxf(fmaxf(acc[t][g][0], acc[t][g][1]),
                                       fmaxf(acc[t][g][2], acc[t][g][3])));
                if (!ballot(m >= nu[g]))
                    return;
                const float qg = qn_w[g * 16 + col];
#pragma unroll
                for (int t = 0; t < TW; ++t) {
                    const int tt = RS == 2 ? half : t;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float a = acc[t][g][e];
                        uint64_t mk = ballot(a >= nu[g]);
                        const uint32_t key = f2key(fmaf(-2.f, a, qg));
                        const int32_t idx =
                            (int32_t)(rbeg + b * RQ_ROWS + tt * 16 + jg * 4 + e);
                        while (mk) {
                            const int src = __builtin_ctzll(mk);
                            mk &= mk - 1;
                            insert(g, src & 15,
                                   (uint32_t)__builtin_amdgcn_readlane((int)key, src),
                                   __builtin_amdgcn_readlane(idx, src));
                        }
                    }
                }
            });
        }
    }

    // ---- the wave's lists -> workspace [B][n_lists][k], list list_base +
    // c*RS + half of each query, valid entries first (no global-to-LDS load
    // may still be in flight when the workgroup ends)
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
        const size_t o = (size_t)q * A.n_lists + A.list_base + c * RS + half;
        if (valid) {
            const int pos = mbcnt(m);
            A.ckey[o * k + pos] = key;
            A.cidx[o * k + pos] = (int32_t)(uint32_t)v;
        }
        if (lane == 0)
            A.ccnt[o] = popc(m);
    }
}

template <int NKS, int QW, int RS, int SPB, int S>
hipError_t launch_rq_scan(const ScanArgs &a, size_t lds, int grid, hipStream_t s)
{
    auto kern = rq_scan_kernel<NKS, QW, RS, SPB, S>;
    hipError_t e = hipFuncSetAttribute((const void *)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(RQ_WAVES * WAVE), lds, s, a);
    return hipGetLastError();
}

// The instantiations of one row length: the (QW, RS) and (SPB, S) the plan
// may choose for it (plan_knn's tables; QW * NKS * 4 registers of query
// fragments stay within 192).
template <int NKS, int QW, int RS>
hipError_t launch_rq_stages(const KnnPlan &p, const ScanArgs &a, hipStream_t s)
{
    if constexpr (NKS == 12) {
        if (p.spb == 1 && p.stages == 4)
            return launch_rq_scan<NKS, QW, RS, 1, 4>(a, p.lds_bytes, p.grid, s);
    } else {
        if (p.spb == 2 && p.stages == 4)
            return launch_rq_scan<NKS, QW, RS, 2, 4>(a, p.lds_bytes, p.grid, s);
        if (p.spb == 2 && p.stages == 2)
            return launch_rq_scan<NKS, QW, RS, 2, 2>(a, p.lds_bytes, p.grid, s);
    }
    if constexpr (NKS != 32)
        if (p.spb == 1 && p.stages == 2)
            return launch_rq_scan<NKS, QW, RS, 1, 2>(a, p.lds_bytes, p.grid, s);
    return hipErrorInvalidValue;
}

template <int NKS>
hipError_t launch_rq_nks(const KnnPlan &p, const ScanArgs &a, hipStream_t s)
{
#define RB_RQ(QW_, RS_)                                                                          \
    if (p.qw == QW_ && p.rs == RS_)                                                             \
        return launch_rq_stages<NKS, QW_, RS_>(p, a, s);
    if constexpr (NKS == 12) {
        RB_RQ(1, 2)
        RB_RQ(2, 2)
        RB_RQ(4, 2)
        RB_RQ(4, 1)
    } else if constexpr (NKS == 16 || NKS == 24) {
        RB_RQ(1, 2)
        RB_RQ(2, 2)
        RB_RQ(2, 1)
    } else if constexpr (NKS == 32) {
        RB_RQ(1, 2)
        RB_RQ(1, 1)
    }
#undef RB_RQ
    return hipErrorInvalidValue;
}

}  // namespace

}  // namespace rb
