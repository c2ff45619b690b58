// The bank scan of the exact k-nearest-neighbour search (RouteBalance Sec. 4.2:
// the KNN lookup of Alg. 1): templates, instantiated by the scan_*.hip units.
#pragma once

#include "knn_common.hpp"

namespace rb {

namespace {

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

// One workgroup per (bank chunk, tile of 16*NG queries); SCAN_WAVES waves, two
// per SIMD. Each wave owns 16*RT consecutive rows of every
// SCAN_WAVES*16*RT-row iteration and holds their inner products with all tile
// queries in MFMA accumulators. Bank rows go from HBM straight into MFMA
// operand registers (a ring of R k-steps, loads P k-steps ahead; the SIMD's
// other wave covers the rest of the latency). Query fragments come from LDS:
// the first GR query groups of the tile stay resident for the whole kernel;
// the other groups stream through a double buffer one k-step at a time
// (staged through registers two k-steps ahead), and only they need a
// workgroup barrier per k-step. Candidates that pass a register-level test
// against the per-query bound go through per-wave staging into one list of
// the k best per query shared by the workgroup, maintained with 64-bit
// compare-and-swap so that the waves insert without locks.
template <int DT, int NG, int GR, int RT, bool RAGGED>
__global__ __launch_bounds__(SCAN_THREADS, 1) void scan_kernel(const ScanArgs A)
{
    constexpr int BM = NG * 16;
    constexpr int NS = NG - GR;                    // streamed query groups
    constexpr int VEC = Elem<DT>::VEC, ESZ = Elem<DT>::ESZ;
    constexpr int KS = 4 * VEC;                    // elements of one k-step
    constexpr int RW = RT * 16;                    // rows per wave per iteration
    constexpr int RWG = SCAN_WAVES * RW;           // rows per workgroup iteration
    constexpr int QPT = (NS * WAVE + SCAN_THREADS - 1) / SCAN_THREADS;   // stream items per thread
    constexpr int R = scan_ring<NG>(), P = R - 1, QS = 2;
    static_assert(SCAN_KPAD % R == 0, "padded k-steps fill whole ring cycles");
    constexpr int NB = NG < 4 ? NG : 4;            // query fragments in flight
    static_assert(P < R, "prefetch distance must leave a free ring slot");
    static_assert(R % QS == 0 && R % 2 == 0, "staging slots and LDS buffers divide the unroll");
    static_assert(RW <= WAVE, "one bank-norm load per lane per iteration");

    extern __shared__ __align__(16) uint8_t smem[];
    const int k = A.k, nks = A.nks, nksp = A.nksp;
    const ScanLayout L = scan_layout(NG, GR, nksp, k, RT);
    const i32x4 *res = (const i32x4 *)(smem + L.res);
    i32x4 *strm = (i32x4 *)(smem + L.strm);
    uint64_t *list = (uint64_t *)(smem + L.list);
    float *qn_s = (float *)(smem + L.qn);
    uint32_t *gb_s = (uint32_t *)(smem + L.gb);
    uint32_t *lmk_s = (uint32_t *)(smem + L.lmk);
    uint32_t *nu_s = (uint32_t *)(smem + L.nu);   // float bits

    // Workgroup -> (chunk c, query tile t). Workgroups are dispatched to the
    // eight XCDs round robin, so this map puts every query tile of one chunk
    // on the same XCD.
    const int per8 = 8 * A.n_qt;
    const int rem = blockIdx.x % per8;
    const int t = rem / 8;
    const int c = (blockIdx.x / per8) * 8 + rem % 8;
    if (c >= A.n_chunks)
        return;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    __builtin_assume(tid < SCAN_THREADS);
    const int col = lane & 15, jg = lane >> 4;
    const int q0 = t * BM;
    const long rbeg = (long)c * A.rows_per_chunk;
    const long rend = min((long)A.N, rbeg + A.rows_per_chunk);
    const int n_it = rend > rbeg ? (int)((rend - rbeg + RWG - 1) / RWG) : 0;
    const size_t rowb = (size_t)A.d * ESZ;

    float *nx = (float *)(smem + L.nx) + wave * 2 * RW;
    int *sq = (int *)(smem + L.sq) + wave * STAGE_CAP;
    uint32_t *sk = (uint32_t *)(smem + L.sk) + wave * STAGE_CAP;
    int32_t *si = (int32_t *)(smem + L.si) + wave * STAGE_CAP;

    for (int i = tid; i < BM; i += SCAN_THREADS) {
        const int q = q0 + i;
        qn_s[i] = q < A.B ? A.qn[q] : 0.f;
        gb_s[i] = q < A.B ? A.tau[q] : 0u;
        lmk_s[i] = KEY_NONE;
    }
    // empty list slots hold distinct sentinels above every real entry
    for (int e = tid; e < BM * k; e += SCAN_THREADS)
        list[e] = pack(KEY_NONE, IDX_NONE - e % k);
    // resident groups, every k-step (padding k-steps and lanes past d are zero)
    if constexpr (GR > 0) {
        for (int item = tid; item < nksp * GR * WAVE; item += SCAN_THREADS) {
            const int s = item / (GR * WAVE), g = (item / WAVE) % GR, l = item % WAVE;
            const int q = q0 + g * 16 + (l & 15);
            const bool v = q < A.B && s < nks && (!RAGGED || s * KS + (l >> 4) * VEC < A.d);
            const i32x4 z = {0, 0, 0, 0};
            ((i32x4 *)(smem + L.res))[item] =
                v ? load16(A.queries + (size_t)q * rowb + s * KSTEP_BYTES + (l >> 4) * 16) : z;
        }
    }

    // ---- loads of one k-step through buffer resources whose base moves by one
    // k-step (64 bytes of a row) per step; each lane keeps a fixed offset. Rows
    // past the chunk and queries past the batch fall outside the resource and
    // load zero; so does every lane of a padding k-step (empty resource).
    const uint8_t *bank_c = A.bank + (size_t)rbeg * rowb;
    const uint32_t bank_c_bytes = (uint32_t)((rend - rbeg) * (long)rowb);
    const uint32_t q_bytes = (uint32_t)((size_t)A.B * rowb);
    uint32_t qvo[QPT > 0 ? QPT : 1];   // per stream item: q*rowb + (l/16)*16, or OFF_NONE
    int qkk[QPT > 0 ? QPT : 1];        // element offset of the item within a k-step
#pragma unroll
    for (int i = 0; i < QPT; ++i) {
        const int item = tid + SCAN_THREADS * i;
        const int f = item >> 6, l = item & 63;
        const int q = q0 + (GR + f) * 16 + (l & 15);
        qkk[i] = (l >> 4) * VEC;
        qvo[i] = item < NS * WAVE && q < A.B ? (uint32_t)((size_t)q * rowb + (l >> 4) * 16)
                                             : OFF_NONE;
    }
    int pq_s = 0;             // k-step of the next query load (every iteration is the same)
    int pb_it = 0, pb_s = 0;  // k-step of the next bank load
    uint32_t bvo = (uint32_t)((size_t)(wave * RW + col) * rowb + jg * 16);   // tile 0 of pb_it
    auto issue_q = [&](i32x4(&qs)[QPT > 0 ? QPT : 1]) {
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
    auto stage_queries = [&](int slot, const i32x4(&qs)[QPT > 0 ? QPT : 1]) {
#pragma unroll
        for (int i = 0; i < QPT; ++i) {
            const int item = tid + SCAN_THREADS * i;
            if (item < NS * WAVE)
                strm[slot * NS * WAVE + item] = qs[i];
        }
    };
    // -|x|^2/2 of bank row `lane` of this wave in iteration it (-inf past the chunk)
    auto load_norm = [&](int it) -> float {
        const long row = rbeg + (long)it * RWG + wave * RW + lane;
        const bool v = lane < RW && it < n_it && row < rend;
        const float xn = A.bank_norms[v ? row : 0];
        return v ? -0.5f * xn : -INFINITY;
    };
    // the bound of tile query i as a distance key: the shared bound or the
    // workgroup list's largest key, whichever is lower
    auto bound_key = [&](int i) -> uint32_t {
        return min(lds_load_relaxed(gb_s + i), lds_load_relaxed(lmk_s + i));
    };
    // Filter threshold of tile query i: a value is a candidate if acc >= nu (a
    // superset of distance <= the bound; the exact test follows on insertion).
    auto nu_of = [&](int i) -> float {
        const uint32_t tk = bound_key(i);
        const float qq = qn_s[i], th = key2f(tk);
        const float v = 0.5f * (qq - th);
        const float nu = v - ldexpf(fabsf(qq) + fabsf(th) + fabsf(v), -21);
        return q0 + i >= A.B ? INFINITY : tk == KEY_NONE ? -FLT_MAX : nu;
    };
    // Insert (key, idx) into the list of tile query i; every lane inserts its
    // own candidate. The list always holds the k smallest (key, idx) pairs
    // inserted so far: a new pair replaces the largest slot value by
    // compare-and-swap, retried when another lane or wave changed that slot in
    // between (slot values only decrease, so a slot that still holds the
    // observed maximum is still the maximum). Lanes with nothing to insert
    // pass pend = false.
    auto insert_lanes = [&](bool pend, int i, uint32_t key, int32_t idx) {
        const uint64_t cand = pack(key, idx);
        pend = pend && key <= bound_key(i);
        const uint64_t *li = list + (size_t)i * k;
        while (ballot(pend)) {
            if (pend) {
                uint64_t m = 0, m2 = 0;   // largest and second largest slot value
                int mj = 0;
                for (int j = 0; j < k; ++j) {
                    const uint64_t v = lds_load64(li + j);
                    if (v > m) {
                        m2 = m;
                        m = v;
                        mj = j;
                    } else if (v > m2) {
                        m2 = v;
                    }
                }
                if (cand >= m) {
                    pend = false;
                } else if (lds_cas64(const_cast<uint64_t *>(li) + mj, m, cand)) {
                    // an upper bound of the list's new largest key
                    const uint32_t mk = (uint32_t)((cand > m2 ? cand : m2) >> 32);
                    atomicMin(lmk_s + i, mk);
                    if (mk != KEY_NONE)
                        atomicMin(A.tau + q0 + i, mk);
                    pend = false;
                }
            }
        }
    };
    f32x4 acc[RT][NG];
    i32x4 ring[R][RT];
    i32x4 qst[QS][QPT > 0 ? QPT : 1];
    int s_it = 0;   // k-step within the iteration

    // One block of R k-steps.
    // K-step x (counting over all iterations) reads stream buffer x & 1, which
    // k-step x - 1 filled, and fills the other one for k-step x + 1 after a
    // barrier that every wave reaches once it is done with k-step x - 1.
    // Blocks start at multiples of R, so x & 1 = u & 1.
    auto block = [&]() {
#pragma unroll
        for (int u = 0; u < R; ++u) {
            if constexpr (NS > 0) {
                // (after the last k-step this fills a buffer nobody reads)
                lds_barrier();
                stage_queries((u + 1) & 1, qst[(u + 1) % QS]);
                issue_q(qst[(u + 1) % QS]);
            }
            issue_b(ring[(u + P) % R]);
            const i32x4 *rb = res + s_it * GR * WAVE + lane;
            const i32x4 *sb = strm + (u & 1) * NS * WAVE + lane;
            auto frag = [&](int g) -> i32x4 { return g < GR ? rb[g * WAVE] : sb[(g - GR) * WAVE]; };
            i32x4 bq[NB];
#pragma unroll
            for (int j = 0; j < NB; ++j)
                bq[j] = frag(j);
#pragma unroll
            for (int g = 0; g < NG; ++g) {
#pragma unroll
                for (int tt = 0; tt < RT; ++tt)
                    acc[tt][g] = mfma_step<DT>(ring[u][tt], bq[g % NB], acc[tt][g]);
                if (g + NB < NG)
                    bq[g % NB] = frag(g + NB);
            }
            // keep NB fragment reads in flight: NB reads, then per group its RT
            // MFMAs followed by the read NB groups ahead
            __builtin_amdgcn_sched_group_barrier(0x100, NB, 0);
            static_for<0, NG>([&](auto G) {
                __builtin_amdgcn_sched_group_barrier(0x008, RT, 0);
                if constexpr (decltype(G)::value + NB < NG)
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            });
            ++s_it;
        }
    };

    // each query's threshold, recomputed after every iteration's inserts and
    // bound refresh (a value from before a later lowering of the bound is
    // smaller, so it only lets more candidates through)
    auto refresh_nu = [&](int i) { lds_store_relaxed(nu_s + i, __float_as_uint(nu_of(i))); };
    for (int i = tid; i < BM; i += SCAN_THREADS)
        refresh_nu(i);
    auto nu_read = [&](int i) -> float { return __uint_as_float(lds_load_relaxed(nu_s + i)); };

    // ---- pipeline prologue
#pragma unroll
    for (int u = 0; u < P; ++u)
        issue_b(ring[u]);
    if constexpr (NS > 0) {
#pragma unroll
        for (int j = 0; j < QS; ++j)
            issue_q(qst[j]);
        stage_queries(0, qst[0]);
        issue_q(qst[0]);
    }
    if (lane < RW)
        nx[lane] = load_norm(0);
    float nx_next = load_norm(1);
    __syncthreads();

    for (int it = 0; it < n_it; ++it) {
        // the accumulators start from -|x|^2/2 of their rows
#pragma unroll
        for (int tt = 0; tt < RT; ++tt) {
            const f32x4 nxh = *(const f32x4 *)(nx + (it & 1) * RW + tt * 16 + jg * 4);
#pragma unroll
            for (int g = 0; g < NG; ++g)
                acc[tt][g] = nxh;
        }
        s_it = 0;
        for (int s0 = 0; s0 < nksp; s0 += R)
            block();

        // ---- end of iteration `it`: acc = -|x|^2/2 + <q, x>; dist = |q|^2 - 2*acc
        if (lane < RW)
            nx[((it + 1) & 1) * RW + lane] = nx_next;
        nx_next = load_norm(it + 2);
        // Phase 1: stage every candidate of this iteration, in (group, tile,
        // element, lane) order, in LDS and past STAGE_CAP in this wave's
        // overflow area (an iteration has at most RW*BM of them).
        const long wr0 = rbeg + (long)it * RWG + wave * RW;
        uint32_t *ovf = A.ovf + (size_t)(blockIdx.x * SCAN_WAVES + wave) * 3 * A.ovf_cap;
        int nst = 0;
        // One test per group over its RT*4 accumulators, four groups at a time
        // so that their threshold reads from LDS overlap; then staging for the
        // groups with a hit.
        constexpr int TB = NG < 4 ? NG : 4;
        uint32_t hits = 0;
        static_for<0, NG / TB>([&](auto GB) {
            constexpr int g0 = decltype(GB)::value * TB;
            float nus[TB];
            static_for<0, TB>([&](auto G) { nus[G.value] = nu_read((g0 + G.value) * 16 + col); });
            static_for<0, TB>([&](auto G) {
                constexpr int g = g0 + decltype(G)::value;
                float m = -INFINITY;
                static_for<0, RT>([&](auto TT) {
                    constexpr int tt = decltype(TT)::value;
                    m = fmaxf(m, fmaxf(fmaxf(acc[tt][g][0], acc[tt][g][1]),
                                       fmaxf(acc[tt][g][2], acc[tt][g][3])));
                });
                hits |= ballot(m >= nus[G.value]) ? 1u << g : 0u;
            });
        });
        static_for<0, NG>([&](auto G) {
            constexpr int g = decltype(G)::value;
            if (!(hits >> g & 1u))
                return;
            const int i = g * 16 + col;
            const float nu = nu_read(i);
            const float qq = qn_s[i];
            static_for<0, RT>([&](auto TT) {
                constexpr int tt = decltype(TT)::value;
                static_for<0, 4>([&](auto E) {
                    constexpr int e = decltype(E)::value;
                    const float a = acc[tt][g][e];
                    const bool cnd = a >= nu;
                    const uint64_t mk = ballot(cnd);
                    if (cnd) {
                        const int pos = nst + mbcnt(mk);
                        const uint32_t key = f2key(fmaf(-2.f, a, qq));
                        const int32_t idx = (int32_t)(wr0 + tt * 16 + jg * 4 + e);
                        if (pos < STAGE_CAP) {
                            sq[pos] = i;
                            sk[pos] = key;
                            si[pos] = idx;
                        } else {
                            uint32_t *o = ovf + (pos - STAGE_CAP);
                            o[0] = (uint32_t)i;
                            o[A.ovf_cap] = key;
                            o[2 * A.ovf_cap] = (uint32_t)idx;
                        }
                    }
                    nst += popc(mk);
                });
            });
        });
        // Phase 2 (the accumulators are no longer needed): insert them, 64
        // staged entries per round, one per lane.
        for (int s0 = 0; s0 < nst; s0 += WAVE) {
            const int s = s0 + lane;
            int vi = 0, vx = 0;
            uint32_t vk = 0;
            if (s < min(nst, STAGE_CAP)) {
                vi = sq[s];
                vk = sk[s];
                vx = si[s];
            } else if (s < nst) {
                vi = (int)ovf[s - STAGE_CAP];
                vk = ovf[A.ovf_cap + s - STAGE_CAP];
                vx = (int)ovf[2 * A.ovf_cap + s - STAGE_CAP];
            }
            insert_lanes(s < nst, vi, vk, vx);
        }
        // pick up bounds other workgroups have lowered
        for (int i = tid; i < BM; i += SCAN_THREADS) {
            if (q0 + i < A.B)
                lds_store_relaxed(gb_s + i, __hip_atomic_load(A.tau + q0 + i, __ATOMIC_RELAXED,
                                                              __HIP_MEMORY_SCOPE_AGENT));
            refresh_nu(i);
        }
    }

    // ---- the workgroup's lists -> workspace [B][n_chunks][k], valid entries first
    __syncthreads();
    for (int i = wave; i < BM; i += SCAN_WAVES) {
        const int q = q0 + i;
        if (q >= A.B)
            break;
        const uint64_t v = lane < k ? lds_load64(list + (size_t)i * k + lane) : pack(KEY_NONE, 0);
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

template <int DT, int NG, int GR, bool RAGGED>
hipError_t launch_scan(const ScanArgs &a, size_t lds, int grid, hipStream_t s)
{
    auto kern = scan_kernel<DT, NG, GR, SCAN_RT, RAGGED>;
    hipError_t e = hipFuncSetAttribute((const void *)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(SCAN_THREADS), lds, s, a);
    return hipGetLastError();
}

template <int DT, int NG, bool RAGGED>
hipError_t launch_scan_g(const KnnPlan &p, const ScanArgs &a, int grid, hipStream_t s)
{
    if (p.gr == NG)
        return launch_scan<DT, NG, NG, RAGGED>(a, p.lds_bytes, grid, s);
    if constexpr (NG >= 2)
        if (p.gr == NG / 2)
            return launch_scan<DT, NG, NG / 2, RAGGED>(a, p.lds_bytes, grid, s);
    if constexpr (NG >= 4)
        if (p.gr == NG / 4)
            return launch_scan<DT, NG, NG / 4, RAGGED>(a, p.lds_bytes, grid, s);
    if (p.gr == 0)
        return launch_scan<DT, NG, 0, RAGGED>(a, p.lds_bytes, grid, s);
    return hipErrorInvalidValue;
}

template <int DT, bool RAGGED>
hipError_t launch_scan_r(const KnnPlan &p, const ScanArgs &a, int grid, hipStream_t s)
{
    switch (p.ng) {
    case 16: return launch_scan_g<DT, 16, RAGGED>(p, a, grid, s);
    case 8: return launch_scan_g<DT, 8, RAGGED>(p, a, grid, s);
    case 4: return launch_scan_g<DT, 4, RAGGED>(p, a, grid, s);
    case 2: return launch_scan_g<DT, 2, RAGGED>(p, a, grid, s);
    case 1: return launch_scan_g<DT, 1, RAGGED>(p, a, grid, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace

}  // namespace rb
