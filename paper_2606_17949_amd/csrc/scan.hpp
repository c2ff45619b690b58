// The bank scan of the exact k-nearest-neighbour search (RouteBalance Sec. 4.2:
// the KNN lookup of Alg. 1): templates, instantiated by the scan_*.hip units.
#pragma once

#include "knn_common.hpp"

namespace rb {

namespace {

// One workgroup per (bank chunk, tile of 16*NG queries); SCAN_WAVES waves, two
// per SIMD. Each wave owns 16*RT consecutive rows of every
// SCAN_WAVES*16*RT-row iteration and holds their inner products with all tile
// queries in MFMA accumulators. Bank rows go from HBM straight into MFMA
// operand registers (a ring of R k-steps, loads P = R - 1 k-steps ahead; the
// SIMD's other wave covers the rest of the latency). Query fragments come
// from LDS: the first GR query groups of the tile stay resident for the
// whole kernel; the other groups stream from L2 by global-to-LDS loads into a
// ring of R slots of one k-step each, also P k-steps ahead, and only they
// need a workgroup barrier per k-step. Candidates that pass a register-level test
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
    constexpr int R = scan_ring(DT, NG, GR, RAGGED), P = R - 1;
    static_assert(SCAN_KPAD % R == 0, "padded k-steps fill whole ring cycles");
    constexpr int NB = NG < 4 ? NG : 4;            // query fragments in flight
    // streamed fragments of one k-step: wave w loads fragments w, w + 8, ...;
    // every wave issues NDJ loads per k-step, those past the last fragment
    // into a sink slot
    constexpr int NDJ = (NS + SCAN_WAVES - 1) / SCAN_WAVES;
    static_assert(RW <= WAVE, "one bank-norm load per lane per iteration");

    extern __shared__ __align__(16) uint8_t smem[];
    const int k = A.k, nks = A.nks, nksp = A.nksp;
    const ScanLayout L = scan_layout(NG, GR, nksp, k, RT, R);
    const i32x4 *res = (const i32x4 *)(smem + L.res);
    i32x4 *strm = (i32x4 *)(smem + L.strm);
    i32x4 *sink = strm + R * NS * WAVE;   // target of the loads past the last fragment
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
    const int tid = threadIdx.x, lane = tid & 63;
    __builtin_assume(tid < SCAN_THREADS);
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar branches on it
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
    uint32_t dvo[NDJ > 0 ? NDJ : 1];   // per streamed fragment of this wave: q*rowb + (lane/16)*16
#pragma unroll
    for (int j = 0; j < NDJ; ++j) {
        const int f = wave + SCAN_WAVES * j;
        const int q = q0 + (GR + f) * 16 + col;
        dvo[j] = f < NS && q < A.B ? (uint32_t)((size_t)q * rowb + jg * 16) : OFF_NONE;
    }
    int pq_s = 0;             // k-step of the next query load (every iteration is the same)
    int pb_it = 0, pb_s = 0;  // k-step of the next bank load
    uint32_t bvo = (uint32_t)((size_t)(wave * RW + col) * rowb + jg * 16);   // tile 0 of pb_it
    // this wave's streamed fragments of k-step pq_s into ring slot `slot`
    auto issue_q = [&](int slot) {
        const bool real = pq_s < nks;
        const __amdgpu_buffer_rsrc_t r =
            make_rsrc(A.queries + pq_s * KSTEP_BYTES, real ? q_bytes - pq_s * KSTEP_BYTES : 0u);
        const bool lane_ok = !RAGGED || pq_s * KS + jg * VEC < A.d;
#pragma unroll
        for (int j = 0; j < NDJ; ++j) {
            const int f = wave + SCAN_WAVES * j;
            dma16(r, f < NS ? strm + (slot * NS + f) * WAVE : sink, lane_ok ? dvo[j] : OFF_NONE);
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
    // |x|^2 of bank row `lane` of this wave in iteration it, and whether that
    // row exists; its accumulator start -|x|^2/2 (-inf past the chunk) is
    // formed an iteration later, so that no wait for the load holds up the
    // loads in flight
    auto load_norm = [&](int it, bool &ok) -> float {
        const long row = rbeg + (long)it * RWG + wave * RW + lane;
        ok = lane < RW && it < n_it && row < rend;
        return A.bank_norms[ok ? row : 0];
    };
    auto norm_start = [](float xn, bool ok) -> float { return ok ? -0.5f * xn : -INFINITY; };
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
    int s_it = 0;   // k-step within the iteration

    // One block of R k-steps. K-step x (counting over all iterations; blocks
    // start at multiples of R, so x % R = u) uses bank ring slot u and stream
    // slot u, both loaded at k-step x - P, and loads k-step x + P into the
    // slots of k-step x - 1. Every k-step issues the same loads, in the same
    // order (first the streamed fragments, then the bank rows), whether or not
    // they fetch anything, so a fixed count of later loads tells when this
    // wave's part of stream slot u has landed; the barrier after that wait
    // tells that every wave's part has, and that every wave is done with
    // k-step x - 1.
    auto block = [&]() {
#pragma unroll
        for (int u = 0; u < R; ++u) {
            if constexpr (NS > 0) {
                __builtin_amdgcn_sched_barrier(0);
                wait_vmcnt<RT + (P - 1) * (NDJ + RT)>();
                stream_barrier();
                // (past the last k-step this loads slots nobody reads)
                issue_q((u + P) % R);
                __builtin_amdgcn_sched_barrier(0);
            }
            issue_b(ring[(u + P) % R]);
            const i32x4 *rb = res + s_it * GR * WAVE + lane;
            const i32x4 *sb = strm + u * NS * WAVE + lane;
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

    bool nx_ok;
    const float nx0 = load_norm(0, nx_ok);
    if (lane < RW)
        nx[lane] = norm_start(nx0, nx_ok);

    // ---- pipeline prologue: k-steps 0 .. P-1, in the steady-state order
#pragma unroll
    for (int u = 0; u < P; ++u) {
        if constexpr (NS > 0) {
            __builtin_amdgcn_sched_barrier(0);
            issue_q(u);
            __builtin_amdgcn_sched_barrier(0);
        }
        issue_b(ring[u]);
    }
    float nx_next = load_norm(1, nx_ok);
    // the shared bound of tile query tid as the next refresh takes it (loaded
    // an iteration ahead for the same reason)
    static_assert(BM <= SCAN_THREADS, "one tile query per thread");
    const bool own_q = tid < BM && q0 + tid < A.B;
    uint32_t tau_next = own_q ? A.tau[q0 + tid] : KEY_NONE;
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
        int s0 = 0;
        do {   // (nksp >= R: the loads of at least one block follow those before it)
            block();
            s0 += R;
        } while (s0 < nksp);

        // ---- end of iteration `it`: acc = -|x|^2/2 + <q, x>; dist = |q|^2 - 2*acc
        if (lane < RW)
            nx[((it + 1) & 1) * RW + lane] = norm_start(nx_next, nx_ok);
        nx_next = load_norm(it + 2, nx_ok);
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
        // pick up bounds other workgroups have lowered (as of the previous
        // iteration: the shared bound only decreases, so any value of it is
        // a bound)
        if (tid < BM) {
            if (own_q)
                lds_store_relaxed(gb_s + tid, tau_next);
            refresh_nu(tid);
            if (own_q)
                tau_next = __hip_atomic_load(A.tau + q0 + tid, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
        }
    }

    // ---- the workgroup's lists -> workspace [B][n_chunks][k], valid entries first
    // (no global-to-LDS load may still be in flight when the workgroup ends)
    wait_vmcnt<0>();
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
    if constexpr (NG >= 8)
        if (p.gr == NG / 8)
            return launch_scan<DT, NG, NG / 8, RAGGED>(a, p.lds_bytes, grid, s);
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
