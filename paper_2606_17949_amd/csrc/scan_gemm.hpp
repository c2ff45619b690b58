// The bank scan of the exact k-nearest-neighbour search (RouteBalance Sec. 4.2:
// the KNN lookup of Alg. 1) for large batches, where the distance pass is a
// dense contraction bound by the matrix cores: bf16 rows whose length d is a
// multiple of 64 (at least 128), batches of more than 256 requests.
#pragma once

#include "knn_common.hpp"

namespace rb {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

// One v_mfma_f32_32x32x16_bf16: D = A*B + C over 16 elements of K, A 32 bank
// rows, B 32 requests. Lane l holds, of both operands, row (or request) l % 32
// at K positions 8*(l/32) .. 8*(l/32)+7; of D, request l % 32 of rows
// 8*(r/4) + 4*(l/32) + r%4 in register r.
__device__ __forceinline__ f32x16 mfma32(const i32x4 &a, const i32x4 &b, const f32x16 &c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// One workgroup of GM_WAVES waves (two per SIMD) per (bank chunk, tile of
// GM_QRY requests). The chunk goes by in macro tiles of GM_ROWS rows; wave w
// holds the inner products of rows 64*(w%4) .. +63 with requests
// 128*(w/4) .. +127 of the tile, 2 x 4 tiles of 32 x 32 in 128 accumulator
// registers, while K goes by in stages of GM_KST elements: each stage brings
// the macro tile's rows and the request tile, one 128-byte line of each row,
// from L2 (the other request tiles of the chunk run on the same XCD, so a
// bank row comes from HBM once) into one of two LDS slots. A load brings 8
// rows x 128 bytes; row ri of load group g keeps its 16-byte chunk c at
// position 8*ri + (c ^ ri ^ (g & 1)), which spreads the rows of a fragment
// read over distinct LDS bank groups. A stage is four k-steps of 16; every
// wave reads the fragments of the next k-step while the MFMAs of the
// current one run (12 fragment reads, 32 MFMAs of 32x32x16 per stage and
// wave). The one barrier of a stage sits before its last k-step, whose
// fragments are already in registers: past it, the slot just read takes the
// loads of the stage after next and the fragments of the next stage's first
// k-step are read, so that the matrix cores keep working across the
// barrier. After a macro tile's last stage, every value is tested against
// its request's bound (the seed pass's shared bound, lowered as lists fill)
// and the few that pass go into one list of the k best per request shared by
// the workgroup, kept with 64-bit compare-and-swap.
__global__ __launch_bounds__(GM_WAVES * WAVE, 1) void gemm_scan_kernel(const ScanArgs A)
{
    constexpr int NLOAD = 2 * GM_ROWS / 8;        // loads of one stage: row groups, then request groups
    constexpr int LPW = NLOAD / GM_WAVES;         // of them, issued by each wave
    constexpr int TPR = 2, TPQ = 4;               // 32-row, 32-request tiles per wave
    static_assert(GM_ROWS == 256 && GM_QRY == 256 && GM_KST == 64 && GM_WAVES == 8 && GM_SLOTS == 2,
                  "the wave, load and stage layout below");
    static_assert((LPW / 2) * GM_WAVES == NLOAD / 2,
                  "each wave's first half of loads takes rows, second half requests");

    extern __shared__ __align__(16) uint8_t smem[];
    const int k = A.k;
    const GemmLayout L = gemm_layout(k);
    i32x4 *ring = (i32x4 *)(smem + L.ring);          // [2][NLOAD][64] fragments
    float *nslot = (float *)(smem + L.norms);        // [2][GM_ROWS] |x|^2 of macro tiles rt & 1
    uint64_t *list = (uint64_t *)(smem + L.list);    // [GM_QRY][k] (key << 32 | index)
    float *qn_s = (float *)(smem + L.qn);            // [GM_QRY] |q|^2
    uint32_t *gb_s = (uint32_t *)(smem + L.gb);      // [GM_QRY] snapshot of the shared bound
    uint32_t *lmk_s = (uint32_t *)(smem + L.lmk);    // [GM_QRY] upper bound of each list's largest key
    uint32_t *nu_s = (uint32_t *)(smem + L.nu);      // [GM_QRY] candidate threshold (float bits)

    // Workgroup -> (chunk c, request tile t): workgroups go to the eight
    // XCDs round robin, so every request tile of one of the first
    // 8 * (n_chunks / 8) chunks lands on one XCD. The last n_chunks % 8
    // chunks take the remaining workgroups in order of XCD (x) and then of
    // dispatch (s): rank L among them, chunk base + L / n_qt, tile L % n_qt,
    // so that a chunk's tiles sit on as few XCDs as the counts allow.
    const int per8 = 8 * A.n_qt;
    const int full = (A.n_chunks / 8) * per8;
    int t, c;
    if ((int)blockIdx.x < full) {
        const int rem = blockIdx.x % per8;
        t = rem / 8;
        c = (blockIdx.x / per8) * 8 + rem % 8;
    } else {
        const int j = blockIdx.x - full, x = j % 8, s = j / 8;
        const int tail = (A.n_chunks % 8) * A.n_qt, q = tail / 8, r = tail % 8;
        const int L = x * q + min(x, r) + s;
        t = L % A.n_qt;
        c = s < q + (x < r) ? (A.n_chunks / 8) * 8 + L / A.n_qt : A.n_chunks;
    }
    if (c >= A.n_chunks)
        return;
    const int tid = threadIdx.x, lane = tid & 63;
    __builtin_assume(tid < GM_WAVES * WAVE);
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wr = wave & 3, wq = wave >> 2;   // row quarter, request half of the macro tile
    const int hl = lane >> 5;                  // K half of a fragment
    const uint32_t rowb = (uint32_t)A.d * 2;
    const long rbeg = (long)c * A.rows_per_chunk;
    const long rend = min((long)A.N, rbeg + A.rows_per_chunk);
    const int nrows = rend > rbeg ? (int)(rend - rbeg) : 0;
    const int n_rt = (nrows + GM_ROWS - 1) / GM_ROWS;
    const int nks = A.d / GM_KST;              // stages of one macro tile (at least 2)
    const int n_stg = n_rt * nks;
    const int q0 = t * GM_QRY;
    const int nq = min(GM_QRY, A.B - q0);      // requests of this tile

    static_assert(GM_QRY <= GM_WAVES * WAVE, "one tile request per thread");
    const bool own_q = tid < nq;
    if (tid < GM_QRY) {
        qn_s[tid] = own_q ? A.qn[q0 + tid] : 0.f;
        gb_s[tid] = own_q ? A.tau[q0 + tid] : 0u;
        lmk_s[tid] = KEY_NONE;
    }
    // empty list slots hold distinct sentinels above every real entry
    for (int e = tid; e < GM_QRY * k; e += GM_WAVES * WAVE)
        list[e] = pack(KEY_NONE, IDX_NONE - e % k);

    // ---- stage z (macro tile z / nks, K part z % nks) into slot z & 1: this
    // wave's LPW loads (rows first, then requests) and, with a macro tile's
    // first stage, the last wave loads its 256 row norms. Every stage issues
    // the same loads whether or not they fetch anything (past the last stage
    // the resource is empty and the slot gets zeros); rows past the chunk and
    // requests past the batch fall outside their resources and load zero.
    const __amdgpu_buffer_rsrc_t rbk =
        make_rsrc(A.bank + (size_t)rbeg * rowb, (uint32_t)nrows * rowb);
    const __amdgpu_buffer_rsrc_t rqr =
        make_rsrc(A.queries + (size_t)q0 * rowb, (uint32_t)max(nq, 0) * rowb);
    const __amdgpu_buffer_rsrc_t rnm = make_rsrc(A.bank_norms + rbeg, (uint32_t)nrows * 4u);
    const __amdgpu_buffer_rsrc_t rnone = make_rsrc(A.bank, 0u);
    // Lane l of every load brings row l/8 of its group, chunk
    // (l % 8) ^ (l/8) ^ (g % 2); a wave's groups g = wave + 8*j all have the
    // parity of the wave, so one byte offset serves all of its loads.
    const uint32_t lo = (uint32_t)(lane >> 3) * rowb +
                        (uint32_t)(((lane & 7) ^ (lane >> 3) ^ (wave & 1)) * 16);
    // load j of stage z
    auto issue_load = [&](int z, int j) {
        const int slot = z & 1, rt = z / nks, kc = z - rt * nks;
        const bool real = z < n_stg;
        const bool rows = j < LPW / 2;
        const int f = wave + GM_WAVES * j;                // load index in the stage
        const int r0 = (rows ? rt * GM_ROWS : 0) + 8 * (f & (NLOAD / 2 - 1));
        dma16(real ? (rows ? rbk : rqr) : rnone, ring + (slot * NLOAD + f) * WAVE,
              lo + (uint32_t)r0 * rowb + (uint32_t)kc * (GM_KST * 2));
    };
    // with a macro tile's first stage, the last wave loads the tile's norms
    // into slot rt & 1 (they are read when that stage's MFMAs begin, before
    // the loads of tile rt + 2 reuse the slot)
    auto issue_norms = [&](int z) {
        const int rt = z / nks;
        if (z - rt * nks == 0 && wave == GM_WAVES - 1)
            dma16(z < n_stg ? rnm : rnone, (i32x4 *)(nslot + (rt & 1) * GM_ROWS),
                  (uint32_t)(rt * GM_ROWS * 4 + lane * 16));
    };
    auto issue = [&](int z) {
#pragma unroll
        for (int j = 0; j < LPW; ++j)
            issue_load(z, j);
        issue_norms(z);
    };

    // Fragment places: tile i of the wave's rows (row ra = 64*wr + 32*i +
    // lane%32: load group ra/8, row ra%8 in it) has chunk cq = 2*s + hl of
    // its k-step s at position (ra/8)*64 + 8*(ra%8) + (cq ^ (ra%8) ^ (ra/8 % 2))
    // of the slot; the same for the requests (tile u: 128*wq + 32*u +
    // lane%32) in the second half of the slot. As a byte address:
    // p ^ (32*s) ^ (slot << 16), p the address of k-step 0 in slot 0 (the
    // ring starts the LDS allocation and a slot is 64 KiB).
    static_assert(NLOAD * WAVE * 16 == 1 << 16, "slot offset as one address bit");
    uint32_t pa[TPR], pb[TPQ];
#pragma unroll
    for (int i = 0; i < TPR; ++i) {
        const int ra = 64 * wr + 32 * i + (lane & 31);
        pa[i] = (uint32_t)((ra >> 3) * WAVE + 8 * (ra & 7) + (hl ^ (ra & 7) ^ ((ra >> 3) & 1))) * 16;
    }
#pragma unroll
    for (int u = 0; u < TPQ; ++u) {
        const int rq = 128 * wq + 32 * u + (lane & 31);
        pb[u] = (uint32_t)((NLOAD / 2 + (rq >> 3)) * WAVE + 8 * (rq & 7) +
                           (hl ^ (rq & 7) ^ ((rq >> 3) & 1))) * 16;
    }
    // fragments of k-step s from the slot whose address bit is sx
    auto frag_a = [&](uint32_t sx, auto S, int i) -> i32x4 {
        return *(const i32x4 *)(smem + L.ring + (pa[i] ^ (sx ^ (32u * decltype(S)::value))));
    };
    auto frag_b = [&](uint32_t sx, auto S, int u) -> i32x4 {
        return *(const i32x4 *)(smem + L.ring + (pb[u] ^ (sx ^ (32u * decltype(S)::value))));
    };
    f32x16 acc[TPR][TPQ];
    // the MFMAs of one k-step on (fa, fb), request tile by request tile;
    // with NEXT, the fragments of k-step S of the slot at sx come in
    // meanwhile: the row fragments first, each request fragment as soon as
    // the MFMAs that read its register have been issued; with LOADS, loads
    // j0 .. j0+3 of stage zl go out one per request tile, so that the
    // address unit takes them while the matrix cores work
    auto mma_step = [&](i32x4(&fa)[TPR], i32x4(&fb)[TPQ], uint32_t sx, auto S, auto NEXT,
                        auto LOADS, int zl, int j0) {
        constexpr bool next = decltype(NEXT)::value, loads = decltype(LOADS)::value;
        // (no instruction moves across a k-step's bounds, which keeps the
        // fragments of at most two k-steps live)
        __builtin_amdgcn_sched_barrier(0);
        i32x4 na[TPR];
        if constexpr (next) {
#pragma unroll
            for (int i = 0; i < TPR; ++i)
                na[i] = frag_a(sx, S, i);
        }
#pragma unroll
        for (int u = 0; u < TPQ; ++u) {
#pragma unroll
            for (int i = 0; i < TPR; ++i)
                acc[i][u] = mfma32(fa[i], fb[u], acc[i][u]);
            if constexpr (next)
                fb[u] = frag_b(sx, S, u);
            if constexpr (loads)
                issue_load(zl, j0 + u);
        }
        if constexpr (next) {
#pragma unroll
            for (int i = 0; i < TPR; ++i)
                fa[i] = na[i];
        }
        // the order above, kept by the scheduler
        if constexpr (next)
            __builtin_amdgcn_sched_group_barrier(0x100, TPR, 0);
        static_for<0, TPQ>([&](auto) {
            __builtin_amdgcn_sched_group_barrier(0x008, TPR, 0);
            if constexpr (next)
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            if constexpr (loads)
                __builtin_amdgcn_sched_group_barrier(0x010, 1, 0);
        });
        __builtin_amdgcn_sched_barrier(0);
    };
    static_assert(LPW == 2 * TPQ, "a stage's loads: two k-steps of one load per request tile");

    // the bound of tile request i as a distance key: the shared bound or the
    // workgroup list's largest key, whichever is lower
    auto bound_key = [&](int i) -> uint32_t {
        return min(lds_load_relaxed(gb_s + i), lds_load_relaxed(lmk_s + i));
    };
    // filter threshold of tile request i: a value is a candidate if acc >= nu
    // (a superset of distance <= the bound; the exact test follows on insertion)
    auto nu_of = [&](int i) -> float {
        const uint32_t tk = bound_key(i);
        const float qq = qn_s[i], th = key2f(tk);
        const float v = 0.5f * (qq - th);
        const float nu = v - ldexpf(fabsf(qq) + fabsf(th) + fabsf(v), -21);
        return i >= nq ? INFINITY : tk == KEY_NONE ? -FLT_MAX : nu;
    };
    // Insert (key, idx) into the list of tile request i; every lane inserts
    // its own candidate. The list always holds the k smallest (key, idx)
    // pairs inserted so far: a new pair replaces the largest slot value by
    // compare-and-swap, retried when another lane or wave changed that slot in
    // between (slot values only decrease, so a slot that still holds the
    // observed maximum is still the maximum).
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
    // per-wave staging of a macro tile's candidates: tile request, distance
    // key, bank row; past GM_STAGE entries in this wave's overflow area of
    // the workspace (a macro tile gives a wave at most 64 x 128 of them)
    int *sq = (int *)(smem + L.sq) + wave * GM_STAGE;
    uint32_t *sk = (uint32_t *)(smem + L.sk) + wave * GM_STAGE;
    int32_t *si = (int32_t *)(smem + L.si) + wave * GM_STAGE;
    uint32_t *ovf = A.ovf + (size_t)(blockIdx.x * GM_WAVES + wave) * 3 * A.ovf_cap;

    // the shared bound of tile request tid as the next refresh takes it
    // (loaded a macro tile ahead, so that no wait for it holds up the loads)
    uint32_t tau_next = own_q ? A.tau[q0 + tid] : KEY_NONE;
    __builtin_amdgcn_sched_barrier(0);
    issue(0);
#pragma unroll
    for (int j = 0; j < LPW / 2; ++j)
        issue_load(1, j);
    // stage 0 has landed once at most the first half of the loads of stage 1
    // is outstanding; after the barrier, every wave's part has
    wait_vmcnt<LPW / 2>();
    stream_barrier();
    __builtin_amdgcn_sched_barrier(0);
    i32x4 fa[TPR], fb[TPQ];
#pragma unroll
    for (int i = 0; i < TPR; ++i)
        fa[i] = frag_a(0u, Int<0>{}, i);
#pragma unroll
    for (int u = 0; u < TPQ; ++u)
        fb[u] = frag_b(0u, Int<0>{}, u);
    for (int z = 0, rt = 0, kc = 0; z < n_stg; ++z) {
        const uint32_t rs = (uint32_t)(z & 1) << 16, rn = rs ^ (1u << 16);
        if (kc == 0) {
            // a macro tile's accumulators start from -|x|^2/2 of their rows
            // (-inf for rows past the chunk), so that they end as
            // <q, x> - |x|^2/2; the tile's norms landed two barriers ago
            const float *nm = nslot + (rt & 1) * GM_ROWS;
#pragma unroll
            for (int i = 0; i < TPR; ++i) {
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int r0 = 64 * wr + 32 * i + 8 * g + 4 * hl;
                    const f32x4 xn = *(const f32x4 *)(nm + r0);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float h = rt * GM_ROWS + r0 + e < nrows ? -0.5f * xn[e] : -INFINITY;
#pragma unroll
                        for (int u = 0; u < TPQ; ++u)
                            acc[i][u][4 * g + e] = h;
                    }
                }
            }
        }
        // k-steps 0-2 of the stage, each with the next one's fragment reads;
        // k-step 0 also sends the second half of the loads of stage z + 1
        mma_step(fa, fb, rs, Int<1>{}, Bool<true>{}, Bool<true>{}, z + 1, LPW / 2);
        mma_step(fa, fb, rs, Int<2>{}, Bool<true>{}, Bool<false>{}, 0, 0);
        mma_step(fa, fb, rs, Int<3>{}, Bool<true>{}, Bool<false>{}, 0, 0);
        // this wave's loads of stage z + 1 (sent with the previous stage's
        // last k-step and this stage's first) have landed and its reads of
        // slot z & 1 are done; after the barrier the same holds for every
        // wave, so the slot takes stage z + 2
        __builtin_amdgcn_sched_barrier(0);
        wait_vmcnt<0>();
        stream_barrier();
        if (kc == 0) {
            // pick up bounds other workgroups have lowered (the previous
            // macro tile's inserts are done: every wave passed the barrier);
            // the test of this macro tile comes at least one barrier later.
            // (Before the next loads, so that nothing here waits for them.)
            if (own_q)
                lds_store_relaxed(gb_s + tid, tau_next);
            if (tid < GM_QRY)
                lds_store_relaxed(nu_s + tid, __float_as_uint(nu_of(tid)));
            if (own_q)
                tau_next = __hip_atomic_load(A.tau + q0 + tid, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
        }
        // k-step 3, with the reads of the next stage's first k-step and the
        // first half of the loads of stage z + 2 (after a macro tile's last
        // stage the fragments are read again once its values are out, which
        // keeps them from being held through that work)
        issue_norms(z + 2);
        mma_step(fa, fb, rn, Int<0>{}, Bool<true>{}, Bool<true>{}, z + 2, 0);
        if (kc != nks - 1) {
            ++kc;
            continue;
        }
        kc = 0;
        // ---- end of macro tile rt: acc = v = <q, x> - |x|^2/2 (-inf for rows
        // past the chunk), distance |q|^2 - 2*v. Phase 1: stage every
        // candidate (v >= nu of its request), in (row tile, request tile,
        // register, lane) order.
        const int rbase = rt * GM_ROWS;
        int nst = 0;
        float nus[TPQ];
#pragma unroll
        for (int u = 0; u < TPQ; ++u)
            nus[u] = __uint_as_float(lds_load_relaxed(nu_s + 128 * wq + 32 * u + (lane & 31)));
        // one 32 x 32 tile at a time (the scheduling barriers keep the
        // compiler from reading every accumulator out at once)
        static_for<0, TPR>([&](auto I) {
            constexpr int i = decltype(I)::value;
            static_for<0, TPQ>([&](auto U) {
                constexpr int u = decltype(U)::value;
                const int qi = 128 * wq + 32 * u + (lane & 31);
                __builtin_amdgcn_sched_barrier(0);
                const f32x16 &v = acc[i][u];
                float m = v[0];
#pragma unroll
                for (int r = 1; r < 16; ++r)
                    m = fmaxf(m, v[r]);
                if (ballot(m >= nus[u])) {
                    const float qq = qn_s[qi];
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const bool cnd = v[r] >= nus[u];
                        const uint64_t mk = ballot(cnd);
                        if (cnd) {
                            const int pos = nst + mbcnt(mk);
                            const uint32_t key = f2key(fmaf(-2.f, v[r], qq));
                            const int row = 64 * wr + 32 * i + 8 * (r / 4) + 4 * hl + (r % 4);
                            const int32_t idx = (int32_t)(rbeg + (long)rbase + row);
                            if (pos < GM_STAGE) {
                                sq[pos] = qi;
                                sk[pos] = key;
                                si[pos] = idx;
                            } else {
                                uint32_t *o = ovf + (pos - GM_STAGE);
                                o[0] = (uint32_t)qi;
                                o[A.ovf_cap] = key;
                                o[2 * A.ovf_cap] = (uint32_t)idx;
                            }
                        }
                        nst += popc(mk);
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            });
        });
        // Phase 2 (the accumulators are no longer read): insert them, 64
        // staged entries per round, one per lane.
        for (int s0 = 0; s0 < nst; s0 += WAVE) {
            const int sx = s0 + lane;
            int vi = 0, vx = 0;
            uint32_t vk = 0;
            if (sx < min(nst, GM_STAGE)) {
                vi = sq[sx];
                vk = sk[sx];
                vx = si[sx];
            } else if (sx < nst) {
                vi = (int)ovf[sx - GM_STAGE];
                vk = ovf[A.ovf_cap + sx - GM_STAGE];
                vx = (int)ovf[2 * A.ovf_cap + sx - GM_STAGE];
            }
            insert_lanes(sx < nst, vi, vk, vx);
        }
#pragma unroll
        for (int i = 0; i < TPR; ++i)
            fa[i] = frag_a(rn, Int<0>{}, i);
#pragma unroll
        for (int u = 0; u < TPQ; ++u)
            fb[u] = frag_b(rn, Int<0>{}, u);
        ++rt;
    }

    // ---- the workgroup's lists -> workspace [B][n_chunks][k], valid entries
    // first (no global-to-LDS load may still be in flight when the workgroup
    // ends)
    wait_vmcnt<0>();
    __syncthreads();
    for (int i = wave; i < nq; i += GM_WAVES) {
        const int q = q0 + i;
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

}  // namespace

}  // namespace rb
