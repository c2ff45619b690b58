// Request-instance scoring and the greedy online assignment (RouteBalance
// Eq. 1 score, Eq. 2 cost, the dead-reckoned latency of Sec. 4.2, and the
// greedy per-batch loop of Alg. 1), for gfx950.
//
// Both kernels evaluate the score with the same arithmetic (explicit fused
// multiply-adds, reciprocal rates, and the two Eq. 1 ratios as IEEE divisions
// so that the instance at a maximum gets exactly 1), so the dense score matrix
// and the scores the greedy loop sees at the batch-start state agree bit for
// bit.
#include "common.hpp"
#include "kernels.hpp"

namespace rb {

namespace {

// Latency of a request with prompt l and predicted output lv on an instance
// with queued prefill p, active decode a and reciprocal rates rP = 1/P,
// rD = 1/D: the queued prefill plus this prompt drains at P, then the active
// decode plus this output at D.
__device__ __forceinline__ float latency(float p, float a, float rP, float rD, float l, float lv)
{
    return fmaf(p + l, rP, (a + lv) * rD);
}

// Eq. 2 expected cost: input tokens at the input price plus predicted output
// tokens at the output price.
__device__ __forceinline__ float cost(float l, float lv, float cin, float cout)
{
    return fmaf(l, cin, lv * cout);
}

// x / max, or 0 for a zero maximum.
__device__ __forceinline__ float ratio(float x, float m) { return m > 0.f ? x / m : 0.f; }

// The state-independent part of Eq. 1: w_qual*Q + w_cost*(1 - C/Cmax).
__device__ __forceinline__ float base_score(float qv, float C, float cmax, float wq, float wc)
{
    return fmaf(wq, qv, wc * (1.f - ratio(C, cmax)));
}

// Eq. 1: base + w_lat*(1 - T/Tmax).
__device__ __forceinline__ float full_score(float base, float T, float tmax, float wl)
{
    return fmaf(wl, 1.f - ratio(T, tmax), base);
}

// Alg. 1 budget filter on the Eq. 2 cost C of a request with budget b, and
// the availability mask: whether instance i is a candidate.
__device__ __forceinline__ bool admitted(float C, float b, const uint8_t *mask, int i)
{
    return (!mask || mask[i] != 0) && C <= b;
}

// One wave per request row of the dense score matrix. With a budget or a
// mask (opt.budget, opt.mask; opt.order is not read) the maxima run over the
// request's candidates and the other instances score NaN, as in the greedy
// loop's first step.
__global__ __launch_bounds__(256) void score_kernel(const float *__restrict__ q_hat,
                                                    const float *__restrict__ l_hat,
                                                    const int32_t *__restrict__ plen, int B, int M,
                                                    const InstArgs in, int I, float wq, float wl,
                                                    float wc, const AssignOpts opt,
                                                    float *__restrict__ S0)
{
    const int lane = lane_id();
    const int r = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    if (r >= B)
        return;
    const float l = (float)plen[r];
    const float *qr = q_hat + (size_t)r * M;
    const float *lr = l_hat + (size_t)r * M;
    const float nan = __builtin_nanf("");
    const float budget = opt.budget ? opt.budget[r] : INFINITY;
    float cmax = -INFINITY, tmax = -INFINITY;
    for (int i = lane; i < I; i += WAVE) {
        const int m = in.model[i];
        const float lv = (unsigned)m < (unsigned)M ? lr[m] : nan;
        const float C = cost(l, lv, in.cin[i], in.cout[i]);
        if (!admitted(C, budget, opt.mask, i))
            continue;
        cmax = fmaxf(cmax, C);
        tmax = fmaxf(tmax, latency(in.p[i], in.a[i], 1.f / in.P[i], 1.f / in.D[i], l, lv));
    }
    cmax = wave_max(cmax);
    tmax = wave_max(tmax);
    for (int i = lane; i < I; i += WAVE) {
        const int m = in.model[i];
        const bool mv = (unsigned)m < (unsigned)M;
        const float lv = mv ? lr[m] : nan;
        const float qv = mv ? qr[m] : nan;
        const float C = cost(l, lv, in.cin[i], in.cout[i]);
        const float T = latency(in.p[i], in.a[i], 1.f / in.P[i], 1.f / in.D[i], l, lv);
        S0[(size_t)r * I + i] = admitted(C, budget, opt.mask, i)
                                    ? full_score(base_score(qv, C, cmax, wq, wc), T, tmax, wl)
                                    : nan;
    }
}

// Longest-predicted-first order (Alg. 1; Sec. 4.1 keys a request by the
// maximum over models of its predicted length). Each request's position is
// the number of requests before it under (key descending, index ascending),
// a total order, so the positions form a permutation: order[pos] = r. Every
// workgroup ranks LPT_THREADS requests against all B keys, which it computes
// tile by tile into LDS.
constexpr int LPT_THREADS = 256;

__global__ __launch_bounds__(LPT_THREADS) void lpt_order_kernel(const float *__restrict__ l_hat,
                                                                 int B, int M,
                                                                 int32_t *__restrict__ order)
{
    __shared__ uint64_t keys[LPT_THREADS];
    // ascending in this 64-bit key is descending in the length, then
    // ascending in the index
    auto key_of = [&](int r) {
        const float *row = l_hat + (size_t)r * M;
        float mx = row[0];
        for (int m = 1; m < M; ++m)
            mx = fmaxf(mx, row[m]);
        return ((uint64_t)~f2key(mx) << 32) | (uint32_t)r;
    };
    const int r = blockIdx.x * LPT_THREADS + threadIdx.x;
    const uint64_t mine = r < B ? key_of(r) : ~0ull;
    int pos = 0;
    for (int base = 0; base < B; base += LPT_THREADS) {
        const int s = base + threadIdx.x;
        keys[threadIdx.x] = s < B ? key_of(s) : ~0ull;
        __syncthreads();
        const int n = min(LPT_THREADS, B - base);
        for (int j = 0; j < n; ++j)
            pos += keys[j] < mine ? 1 : 0;
        __syncthreads();
    }
    if (r < B)
        order[pos] = r;
}

// Greedy assignment. Wave 0 runs the sequential loop over requests; waves
// 1..15 fill, one chunk of steps ahead, an LDS double buffer with what does
// not depend on the state: per (request, instance) the base score and the
// predicted output length on the instance's model. Step t decides request
// order[t] (arrival order when order is null). An instance outside the
// request's candidate set (unavailable in mask, or over the request's budget
// in the Eq. 2 cost) gets a NaN base score: it is left out of both maxima and
// never picked. WIDTH = 16 (I <= 16):
// instance i = lane % 16, replicated in the four rows of 16 lanes, so every
// reduction stays inside a row and leaves its result in every lane. WIDTH = 64:
// instance i = lane + 64*u in register slot u. Per request: the latency
// maximum, then the pick. Latencies are positive (queues and lengths are
// non-negative, prompts at least one token, rates positive), so the Eq. 1
// score orders the candidates as S*Tmax = base*Tmax + w_lat*(Tmax - T) does,
// which needs no division; both T and S*Tmax are non-negative (scores lie in
// [0, 1]), so their float bits order as unsigned integers, and one more than
// the bits of S*Tmax is never 0, which marks a non-candidate. One unsigned
// maximum, a ballot of the lanes that hold it and a find-first-set give the
// largest score and, among equal scores, the lowest instance index;
// the lanes holding that instance update its state. The pick's base score,
// latency and Tmax are captured, one step per lane, and every 64 steps the
// wave writes the picks and computes their Eq. 1 scores (with the division,
// exactly as the dense score kernel does) in one vector pass. A request
// without candidates gets -1 and changes no state.
// 16 waves; 8 for 16 register slots per lane (more than 512 instances), whose
// state and scores need the larger register share of a half-size workgroup
template <int IPL>
constexpr int assign_threads() { return IPL >= 16 ? 512 : 1024; }
constexpr int ASSIGN_LDS_FLOATS = 8192;   // per buffer: chunk rows x instances x 2

template <int IPL, int WIDTH>
__global__ __launch_bounds__(assign_threads<IPL>()) void assign_kernel(
    const float *__restrict__ q_hat, const float *__restrict__ l_hat,
    const int32_t *__restrict__ plen, int B, int M, const InstArgs in, int I, float wq, float wl,
    float wc, const AssignOpts opt, int32_t *__restrict__ assign, float *__restrict__ chosen,
    float *__restrict__ decided)
{
    static_assert(WIDTH == 64 || IPL == 1, "a 16-lane row holds one slot");
    constexpr int IP = IPL * WIDTH;                       // instances per LDS row
    constexpr int CH = ASSIGN_LDS_FLOATS / (2 * IP);      // requests per chunk
    __shared__ float base_s[2][CH][IP];
    __shared__ float lv_s[2][CH][IP];
    __shared__ float l_s[2][CH];
    __shared__ int32_t r_s[2][CH];
    const int lane = lane_id(), wave = threadIdx.x >> 6;
    const int n_ch = (B + CH - 1) / CH;
    auto inst = [&](int u) { return WIDTH == 16 ? (lane & 15) : lane + WAVE * u; };
    // maximum over the instance set, as an unsigned maximum of order-preserving
    // keys (a DPP step folds into one v_max_u32; no NaN canonicalisation)
    auto fmax_all = [&](float v) {
        const auto umax = [](uint32_t x, uint32_t y) { return x > y ? x : y; };
        if constexpr (WIDTH == 16)
            return key2f(row16_reduce(f2key(v), umax));
        else
            return key2f(wave_reduce(f2key(v), umax));
    };

    // producers: step t = c*CH + j into slot j of buffer c & 1, one wave per step
    auto produce = [&](int c) {
        const int buf = c & 1;
        for (int j = wave - 1; j < CH; j += assign_threads<IPL>() / WAVE - 1) {
            const int t = c * CH + j;
            if (t >= B)
                break;
            const int r = opt.order ? opt.order[t] : t;
            const float l = (float)plen[r];
            const float *qr = q_hat + (size_t)r * M;
            const float *lr = l_hat + (size_t)r * M;
            const float budget = opt.budget ? opt.budget[r] : INFINITY;
            float qv[IPL], lv[IPL], C[IPL];
            bool cand[IPL];
            float cmax = -INFINITY;
#pragma unroll
            for (int u = 0; u < IPL; ++u) {
                const int i = inst(u);
                const int m = i < I ? in.model[i] : -1;
                const bool ok = (unsigned)m < (unsigned)M;
                qv[u] = ok ? qr[m] : 0.f;
                lv[u] = ok ? lr[m] : 0.f;
                C[u] = cost(l, lv[u], ok ? in.cin[i] : 0.f, ok ? in.cout[i] : 0.f);
                // Alg. 1 budget filter on the Eq. 2 cost, and availability
                cand[u] = ok && admitted(C[u], budget, opt.mask, i);
                if (cand[u])
                    cmax = fmaxf(cmax, C[u]);
            }
            cmax = fmax_all(cmax);
            if (lane < (WIDTH == 16 ? 16 : WAVE)) {
#pragma unroll
                for (int u = 0; u < IPL; ++u) {
                    base_s[buf][j][lane + WAVE * u] =
                        cand[u] ? base_score(qv[u], C[u], cmax, wq, wc) : __builtin_nanf("");
                    lv_s[buf][j][lane + WAVE * u] = lv[u];
                }
            }
            if (lane == 0) {
                l_s[buf][j] = l;
                r_s[buf][j] = r;
            }
        }
    };

    if (wave > 0) {
        produce(0);
        __syncthreads();
        for (int c = 0; c < n_ch; ++c) {
            if (c + 1 < n_ch)
                produce(c + 1);
            __syncthreads();
        }
        return;
    }

    // consumer: instance state in registers
    const int col = WIDTH == 16 ? (lane & 15) : lane;   // this lane's column of an LDS row
    float p[IPL], a[IPL], rP[IPL], rD[IPL];
    bool valid[IPL];
#pragma unroll
    for (int u = 0; u < IPL; ++u) {
        const int i = inst(u);
        // an instance whose model id is outside [0, M) is never chosen
        const int m = i < I ? in.model[i] : -1;
        valid[u] = (unsigned)m < (unsigned)M;
        p[u] = valid[u] ? in.p[i] : 0.f;
        a[u] = valid[u] ? in.a[i] : 0.f;
        rP[u] = valid[u] ? 1.f / in.P[i] : 0.f;
        rD[u] = valid[u] ? 1.f / in.D[i] : 0.f;
    }
    const auto umax = [](uint32_t x, uint32_t y) { return x > y ? x : y; };
    // maximum over the instance set (every lane of the row, or of the wave)
    auto umax_all = [&](uint32_t v) {
        if constexpr (WIDTH == 16)
            return row16_reduce(v, umax);
        else
            return wave_reduce(v, umax);
    };
    // Steps go in blocks of 64: lane s holds step (block + s)'s request index
    // and prompt length, read from LDS once per block (a step takes its
    // prompt length with a lane read, not an LDS round trip), and captures
    // that step's pick.
    int cap_i = -1;
    float cap_b = 0.f, cap_t = 0.f, cap_m = 0.f;
    __syncthreads();   // chunk 0 is ready
    for (int c = 0; c < n_ch; ++c) {
        const int buf = c & 1;
        const int rows = min(CH, B - c * CH);
        float bs[IPL], lv[IPL];
#pragma unroll
        for (int u = 0; u < IPL; ++u) {
            bs[u] = base_s[buf][0][col + WAVE * u];
            lv[u] = lv_s[buf][0][col + WAVE * u];
        }
        for (int jb = 0; jb < rows; jb += WAVE) {
            const int nb = min(WAVE, rows - jb);   // steps of this block
            const int jj = jb + min(lane, nb - 1);
            const int rblk = r_s[buf][jj];
            const float lblk = l_s[buf][jj];
            for (int slot = 0; slot < nb; ++slot) {
                const int j = jb + slot;
                const float l = __builtin_bit_cast(
                    float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, lblk), slot));
                // next step's values, in flight while this one is decided
                const int jn = j + 1 < rows ? j + 1 : j;
                float bsn[IPL], lvn[IPL];
#pragma unroll
                for (int u = 0; u < IPL; ++u) {
                    bsn[u] = base_s[buf][jn][col + WAVE * u];
                    lvn[u] = lv_s[buf][jn][col + WAVE * u];
                }
                // latency maximum over the candidates (a non-candidate, NaN
                // base score, contributes 0)
                float T[IPL];
                uint32_t tb = 0;
#pragma unroll
                for (int u = 0; u < IPL; ++u) {
                    T[u] = latency(p[u], a[u], rP[u], rD[u], l, lv[u]);
                    tb = umax(tb, bs[u] == bs[u] ? __float_as_uint(T[u]) : 0u);
                }
                const float tmax = __uint_as_float(umax_all(tb));
                // keys of S * Tmax; 0 for a non-candidate
                uint32_t key[IPL], kb = 0;
#pragma unroll
                for (int u = 0; u < IPL; ++u) {
                    const float v = fmaf(bs[u], tmax, wl * (tmax - T[u]));
                    key[u] = bs[u] == bs[u] ? __float_as_uint(v) + 1u : 0u;
                    kb = umax(kb, key[u]);
                }
                const uint32_t kmax = umax_all(kb);
                // lowest instance holding the maximum (slots ascend in index)
                int istar = -1, ustar = 0;
                if (kmax != 0) {
#pragma unroll
                    for (int u = 0; u < IPL; ++u) {
                        uint64_t mk = ballot(key[u] == kmax);
                        if (WIDTH == 16)
                            mk &= 0xffffull;   // the four rows hold the same instances
                        if (istar < 0 && mk != 0) {
                            istar = WAVE * u + (int)__builtin_ctzll(mk);
                            ustar = u;
                        }
                    }
                }
                // capture the pick in lane `slot`: the instance, Tmax and, for
                // the scores, the pick's base score and latency from the lane
                // and slot holding it
                const bool mine = lane == slot;
                cap_i = mine ? istar : cap_i;
                cap_m = mine ? tmax : cap_m;
                if (chosen && istar >= 0) {
                    float vb = bs[0], vt = T[0];
#pragma unroll
                    for (int u = 1; u < IPL; ++u) {
                        vb = ustar == u ? bs[u] : vb;
                        vt = ustar == u ? T[u] : vt;
                    }
                    const int src = istar & (WAVE - 1);
                    vb = __builtin_bit_cast(
                        float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, vb), src));
                    vt = __builtin_bit_cast(
                        float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, vt), src));
                    cap_b = mine ? vb : cap_b;
                    cap_t = mine ? vt : cap_t;
                }
                if (decided) {
                    // the row of Eq. 1 scores this step saw, at the state
                    // before its update (NaN outside the candidate set), with
                    // the division of the dense score kernel
                    const int rq = __builtin_amdgcn_readlane(rblk, slot);
                    float *drow = decided + (size_t)rq * I;
#pragma unroll
                    for (int u = 0; u < IPL; ++u) {
                        const int i = inst(u);
                        if (lane < (WIDTH == 16 ? 16 : WAVE) && i < I)
                            drow[i] = bs[u] == bs[u] ? full_score(bs[u], T[u], tmax, wl)
                                                     : __builtin_nanf("");
                    }
                }
#pragma unroll
                for (int u = 0; u < IPL; ++u) {
                    if (inst(u) == istar) {
                        p[u] += l;
                        a[u] += lv[u];
                    }
                }
#pragma unroll
                for (int u = 0; u < IPL; ++u) {
                    bs[u] = bsn[u];
                    lv[u] = lvn[u];
                }
            }
            // write the block's picks and their Eq. 1 scores in one pass
            if (lane < nb) {
                assign[rblk] = cap_i;
                if (chosen)
                    chosen[rblk] = cap_i >= 0 ? full_score(cap_b, cap_t, cap_m, wl)
                                              : __builtin_nanf("");
            }
        }
        __syncthreads();   // buffer c & 1 may now be refilled; chunk c + 1 is ready
    }
#pragma unroll
    for (int u = 0; u < IPL; ++u) {
        const int i = inst(u);
        if (lane < (WIDTH == 16 ? 16 : WAVE) && i < I && valid[u]) {
            in.p[i] = p[u];
            in.a[i] = a[u];
        }
    }
}

__global__ __launch_bounds__(256) void iota_kernel(int32_t *__restrict__ out, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        out[i] = i;
}

__global__ __launch_bounds__(256) void advance_kernel(const InstArgs in, int I, float dt)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= I)
        return;
    in.p[i] = fmaxf(0.f, in.p[i] - in.P[i] * dt);
    in.a[i] = fmaxf(0.f, in.a[i] - in.D[i] * dt);
}

}  // namespace

hipError_t launch_score(const float *q_hat, const float *l_hat, const int32_t *plen, int B, int M,
                        const InstArgs &in, int I, float wq, float wl, float wc,
                        const AssignOpts &opt, float *S0, hipStream_t s)
{
    hipLaunchKernelGGL(score_kernel, dim3((B + 3) / 4), dim3(256), 0, s, q_hat, l_hat, plen, B, M,
                       in, I, wq, wl, wc, opt, S0);
    return hipGetLastError();
}

hipError_t launch_lpt_order(const float *l_hat, int B, int M, int32_t *order, hipStream_t s)
{
    hipLaunchKernelGGL(lpt_order_kernel, dim3((B + LPT_THREADS - 1) / LPT_THREADS),
                       dim3(LPT_THREADS), 0, s, l_hat, B, M, order);
    return hipGetLastError();
}

hipError_t launch_assign(const float *q_hat, const float *l_hat, const int32_t *plen, int B,
                         int M, const InstArgs &in, int I, float wq, float wl, float wc,
                         const AssignOpts &opt, int32_t *assign, float *chosen, float *decided,
                         hipStream_t s)
{
    const int ipl = (I + WAVE - 1) / WAVE;
#define RB_ASSIGN(N, W)                                                                          \
    hipLaunchKernelGGL((assign_kernel<N, W>), dim3(1), dim3(assign_threads<N>()), 0, s, q_hat,   \
                       l_hat, plen, B, M, in, I, wq, wl, wc, opt, assign, chosen, decided)
    if (I <= 16) RB_ASSIGN(1, 16);
    else if (ipl <= 1) RB_ASSIGN(1, 64);
    else if (ipl <= 2) RB_ASSIGN(2, 64);
    else if (ipl <= 4) RB_ASSIGN(4, 64);
    else if (ipl <= 8) RB_ASSIGN(8, 64);
    else if (ipl <= 16) RB_ASSIGN(16, 64);
    else return hipErrorInvalidValue;
#undef RB_ASSIGN
    return hipGetLastError();
}

hipError_t launch_iota(int32_t *out, int n, hipStream_t s)
{
    hipLaunchKernelGGL(iota_kernel, dim3((n + 255) / 256), dim3(256), 0, s, out, n);
    return hipGetLastError();
}

hipError_t launch_advance(const InstArgs &in, int I, float dt, hipStream_t s)
{
    hipLaunchKernelGGL(advance_kernel, dim3((I + 255) / 256), dim3(256), 0, s, in, I, dt);
    return hipGetLastError();
}

}  // namespace rb
