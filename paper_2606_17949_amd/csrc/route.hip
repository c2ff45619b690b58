// Request-instance scoring and the greedy online assignment (RouteBalance
// Eq. 1 score, Eq. 2 cost, the dead-reckoned latency of Sec. 4.2, and the
// greedy per-batch loop of Alg. 1), for gfx950.
#include "common.hpp"
#include "kernels.hpp"

namespace rb {

namespace {

// Latency of a request with prompt l and predicted output lv on an instance
// with queued prefill p, active decode a and rates P, D: the queued prefill
// plus this prompt drains at P, then the active decode plus this output at D.
__device__ __forceinline__ float latency(float p, float a, float P, float D, float l, float lv)
{
    return (p + l) / P + (a + lv) / D;
}

// Eq. 2 expected cost: input tokens at the input price plus predicted output
// tokens at the output price.
__device__ __forceinline__ float cost(float l, float lv, float cin, float cout)
{
    return l * cin + lv * cout;
}

// Eq. 1 with per-request maxima; a zero maximum makes its ratio 0.
__device__ __forceinline__ float score_of(float qv, float C, float Cmax, float T, float Tmax,
                                          float wq, float wl, float wc)
{
    const float rc = Cmax > 0.f ? C / Cmax : 0.f;
    const float rt = Tmax > 0.f ? T / Tmax : 0.f;
    return wq * qv + wc * (1.f - rc) + wl * (1.f - rt);
}

// One wave per request row of the dense score matrix.
__global__ __launch_bounds__(256) void score_kernel(const float *__restrict__ q_hat,
                                                    const float *__restrict__ l_hat,
                                                    const int32_t *__restrict__ plen, int B, int M,
                                                    const InstArgs in, int I, float wq, float wl,
                                                    float wc, float *__restrict__ S0)
{
    const int lane = lane_id();
    const int r = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    if (r >= B)
        return;
    const float l = (float)plen[r];
    const float *qr = q_hat + (size_t)r * M;
    const float *lr = l_hat + (size_t)r * M;
    float cmax = -INFINITY, tmax = -INFINITY;
    for (int i = lane; i < I; i += WAVE) {
        const int m = in.model[i];
        const float lv = (unsigned)m < (unsigned)M ? lr[m] : __builtin_nanf("");
        cmax = fmaxf(cmax, cost(l, lv, in.cin[i], in.cout[i]));
        tmax = fmaxf(tmax, latency(in.p[i], in.a[i], in.P[i], in.D[i], l, lv));
    }
    cmax = wave_max(cmax);
    tmax = wave_max(tmax);
    for (int i = lane; i < I; i += WAVE) {
        const int m = in.model[i];
        const bool mv = (unsigned)m < (unsigned)M;
        const float lv = mv ? lr[m] : __builtin_nanf("");
        const float qv = mv ? qr[m] : __builtin_nanf("");
        const float C = cost(l, lv, in.cin[i], in.cout[i]);
        const float T = latency(in.p[i], in.a[i], in.P[i], in.D[i], l, lv);
        S0[(size_t)r * I + i] = score_of(qv, C, cmax, T, tmax, wq, wl, wc);
    }
}

// Greedy assignment on one wavefront. Instance i = lane + 64*u lives in
// register slot u of its lane, with its state; each step is two wave maxima
// (cost and latency), the scores, and an argmax with the lowest index among
// equal scores, then the owner lane updates the chosen instance.
template <int IPL>
__global__ __launch_bounds__(64) void assign_kernel(const float *__restrict__ q_hat,
                                                    const float *__restrict__ l_hat,
                                                    const int32_t *__restrict__ plen, int B, int M,
                                                    const InstArgs in, int I, float wq, float wl,
                                                    float wc, int32_t *__restrict__ assign,
                                                    float *__restrict__ chosen)
{
    const int lane = threadIdx.x;
    int model[IPL];
    float p[IPL], a[IPL], P[IPL], D[IPL], cin[IPL], cout[IPL];
    bool valid[IPL];
#pragma unroll
    for (int u = 0; u < IPL; ++u) {
        const int i = lane + WAVE * u;
        // an instance whose model id is outside [0, M) is never chosen
        const int m = i < I ? in.model[i] : 0;
        valid[u] = i < I && (unsigned)m < (unsigned)M;
        model[u] = valid[u] ? m : 0;
        p[u] = valid[u] ? in.p[i] : 0.f;
        a[u] = valid[u] ? in.a[i] : 0.f;
        P[u] = valid[u] ? in.P[i] : 1.f;
        D[u] = valid[u] ? in.D[i] : 1.f;
        cin[u] = valid[u] ? in.cin[i] : 0.f;
        cout[u] = valid[u] ? in.cout[i] : 0.f;
    }
    for (int r = 0; r < B; ++r) {
        const float l = (float)plen[r];
        const float *qr = q_hat + (size_t)r * M;
        const float *lr = l_hat + (size_t)r * M;
        float qv[IPL], lv[IPL], C[IPL], T[IPL];
        float cm = -INFINITY, tm = -INFINITY;
#pragma unroll
        for (int u = 0; u < IPL; ++u) {
            qv[u] = qr[model[u]];
            lv[u] = lr[model[u]];
            C[u] = cost(l, lv[u], cin[u], cout[u]);
            T[u] = latency(p[u], a[u], P[u], D[u], l, lv[u]);
            if (valid[u]) {
                cm = fmaxf(cm, C[u]);
                tm = fmaxf(tm, T[u]);
            }
        }
        cm = wave_max(cm);
        tm = wave_max(tm);
        float best = -INFINITY;
        int besti = 0x7fffffff;
#pragma unroll
        for (int u = 0; u < IPL; ++u) {
            const float S = score_of(qv[u], C[u], cm, T[u], tm, wq, wl, wc);
            if (valid[u] && S > best) {   // slots ascend in index, so ties keep the lower
                best = S;
                besti = lane + WAVE * u;
            }
        }
        const float bs = wave_max(best);
        // lowest index among lanes holding the maximum (indices < 2^24 are exact in fp32)
        const float bi = -wave_max(best == bs ? -(float)besti : -INFINITY);
        const int istar = (int)bi;
        if (lane == 0) {
            assign[r] = istar;
            if (chosen)
                chosen[r] = bs;
        }
        if ((istar & (WAVE - 1)) == lane) {
            const int us = istar / WAVE;
#pragma unroll
            for (int u = 0; u < IPL; ++u) {
                if (u == us) {
                    p[u] += l;
                    a[u] += lv[u];
                }
            }
        }
    }
#pragma unroll
    for (int u = 0; u < IPL; ++u) {
        const int i = lane + WAVE * u;
        if (i < I) {
            in.p[i] = p[u];
            in.a[i] = a[u];
        }
    }
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
                        const InstArgs &in, int I, float wq, float wl, float wc, float *S0,
                        hipStream_t s)
{
    hipLaunchKernelGGL(score_kernel, dim3((B + 3) / 4), dim3(256), 0, s, q_hat, l_hat, plen, B, M,
                       in, I, wq, wl, wc, S0);
    return hipGetLastError();
}

hipError_t launch_assign(const float *q_hat, const float *l_hat, const int32_t *plen, int B,
                         int M, const InstArgs &in, int I, float wq, float wl, float wc,
                         int32_t *assign, float *chosen, hipStream_t s)
{
    const int ipl = (I + WAVE - 1) / WAVE;
#define RB_ASSIGN(N)                                                                             \
    hipLaunchKernelGGL(assign_kernel<N>, dim3(1), dim3(64), 0, s, q_hat, l_hat, plen, B, M, in, \
                       I, wq, wl, wc, assign, chosen)
    if (ipl <= 1) RB_ASSIGN(1);
    else if (ipl <= 2) RB_ASSIGN(2);
    else if (ipl <= 4) RB_ASSIGN(4);
    else if (ipl <= 8) RB_ASSIGN(8);
    else if (ipl <= 16) RB_ASSIGN(16);
    else return hipErrorInvalidValue;
#undef RB_ASSIGN
    return hipGetLastError();
}

hipError_t launch_advance(const InstArgs &in, int I, float dt, hipStream_t s)
{
    hipLaunchKernelGGL(advance_kernel, dim3((I + 255) / 256), dim3(256), 0, s, in, I, dt);
    return hipGetLastError();
}

}  // namespace rb
