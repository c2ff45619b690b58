/*
 * CPU oracle for RouteBalance's batched request-to-instance scoring path.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the slow, plain reference that the
 * GPU library is checked against. Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load it. It shares no code, header, table
 * or helper with the GPU library.
 *
 * Paper: "RouteBalance: Fused Model Routing and Load Balancing for
 * Heterogeneous LLM Serving" (arXiv 2606.17949).
 *
 * Arithmetic is fp64 throughout. bf16 inputs are widened exactly
 * (bits << 16 -> fp32 -> fp64). Each function names the passage it follows.
 *
 * Readings of the paper used here (the paper is silent or loose on these):
 *   - distance: squared Euclidean distance on the stored values (Sec. 4.2
 *     says only "distance-weighted KNN");
 *   - top-k order: distance ascending, ties to the lower bank index;
 *   - averaging: uniform mean over the k neighbours by default; the
 *     distance-weighted option uses w_j = 1/(sqrt(max(d_j, 0)) + 1e-6) on the
 *     squared distance d_j, normalised to sum 1 (the paper names a
 *     distance-weighted KNN without giving the weights);
 *   - latency: T = (p_i + l_r)/P_i + (a_i + L_{r,m(i)})/D_i, the instance's
 *     queued prefill plus this prompt drained at its prefill rate, then its
 *     active decode plus this request's predicted output drained at its
 *     decode rate (the state-and-rate form of the estimate in Sec. 4.2);
 *   - normalisation: per request, by the maximum over the candidate set
 *     (Eq. 1; Sec. 4.1 scales by the candidates' maxima); without a budget or
 *     an availability mask every instance is a candidate; a zero maximum makes
 *     that ratio 0;
 *   - candidate set (Alg. 1 budget filter, Eq. 2): an instance is a candidate
 *     when it is available and its expected cost l_r*c_in + L*c_out, taken
 *     in fp64 like every other value here, is at most the request's budget
 *     b_r; a request with no candidate is left unassigned (-1) and changes no
 *     state;
 *   - argmax ties go to the lowest instance index;
 *   - processing order: arrival order (batch index order) by default; the LPT
 *     option (Alg. 1, Sec. 4.1) sorts by max over models of L[r][m], longest
 *     first, equal keys in arrival order;
 *   - update after a pick (Sec. 4.2, "Dead reckoning"): p_i* += l_r and
 *     a_i* += L_{r,m(i*)};
 *   - carry between batches: p <- max(0, p - P*dt), a <- max(0, a - D*dt).
 *
 * Parity pins: KNN and predict are pinned by brute force and hand examples;
 * score and assign by a hand-computed 2x3 example and simplex-corner,
 * conservation and scale invariants; the LPT order, the weighted average and
 * the candidate set by hand examples, closed forms and a library sort; carry
 * by its closed form. The paper
 * prints no worked example of its own, so nothing is pinned to a printed
 * paper value.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_F32 = 0, ORC_BF16 = 1 };

/* Exact widening of one stored element to double. */
static double load_elem(const void *base, int dtype, size_t i)
{
    if (dtype == ORC_F32)
        return (double)((const float *)base)[i];
    uint32_t bits = (uint32_t)((const uint16_t *)base)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/* (d1, i1) < (d2, i2) in the order: distance ascending, then index ascending. */
static int pair_less(double d1, int32_t i1, double d2, int32_t i2)
{
    return d1 < d2 || (d1 == d2 && i1 < i2);
}

/* ------------------------------------------------------------------------ */
/* Exact k-nearest neighbours (Sec. 4.2, the KNN lookup of Alg. 1).         */
/* ------------------------------------------------------------------------ */

typedef struct {
    const void *q, *bank;
    int dtype, B, N, d, k;
    int32_t *idx;
    double *dist;
    int b0, b1;
} knn_job;

/* For one request: scan every bank row, keep the k smallest (dist, idx)
 * pairs in an ascending array by insertion. */
static void knn_one(const knn_job *J, int b)
{
    int32_t *bi = J->idx + (size_t)b * J->k;
    double *bd = J->dist + (size_t)b * J->k;
    int filled = 0;
    for (int n = 0; n < J->N; ++n) {
        double s = 0.0;
        for (int t = 0; t < J->d; ++t) {
            double diff = load_elem(J->q, J->dtype, (size_t)b * J->d + t) -
                          load_elem(J->bank, J->dtype, (size_t)n * J->d + t);
            s += diff * diff;
        }
        if (filled == J->k && !pair_less(s, n, bd[J->k - 1], bi[J->k - 1]))
            continue;
        int pos = filled < J->k ? filled : J->k - 1;
        while (pos > 0 && pair_less(s, n, bd[pos - 1], bi[pos - 1])) {
            bd[pos] = bd[pos - 1];
            bi[pos] = bi[pos - 1];
            --pos;
        }
        bd[pos] = s;
        bi[pos] = n;
        if (filled < J->k)
            ++filled;
    }
}

static void *knn_worker(void *arg)
{
    const knn_job *J = (const knn_job *)arg;
    for (int b = J->b0; b < J->b1; ++b)
        knn_one(J, b);
    return NULL;
}

/* queries [B][d], bank [N][d] (dtype 0 = fp32, 1 = bf16 bits), 1 <= k <= N.
 * Writes idx [B][k] and dist [B][k] sorted ascending. Returns 0, or -1 on bad
 * arguments. Threads split the requests. */
int oracle_knn(const void *queries, const void *bank, int dtype, int B, int N, int d, int k,
               int32_t *idx, double *dist, int nthreads)
{
    if (!queries || !bank || !idx || !dist || B < 0 || N < 1 || d < 1 || k < 1 || k > N)
        return -1;
    if (dtype != ORC_F32 && dtype != ORC_BF16)
        return -1;
    if (B == 0)
        return 0;
    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > B)
        nthreads = B;
    knn_job *jobs = (knn_job *)calloc((size_t)nthreads, sizeof(knn_job));
    pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    for (int t = 0; t < nthreads; ++t) {
        knn_job J = {queries, bank, dtype, B, N, d, k, idx, dist,
                     (int)((long)B * t / nthreads), (int)((long)B * (t + 1) / nthreads)};
        jobs[t] = J;
    }
    for (int t = 1; t < nthreads; ++t)
        pthread_create(&th[t], NULL, knn_worker, &jobs[t]);
    knn_worker(&jobs[0]);
    for (int t = 1; t < nthreads; ++t)
        pthread_join(th[t], NULL);
    free(jobs);
    free(th);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* KNN-averaged predictions (Sec. 4.2: each neighbour stores per-model       */
/* quality and output length, one lookup predicts for every model).        */
/* ------------------------------------------------------------------------ */

/* Weight of a neighbour at squared distance d under the distance-weighted
 * option: the inverse of its Euclidean distance, kept finite at distance 0. */
static double inv_dist_weight(double d)
{
    return 1.0 / (sqrt(fmax(d, 0.0)) + 1e-6);
}

/* nbr [B][k] bank indices; dist [B][k] their squared distances (read only by
 * the weighted option); qual, len [N][M] fp32. q_hat, l_hat [B][M] are the
 * weighted mean over the k neighbours of each model's label, the weights being
 * 1 (weighting 0, the plain mean) or inv_dist_weight (weighting 1), divided by
 * their sum. */
int oracle_predict_ex(const int32_t *nbr, const double *dist, int B, int k, const float *qual,
                      const float *len, int N, int M, int weighting, double *q_hat,
                      double *l_hat)
{
    if (!nbr || !qual || !len || !q_hat || !l_hat || k < 1 || M < 1)
        return -1;
    if (weighting != 0 && (weighting != 1 || !dist))
        return -1;
    for (int b = 0; b < B; ++b) {
        for (int m = 0; m < M; ++m) {
            double sq = 0.0, sl = 0.0, sw = 0.0;
            for (int j = 0; j < k; ++j) {
                int32_t n = nbr[(size_t)b * k + j];
                if (n < 0 || n >= N)
                    return -1;
                double wj = weighting ? inv_dist_weight(dist[(size_t)b * k + j]) : 1.0;
                sq += wj * (double)qual[(size_t)n * M + m];
                sl += wj * (double)len[(size_t)n * M + m];
                sw += wj;
            }
            q_hat[(size_t)b * M + m] = sq / sw;
            l_hat[(size_t)b * M + m] = sl / sw;
        }
    }
    return 0;
}

/* The plain mean (weighting 0). */
int oracle_predict(const int32_t *nbr, int B, int k, const float *qual, const float *len, int N,
                   int M, double *q_hat, double *l_hat)
{
    return oracle_predict_ex(nbr, NULL, B, k, qual, len, N, M, 0, q_hat, l_hat);
}

/* ------------------------------------------------------------------------ */
/* Score of one request against every instance (Eq. 1, cost of Eq. 2).     */
/* ------------------------------------------------------------------------ */

/* Instance state (all length I). */
typedef struct {
    const int32_t *model;
    const double *P, *D, *cin, *cout;
} orc_inst;

/* Candidate set of one request (Alg. 1 budget filter; Eq. 2): instance i is
 * a candidate when mask is NULL or mask[i] != 0, and budget_r is NULL or the
 * expected cost of Eq. 2, input tokens at the input price plus predicted
 * output tokens at the output price, is at most the budget. The cost is the
 * same fp64 value the score uses (for fp32 inputs the two products are exact
 * and the sum is rounded once), compared with the budget widened exactly.
 * A NaN budget admits nothing. Writes cand[I] (0/1). */
static void candidates(const double *l_hat_r, double plen, const orc_inst *in, int I,
                       const float *budget_r, const uint8_t *mask, unsigned char *cand)
{
    for (int i = 0; i < I; ++i) {
        int ok = mask ? mask[i] != 0 : 1;
        if (ok && budget_r) {
            double c = plen * in->cin[i] + l_hat_r[in->model[i]] * in->cout[i];
            ok = c <= (double)*budget_r;
        }
        cand[i] = (unsigned char)ok;
    }
}

/* q_hat_r, l_hat_r: this request's [M] predictions; plen: its prompt tokens.
 * p, a: current queued prefill and active decode per instance.
 * w = (w_qual, w_lat, w_cost) in the order of Alg. 1.
 * cand [I] (NULL = every instance): the candidate set; the cost and latency
 * maxima run over it and non-candidates get S = NaN.
 * Writes S[I], T[I] (latency) and C[I] (cost); returns the number of
 * candidates. */
static int score_row(const double *q_hat_r, const double *l_hat_r, double plen,
                     const orc_inst *in, const double *p, const double *a, int I,
                     const double w[3], const unsigned char *cand, double *S, double *T,
                     double *C)
{
    double tmax = 0.0, cmax = 0.0;
    int seen = 0;
    for (int i = 0; i < I; ++i) {
        int m = in->model[i];
        /* Eq. 2: input tokens at the input price plus predicted output tokens
         * at the output price. */
        C[i] = plen * in->cin[i] + l_hat_r[m] * in->cout[i];
        /* Latency: queued prefill plus own prompt at the prefill rate, then
         * active decode plus own predicted output at the decode rate. */
        T[i] = (p[i] + plen) / in->P[i] + (a[i] + l_hat_r[m]) / in->D[i];
        if (cand && !cand[i])
            continue;
        if (!seen || C[i] > cmax)
            cmax = C[i];
        if (!seen || T[i] > tmax)
            tmax = T[i];
        seen = 1;
    }
    for (int i = 0; i < I; ++i) {
        int m = in->model[i];
        if (cand && !cand[i]) {
            S[i] = NAN;
            continue;
        }
        double cost_ratio = cmax > 0.0 ? C[i] / cmax : 0.0;
        double lat_ratio = tmax > 0.0 ? T[i] / tmax : 0.0;
        S[i] = w[0] * q_hat_r[m] + w[2] * (1.0 - cost_ratio) + w[1] * (1.0 - lat_ratio);
    }
    return seen;
}

/* One row of scores at a given state, exported for step-by-step replay.
 * budget_r (one value) and mask [I] may be NULL; cand [I] receives the
 * candidate set (0/1). */
int oracle_score_row_ex(const double *q_hat_r, const double *l_hat_r, int M, double plen,
                        const int32_t *model, const double *p, const double *a, const double *P,
                        const double *D, const double *cin, const double *cout, int I,
                        double w_qual, double w_lat, double w_cost, const float *budget_r,
                        const uint8_t *mask, double *S, double *T, double *C,
                        unsigned char *cand)
{
    if (!q_hat_r || !l_hat_r || !model || !p || !a || !P || !D || !cin || !cout || !S || !T || !C ||
        !cand || I < 1 || M < 1)
        return -1;
    for (int i = 0; i < I; ++i)
        if (model[i] < 0 || model[i] >= M)
            return -1;
    orc_inst in = {model, P, D, cin, cout};
    double w[3] = {w_qual, w_lat, w_cost};
    candidates(l_hat_r, plen, &in, I, budget_r, mask, cand);
    score_row(q_hat_r, l_hat_r, plen, &in, p, a, I, w, cand, S, T, C);
    return 0;
}

int oracle_score_row(const double *q_hat_r, const double *l_hat_r, int M, double plen,
                     const int32_t *model, const double *p, const double *a, const double *P,
                     const double *D, const double *cin, const double *cout, int I, double w_qual,
                     double w_lat, double w_cost, double *S, double *T, double *C)
{
    if (I < 1)
        return -1;
    unsigned char *cand = (unsigned char *)malloc((size_t)I);
    int rc = oracle_score_row_ex(q_hat_r, l_hat_r, M, plen, model, p, a, P, D, cin, cout, I,
                                 w_qual, w_lat, w_cost, NULL, NULL, S, T, C, cand);
    free(cand);
    return rc;
}

/* Dense score matrix S0 [B][I] at the batch-start state. */
int oracle_score(const double *q_hat, const double *l_hat, const int32_t *plen, int B, int M,
                 const int32_t *model, const double *p, const double *a, const double *P,
                 const double *D, const double *cin, const double *cout, int I, double w_qual,
                 double w_lat, double w_cost, double *S0)
{
    if (B < 0 || I < 1 || M < 1 || !S0)
        return -1;
    double *T = (double *)malloc(sizeof(double) * (size_t)I);
    double *C = (double *)malloc(sizeof(double) * (size_t)I);
    int rc = 0;
    for (int r = 0; r < B && rc == 0; ++r)
        rc = oracle_score_row(q_hat + (size_t)r * M, l_hat + (size_t)r * M, M, (double)plen[r],
                              model, p, a, P, D, cin, cout, I, w_qual, w_lat, w_cost,
                              S0 + (size_t)r * I, T, C);
    free(T);
    free(C);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Greedy online assignment (Alg. 1 loop; Sec. 4.1; dead reckoning, 4.2).   */
/* ------------------------------------------------------------------------ */

/* LPT processing order (Alg. 1 sorts the batch by predicted length, longest
 * first; Sec. 4.1 takes the key max over models of L[r][m] because the model
 * is not chosen yet). Equal keys keep arrival order. */
typedef struct {
    double key;
    int32_t r;
} lpt_item;

static int lpt_before(const void *x, const void *y)
{
    const lpt_item *u = (const lpt_item *)x, *v = (const lpt_item *)y;
    if (u->key != v->key)
        return u->key > v->key ? -1 : 1;
    return u->r < v->r ? -1 : (u->r > v->r);
}

/* l_hat [B][M]; order [B] receives the request index decided at each step. */
int oracle_lpt_order(const double *l_hat, int B, int M, int32_t *order)
{
    if (!l_hat || !order || B < 0 || M < 1)
        return -1;
    lpt_item *it = (lpt_item *)malloc(sizeof(lpt_item) * (size_t)(B > 0 ? B : 1));
    for (int r = 0; r < B; ++r) {
        double key = l_hat[(size_t)r * M];
        for (int m = 1; m < M; ++m)
            key = fmax(key, l_hat[(size_t)r * M + m]);
        it[r].key = key;
        it[r].r = r;
    }
    qsort(it, (size_t)B, sizeof(lpt_item), lpt_before);
    for (int t = 0; t < B; ++t)
        order[t] = it[t].r;
    free(it);
    return 0;
}

/* For each step t, request r = order[t] (arrival order: r = t; lpt != 0: the
 * LPT order): form its candidate set, score it against the current state,
 * pick the highest score among the candidates (lowest index among equals),
 * record it, then grow the chosen instance's queued prefill by the prompt and
 * its active decode by the request's predicted output on that instance's
 * model. A request without candidates gets -1 (chosen NaN) and changes no
 * state.
 * p, a [I] are updated in place. budget [B] and mask [I] may be NULL.
 * assign [B] and chosen [B] (nullable) are indexed by request; order [B]
 * (nullable) receives the processing order; trace_p, trace_a [(B+1)][I]
 * (nullable) hold the state before each step and after the last. */
int oracle_assign_ex(const double *q_hat, const double *l_hat, const int32_t *plen, int B, int M,
                     const int32_t *model, double *p, double *a, const double *P, const double *D,
                     const double *cin, const double *cout, int I, double w_qual, double w_lat,
                     double w_cost, int lpt, const float *budget, const uint8_t *mask,
                     int32_t *assign, double *chosen, int32_t *order, double *trace_p,
                     double *trace_a)
{
    if (!q_hat || !l_hat || !plen || !model || !p || !a || !P || !D || !cin || !cout || !assign ||
        B < 0 || I < 1 || M < 1)
        return -1;
    for (int i = 0; i < I; ++i)
        if (model[i] < 0 || model[i] >= M)
            return -1;
    orc_inst in = {model, P, D, cin, cout};
    double w[3] = {w_qual, w_lat, w_cost};
    double *S = (double *)malloc(sizeof(double) * (size_t)I);
    double *T = (double *)malloc(sizeof(double) * (size_t)I);
    double *C = (double *)malloc(sizeof(double) * (size_t)I);
    unsigned char *cand = (unsigned char *)malloc((size_t)I);
    int32_t *ord = (int32_t *)malloc(sizeof(int32_t) * (size_t)(B > 0 ? B : 1));
    if (lpt)
        oracle_lpt_order(l_hat, B, M, ord);
    else
        for (int t = 0; t < B; ++t)
            ord[t] = t;
    for (int t = 0; t < B; ++t) {
        const int r = ord[t];
        if (trace_p)
            memcpy(trace_p + (size_t)t * I, p, sizeof(double) * (size_t)I);
        if (trace_a)
            memcpy(trace_a + (size_t)t * I, a, sizeof(double) * (size_t)I);
        const double *qr = q_hat + (size_t)r * M, *lr = l_hat + (size_t)r * M;
        candidates(lr, (double)plen[r], &in, I, budget ? budget + r : NULL, mask, cand);
        score_row(qr, lr, (double)plen[r], &in, p, a, I, w, cand, S, T, C);
        int best = -1;
        for (int i = 0; i < I; ++i)
            if (cand[i] && (best < 0 || S[i] > S[best]))
                best = i;
        assign[r] = best;
        if (chosen)
            chosen[r] = best < 0 ? NAN : S[best];
        if (best < 0)
            continue;
        p[best] += (double)plen[r];
        a[best] += lr[model[best]];
    }
    if (order)
        memcpy(order, ord, sizeof(int32_t) * (size_t)B);
    if (trace_p)
        memcpy(trace_p + (size_t)B * I, p, sizeof(double) * (size_t)I);
    if (trace_a)
        memcpy(trace_a + (size_t)B * I, a, sizeof(double) * (size_t)I);
    free(S);
    free(T);
    free(C);
    free(cand);
    free(ord);
    return 0;
}

/* Arrival order, every instance a candidate. */
int oracle_assign(const double *q_hat, const double *l_hat, const int32_t *plen, int B, int M,
                  const int32_t *model, double *p, double *a, const double *P, const double *D,
                  const double *cin, const double *cout, int I, double w_qual, double w_lat,
                  double w_cost, int32_t *assign, double *chosen, double *trace_p, double *trace_a)
{
    return oracle_assign_ex(q_hat, l_hat, plen, B, M, model, p, a, P, D, cin, cout, I, w_qual,
                            w_lat, w_cost, 0, NULL, NULL, assign, chosen, NULL, trace_p, trace_a);
}

/* ------------------------------------------------------------------------ */
/* Carry the dead-reckoned state across a gap of dt seconds between batches. */
/* ------------------------------------------------------------------------ */

/* Both queues drain linearly at their rates and stop at zero. */
int oracle_advance(double *p, double *a, const double *P, const double *D, int I, double dt)
{
    if (!p || !a || !P || !D || I < 1 || !(dt >= 0.0))
        return -1;
    for (int i = 0; i < I; ++i) {
        p[i] = fmax(0.0, p[i] - P[i] * dt);
        a[i] = fmax(0.0, a[i] - D[i] * dt);
    }
    return 0;
}
