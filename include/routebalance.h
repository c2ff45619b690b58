/*
 * routebalance.h -- C ABI of the MI355X (gfx950) batched request-to-instance
 * scoring path of RouteBalance (arXiv 2606.17949).
 *
 * For a batch of requests the library
 *   1. finds the k nearest reference prompts of each request embedding in a
 *      labelled bank (Sec. 4.2, the KNN lookup of Alg. 1),
 *   2. averages the neighbours' per-model quality and output-length labels into
 *      predictions Q[r][m], L[r][m] (Sec. 4.2),
 *   3. scores every request-instance pair with Eq. 1, using the cost of Eq. 2
 *      and a latency dead-reckoned from instance state (Sec. 4.2), and
 *   4. assigns each request to one instance greedily, updating the chosen
 *      instance's state before the next request is scored (Alg. 1, Sec. 4.1).
 *
 * Conventions shared by every entry point
 *   - Every pointer argument is a DEVICE pointer unless stated otherwise; the
 *     struct arguments themselves (rb_instances, rb_weights) live on the host.
 *   - The caller owns and allocates every buffer, including the workspace. The
 *     library never allocates, frees, copies to the host or synchronises; it
 *     keeps no state between calls beyond a per-device cache of the compute
 *     unit count. Work is enqueued on `stream` (a hipStream_t; NULL = the null
 *     stream) and runs asynchronously.
 *   - Arrays are row-major; "[X][Y]" means Y is contiguous.
 *   - All arguments are validated on the host before anything is enqueued. On
 *     any error nothing is enqueued and no output is touched.
 *   - Faults inside kernels surface at the caller's next synchronisation.
 *   - Values that live in device memory are not checked (documented
 *     preconditions): rates > 0, prices >= 0, prompt lengths >= 1, model ids in
 *     [0, M), queued prefill and active decode >= 0, quality labels in [0, 1],
 *     length labels >= 0, embeddings and norms finite. Violating them is
 *     undefined.
 *   - Results are deterministic: the same inputs give bit-identical outputs on
 *     every call.
 */
#ifndef ROUTEBALANCE_H
#define ROUTEBALANCE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    RB_OK = 0,
    RB_ERR_NULL = -1,        /* a required pointer is NULL */
    RB_ERR_DIMS = -2,        /* a size is out of range (see each call) */
    RB_ERR_DTYPE = -3,       /* dtype is not RB_F32 or RB_BF16 */
    RB_ERR_WEIGHTS = -4,     /* weights not finite, negative, or |sum - 1| > 1e-5 */
    RB_ERR_WORKSPACE = -5,   /* workspace NULL or smaller than rb_workspace_size */
    RB_ERR_UNSUPPORTED = -6, /* an option this version does not implement */
    RB_ERR_HIP = -7,         /* a HIP runtime call or kernel launch failed */
    RB_ERR_ALIGN = -8,       /* a pointer is not aligned as required */
    RB_ERR_SCRATCH = -9      /* rb_route_batch_noalloc: these sizes need more workspace than
                                RB_SCRATCH_BYTES */
} rb_status;

typedef enum { RB_F32 = 0, RB_BF16 = 1 } rb_dtype;

/* Neighbour-averaging rule (Sec. 4.2 calls the paper's KNN "distance-weighted"
 * without giving the weights).
 *   RB_KNN_UNIFORM:   the plain mean over the k neighbours.
 *   RB_KNN_INV_DIST:  weights w_j = 1/(sqrt(max(d_j, 0)) + 1e-6) on the squared
 *                     distances d_j (inverse Euclidean distance, finite at 0),
 *                     normalised to sum 1. */
typedef enum { RB_KNN_UNIFORM = 0, RB_KNN_INV_DIST = 1 } rb_knn_weighting;

/* Order in which the greedy loop decides the batch.
 *   RB_ORDER_ARRIVAL: batch index order r = 0..B-1.
 *   RB_ORDER_LPT:     longest predicted output first (Alg. 1 sorts the batch by
 *                     predicted length, descending; Sec. 4.1 keys request r by
 *                     max over m of L[r][m], the model being unknown yet).
 *                     Equal keys keep arrival order. */
typedef enum { RB_ORDER_ARRIVAL = 0, RB_ORDER_LPT = 1 } rb_order;

#define RB_MAX_K 64      /* largest neighbour count k */
#define RB_MAX_D 2048    /* largest embedding dimension d */
#define RB_MAX_I 1024    /* largest instance count I */
#define RB_MAX_M 1024    /* largest model count M */

/* Scheduling weights on the 3-simplex, in the order of Alg. 1:
 * (w_qual, w_lat, w_cost), each >= 0, summing to 1 within 1e-5. */
typedef struct {
    float w_qual, w_lat, w_cost;
} rb_weights;

/* Instance table (Tab. notation: instances I, model m(i)), a host struct of
 * device pointers, each array of length I:
 *   model        int32, m(i) in [0, M)
 *   prefill_q    fp32, queued prefill tokens p_i          (IN/OUT, dead reckoning)
 *   decode_q     fp32, active decode tokens a_i           (IN/OUT, dead reckoning)
 *   prefill_rate fp32, prefill tokens/s P_i > 0
 *   decode_rate  fp32, decode tokens/s D_i > 0
 *   price_in     fp32, price per input token  (c_in of Eq. 2)  >= 0
 *   price_out    fp32, price per output token (c_out of Eq. 2) >= 0
 * Latency of request r on instance i (the state-and-rate form of the estimate
 * in Sec. 4.2): T = (p_i + l_r)/P_i + (a_i + L[r][m(i)])/D_i.
 * Cost (Eq. 2): C = l_r*price_in[i] + L[r][m(i)]*price_out[i]. */
typedef struct {
    const int32_t *model;
    float *prefill_q;
    float *decode_q;
    const float *prefill_rate;
    const float *decode_rate;
    const float *price_in;
    const float *price_out;
} rb_instances;

/* Human-readable name of a status code (static storage, never NULL). */
const char *rb_status_string(rb_status s);

/* Bytes of device workspace that rb_knn_topk, rb_knn_predict, rb_route_batch and
 * rb_route_batch_ex need for these sizes on the current device (with or without
 * RB_FLAG_OVERLAP), written to *bytes (a host pointer). The value
 * depends on the device's compute-unit count; query it on the device that will
 * run the call. Errors: RB_ERR_NULL (bytes), RB_ERR_DIMS / RB_ERR_DTYPE as for
 * rb_knn_topk, RB_ERR_HIP if the device cannot be queried. */
rb_status rb_workspace_size(int B, int N, int d, rb_dtype dtype, int k, int M, size_t *bytes);

/* Squared L2 norms of the bank rows, norms[n] = sum_t bank[n][t]^2 in fp32
 * (a fixed summation order, so the result is reproducible).
 * The reference bank is static, so this is computed once when the bank is
 * loaded and passed to every rb_knn_topk / rb_route_batch call.
 *   bank  [N][d] of dtype (16-byte aligned); norms [N] fp32 (output).
 * Errors: RB_ERR_NULL, RB_ERR_DTYPE, RB_ERR_DIMS (N < 1, d < 1, d > RB_MAX_D,
 * d % 8 for bf16 or d % 4 for fp32 not 0), RB_ERR_ALIGN, RB_ERR_HIP. */
rb_status rb_bank_norms(const void *bank, rb_dtype dtype, int N, int d, float *norms,
                        void *stream);

/* Exact k-nearest-neighbour search (Sec. 4.2: each request embedding is looked
 * up against the labelled reference bank with k = 10 in the paper).
 * Distance: squared Euclidean, computed as |q|^2 + |x|^2 - 2<q, x> with fp32
 * products and accumulation (bf16 x bf16 products are exact in fp32). Order:
 * distance ascending, equal distances by the lower bank index.
 *   queries    [B][d] of dtype. For a bf16 bank the caller rounds the queries
 *              to bf16 (round to nearest even) before the call.
 *   bank       [N][d] of dtype; bank_norms [N] fp32 from rb_bank_norms.
 *   nbr_idx    [B][k] int32 (output): bank row indices, nearest first.
 *   nbr_dist   [B][k] fp32  (output): their squared distances; may be NULL.
 *   ws         device workspace of ws_bytes >= rb_workspace_size(...), 256-byte
 *              aligned; its contents on entry do not matter.
 * B = 0 enqueues nothing and returns RB_OK.
 * Errors: RB_ERR_NULL; RB_ERR_DTYPE; RB_ERR_DIMS (B < 0, N < 1, k < 1,
 * k > min(N, RB_MAX_K), d < 1, d > RB_MAX_D, d % 8 for bf16 or d % 4 for fp32
 * not 0); RB_ERR_ALIGN (queries, bank not 16-byte aligned, ws not 256-byte
 * aligned); RB_ERR_WORKSPACE; RB_ERR_HIP. */
rb_status rb_knn_topk(const void *queries, const void *bank, const float *bank_norms,
                      rb_dtype dtype, int B, int N, int d, int k, int32_t *nbr_idx,
                      float *nbr_dist, void *ws, size_t ws_bytes, void *stream);

/* KNN-averaged predictions (Sec. 4.2: each neighbour stores a quality label and
 * an output length for every model, so one lookup predicts both for every
 * candidate model). With RB_KNN_UNIFORM:
 *   q_hat[b][m] = (1/k) * sum_j bank_qual[nbr_idx[b][j]][m]
 *   l_hat[b][m] = (1/k) * sum_j bank_len [nbr_idx[b][j]][m]
 * summed in fp32 in neighbour order j = 0..k-1. With RB_KNN_INV_DIST, each
 * neighbour's labels are weighted by w_j = 1/(sqrt(max(nbr_dist[b][j], 0)) +
 * 1e-6) and the sums divided by sum_j w_j (fp32, same order).
 *   nbr_idx [B][k] int32 in [0, N); nbr_dist [B][k] fp32 squared distances as
 *   rb_knn_topk writes them, unused by the uniform rule and may then be NULL;
 *   bank_qual, bank_len [N][M] fp32; q_hat, l_hat [B][M] fp32 (outputs).
 * Errors: RB_ERR_NULL (also nbr_dist NULL with RB_KNN_INV_DIST), RB_ERR_DIMS
 * (B < 0, k < 1, k > RB_MAX_K, N < 1, M < 1, M > RB_MAX_M), RB_ERR_UNSUPPORTED
 * (weighting out of range), RB_ERR_HIP. */
rb_status rb_predict(const int32_t *nbr_idx, const float *nbr_dist, int B, int k,
                     rb_knn_weighting weighting, const float *bank_qual, const float *bank_len,
                     int N, int M, float *q_hat, float *l_hat, void *stream);

/* Dense score matrix at the instances' current state (Eq. 1 for every pair):
 *   S0[r][i] = w_qual*Q[r][m(i)] + w_cost*(1 - C[r][i]/max_j C[r][j])
 *            + w_lat *(1 - T[r][i]/max_j T[r][j])
 * with C and T as in rb_instances; a zero maximum makes its ratio 0. The state
 * is read, not modified. fp32 arithmetic.
 *   q_hat, l_hat [B][M] fp32; prompt_len [B] int32 (input tokens l_r >= 1);
 *   inst: host struct of device arrays of length I; score0 [B][I] fp32 (output).
 * Errors: RB_ERR_NULL, RB_ERR_DIMS (B < 0, M < 1, M > RB_MAX_M, I < 1,
 * I > RB_MAX_I), RB_ERR_WEIGHTS, RB_ERR_HIP. */
rb_status rb_score(const float *q_hat, const float *l_hat, const int32_t *prompt_len, int B,
                   int M, const rb_instances *inst, int I, rb_weights w, float *score0,
                   void *stream);

/* Greedy online assignment in arrival order (Alg. 1 loop; Sec. 4.1; the
 * dead-reckoning update of Sec. 4.2). For r = 0..B-1: score request r against
 * every instance at the CURRENT state (as rb_score does for one row), pick
 * i* = argmax (the lowest index among exactly equal scores), then
 *   prefill_q[i*] += l_r;  decode_q[i*] += L[r][m(i*)].
 * Rates and prices are unchanged. Runs on one wavefront, fp32.
 *   assign [B] int32 (output); chosen_score [B] fp32 (output, may be NULL);
 *   decided [B][I] fp32 (output, may be NULL): row r holds the Eq. 1 scores
 *   of request r against every instance at the state it was decided in (the
 *   logged score matrices Sec. 4.1 compares the greedy pass with), NaN for
 *   an instance outside its candidate set; chosen_score[r] equals
 *   decided[r][assign[r]] bit for bit. Writing it slows the loop.
 *   inst->prefill_q / decode_q are updated in place.
 * Errors: as rb_score, plus RB_ERR_NULL for assign. */
rb_status rb_assign(const float *q_hat, const float *l_hat, const int32_t *prompt_len, int B,
                    int M, const rb_instances *inst, int I, rb_weights w, int32_t *assign,
                    float *chosen_score, float *decided, void *stream);

/* Flags of rb_options.
 *   RB_FLAG_OVERLAP: the bank scan of rb_knn_predict / rb_route_batch_ex
 *     leaves a compute unit free on each XCD so that a greedy pass
 *     (rb_assign_ex) of another batch, enqueued on another stream, runs beside
 *     it instead of waiting for the scan to drain. The scan's rows are spread
 *     over the remaining units (3 % fewer on MI355X for a batch of up to 256
 *     requests, more for larger batches, whose query tiles share an XCD; a
 *     bank whose rows per unit would pass 2 GB is split further and may
 *     leave none free). Results do not change. */
#define RB_FLAG_OVERLAP 1u
/*   RB_FLAG_LISTS_ONLY, RB_FLAG_FROM_LISTS (rb_knn_predict only, not both):
 *     the lookup in two calls, so that its two halves can go on different
 *     streams. With RB_FLAG_LISTS_ONLY the call runs the seed and the bank
 *     scan and leaves the per-chunk candidate lists in the workspace; it
 *     writes none of nbr_idx, nbr_dist, q_hat, l_hat (q_hat and l_hat may
 *     then be NULL). With RB_FLAG_FROM_LISTS it runs only the merge of those
 *     lists and the label average, from the lists that the last
 *     RB_FLAG_LISTS_ONLY call on this workspace left there; that call must
 *     have had the same dtype, B, N, d, k and RB_FLAG_OVERLAP bit, on the same
 *     device, and have completed (same stream, or ordered before this call by
 *     an event). The queries and the bank are then not read. The two calls
 *     give the same outputs as one call without either flag. */
#define RB_FLAG_LISTS_ONLY 2u
#define RB_FLAG_FROM_LISTS 4u

/* Options of rb_assign_ex, rb_knn_predict and rb_route_batch_ex (a host
 * struct; the pointers are device pointers). A zero-initialised struct (or a
 * NULL options pointer) gives the defaults, under which the _ex calls behave
 * as the plain ones.
 *   order          processing order of the greedy loop (rb_order).
 *   weighting      neighbour averaging (rb_knn_weighting); read by
 *                  rb_route_batch_ex only.
 *   budget         [B] fp32 or NULL: per-request cost budget b_r (Alg. 1 budget
 *                  filter). Instance i is admitted for request r when its Eq. 2
 *                  cost fma(l_r, price_in[i], L[r][m(i)]*price_out[i]), in fp32,
 *                  is <= b_r. +INFINITY means no budget; NaN admits nothing.
 *   instance_mask  [I] uint8 or NULL: 0 = instance unavailable for this batch
 *                  (e.g. a lost model tier); NULL = all available.
 *   order_out      [B] int32 or NULL: receives the processing order,
 *                  order_out[t] = request decided at step t. Required by
 *                  rb_assign_ex when order is RB_ORDER_LPT (it also serves as
 *                  that call's scratch); optional for rb_route_batch_ex.
 *   flags          RB_FLAG_* bits (the two split flags for rb_knn_predict
 *                  only); other bits must be 0.
 * The candidate set of a request is the available, admitted instances; Eq. 1's
 * cost and latency maxima run over it (Sec. 4.1: normalised by the candidates'
 * maxima) and the argmax is taken within it. A request with an empty candidate
 * set is left unassigned: assign = -1, chosen_score = NaN, no state change. */
typedef struct {
    rb_order order;
    rb_knn_weighting weighting;
    const float *budget;
    const uint8_t *instance_mask;
    int32_t *order_out;
    uint32_t flags;
} rb_options;

/* rb_assign with options (Alg. 1 with its LPT order and budget filter, and an
 * instance availability mask). assign [B], chosen_score [B] and the rows of
 * decided [B][I] (may be NULL) stay indexed by request whatever the order.
 * Errors: as rb_assign, plus RB_ERR_UNSUPPORTED (order or weighting out of
 * range), RB_ERR_NULL (order_out missing for RB_ORDER_LPT). */
rb_status rb_assign_ex(const float *q_hat, const float *l_hat, const int32_t *prompt_len, int B,
                       int M, const rb_instances *inst, int I, rb_weights w,
                       const rb_options *opts, int32_t *assign, float *chosen_score,
                       float *decided, void *stream);

/* The whole path for one batch (Alg. 1: one batched KNN lookup, the
 * predictions of Sec. 4.2, then the greedy loop): rb_knn_topk, then
 * rb_predict (uniform), then rb_assign, enqueued back to back on `stream`.
 * The intermediate outputs nbr_idx [B][k], nbr_dist [B][k], q_hat [B][M],
 * l_hat [B][M] and chosen_score [B] are written when their pointers are
 * non-NULL and otherwise kept in the workspace. score0 [B][I] (may be NULL)
 * receives the dense Eq. 1 matrix at the batch-start state, as rb_score
 * computes it, before the greedy loop changes the state. inst state is
 * updated in place as by rb_assign.
 * Errors: the union of those of the three calls. */
rb_status rb_route_batch(const void *queries, const void *bank, const float *bank_norms,
                         rb_dtype dtype, int B, int N, int d, int k, const float *bank_qual,
                         const float *bank_len, int M, const int32_t *prompt_len,
                         const rb_instances *inst, int I, rb_weights w, int32_t *assign,
                         float *chosen_score, int32_t *nbr_idx, float *nbr_dist, float *q_hat,
                         float *l_hat, float *score0, void *ws, size_t ws_bytes, void *stream);

/* The estimation half of the path for one batch (Alg. 1's one batched KNN
 * lookup): rb_knn_topk, then the label average of opts->weighting, in one
 * call. Nothing here reads the instance state, so the lookup of the next
 * batch can run on one stream while rb_assign_ex decides the current batch on
 * another (with RB_FLAG_OVERLAP the scan leaves room for it).
 *   q_hat, l_hat [B][M] fp32 (outputs, required but with RB_FLAG_LISTS_ONLY);
 *   nbr_idx, nbr_dist [B][k] (outputs, may be NULL: then kept in the
 *   workspace); opts may be NULL; its order, budget, instance_mask and
 *   order_out are not read; its flags may also hold RB_FLAG_LISTS_ONLY or
 *   RB_FLAG_FROM_LISTS (the lookup split in two calls).
 *   ws: as for rb_route_batch (rb_workspace_size bytes); the call uses only
 *   its own workspace, so concurrent calls need distinct workspaces.
 * Errors: as rb_knn_topk, plus RB_ERR_DIMS (M < 1, M > RB_MAX_M), RB_ERR_NULL
 * (bank_qual, bank_len, q_hat, l_hat), RB_ERR_UNSUPPORTED (weighting or
 * flags out of range, or both split flags). */
rb_status rb_knn_predict(const void *queries, const void *bank, const float *bank_norms,
                         rb_dtype dtype, int B, int N, int d, int k, const float *bank_qual,
                         const float *bank_len, int M, const rb_options *opts, int32_t *nbr_idx,
                         float *nbr_dist, float *q_hat, float *l_hat, void *ws, size_t ws_bytes,
                         void *stream);

/* rb_route_batch with options: the averaging rule of opts->weighting, then
 * rb_assign_ex's order, budgets and mask. score0 (may be NULL) then holds
 * each request's row over its candidate set (the maxima over the candidates,
 * NaN elsewhere), at the batch-start state. The workspace is the same size as
 * for rb_route_batch (rb_workspace_size). Errors: the union of those of
 * rb_route_batch and rb_assign_ex (order_out is optional here). */
rb_status rb_route_batch_ex(const void *queries, const void *bank, const float *bank_norms,
                            rb_dtype dtype, int B, int N, int d, int k, const float *bank_qual,
                            const float *bank_len, int M, const int32_t *prompt_len,
                            const rb_instances *inst, int I, rb_weights w,
                            const rb_options *opts, int32_t *assign, float *chosen_score,
                            int32_t *nbr_idx, float *nbr_dist, float *q_hat, float *l_hat,
                            float *score0, void *ws, size_t ws_bytes, void *stream);

/* Bytes of the library's own per-GPU workspace used by rb_route_batch_noalloc. */
#define RB_SCRATCH_BYTES (64u << 20)

/* rb_route_batch for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * The arguments and results are those of rb_route_batch without ws and
 * ws_bytes; the workspace is instead a static device array of
 * RB_SCRATCH_BYTES that the library holds on every GPU it runs on until the
 * process ends (its address is looked up once per device, on the first call
 * there). The call allocates nothing: no hipMalloc, hipFree or allocating
 * library routine. Every call on one GPU uses that GPU's single array, and
 * nothing in it has to start cleared: calls that overlap in time on one GPU
 * (on different streams, or from different host threads without ordering)
 * race on it and give undefined results; calls ordered on one stream are
 * safe. The workspace these sizes need is rb_workspace_size's; sizes needing
 * more than RB_SCRATCH_BYTES (for instance more than 64 requests of 768-d
 * bf16 rows through the tile scan, whose worst-case candidate overflow area
 * grows with the batch) are refused with RB_ERR_SCRATCH before anything is
 * enqueued. Errors: those of rb_route_batch (RB_ERR_WORKSPACE aside), plus
 * RB_ERR_SCRATCH, and RB_ERR_HIP if the array's address cannot be found. */
rb_status rb_route_batch_noalloc(const void *queries, const void *bank, const float *bank_norms,
                                 rb_dtype dtype, int B, int N, int d, int k,
                                 const float *bank_qual, const float *bank_len, int M,
                                 const int32_t *prompt_len, const rb_instances *inst, int I,
                                 rb_weights w, int32_t *assign, float *chosen_score,
                                 int32_t *nbr_idx, float *nbr_dist, float *q_hat, float *l_hat,
                                 float *score0, void *stream);

/* Carry the dead-reckoned state across a gap of dt_seconds between batches:
 *   prefill_q[i] = max(0, prefill_q[i] - prefill_rate[i]*dt)
 *   decode_q[i]  = max(0, decode_q[i]  - decode_rate[i]*dt)
 * (a clamped linear drain; the paper re-reads telemetry per batch instead).
 * Errors: RB_ERR_NULL, RB_ERR_DIMS (I < 1, I > RB_MAX_I, dt not finite or < 0),
 * RB_ERR_HIP. */
rb_status rb_advance_state(const rb_instances *inst, int I, float dt_seconds, void *stream);

/* Timing hook for the bank scan, the dominant kernel of rb_knn_topk,
 * rb_knn_predict and the rb_route_batch calls. While set, every later call of
 * those entry points that runs the scan (not rb_knn_predict with
 * RB_FLAG_FROM_LISTS) made from the calling host thread records `begin` (a
 * hipEvent_t) on the call's stream immediately before the bank-scan kernel and
 * `end` immediately after it, so hipEventElapsedTime(begin, end) is that
 * kernel's duration (for a scan in two passes, the span of both scan launches
 * and the bound between them). Pass NULL, NULL to stop. The setting is per
 * host thread; the events stay owned by the caller. Always returns RB_OK. */
rb_status rb_profile_scan_events(void *begin, void *end);

#ifdef __cplusplus
}
#endif

#endif /* ROUTEBALANCE_H */
