// C ABI of the routing path: host-side validation, workspace layout and
// kernel dispatch. Nothing here allocates, copies to the host or
// synchronises; every call enqueues on the caller's stream.
#include <math.h>

#include <atomic>
#include <mutex>

#include "../../include/routebalance.h"
#include "kernels.hpp"

namespace {

constexpr int MAX_DEVICES = 64;
std::atomic<int> g_num_cu[MAX_DEVICES];

// The workspace of rb_route_batch_noalloc: one copy on every device the
// library runs on. In host code `scratch` names a host-side stand-in, not
// the device array; its device address comes from hipGetSymbolAddress, once
// per device, and only that address is ever handed to a kernel.
static __device__ __align__(256) uint8_t scratch[RB_SCRATCH_BYTES];
std::atomic<void *> g_scratch[MAX_DEVICES];
std::mutex g_scratch_mu;

// Device address of the current device's scratch array, or null.
void *scratch_ptr()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES)
        return nullptr;
    void *p = g_scratch[dev].load(std::memory_order_acquire);
    if (p)
        return p;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (!p) {
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p)
            return nullptr;
        g_scratch[dev].store(p, std::memory_order_release);
    }
    return p;
}

// Compute units of the current device (cached per device).
int num_cu(int *out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0)
        return -1;
    if (dev < MAX_DEVICES) {
        const int c = g_num_cu[dev].load(std::memory_order_relaxed);
        if (c > 0) {
            *out = c;
            return 0;
        }
    }
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n < 1)
        return -1;
    if (dev < MAX_DEVICES)
        g_num_cu[dev].store(n, std::memory_order_relaxed);
    *out = n;
    return 0;
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

rb_status check_embed_dims(rb_dtype dt, int N, int d)
{
    if (dt != RB_F32 && dt != RB_BF16)
        return RB_ERR_DTYPE;
    if (N < 1 || d < 1 || d > RB_MAX_D)
        return RB_ERR_DIMS;
    if (d % (dt == RB_BF16 ? 8 : 4) != 0)
        return RB_ERR_DIMS;
    return RB_OK;
}

rb_status check_knn_dims(rb_dtype dt, int B, int N, int d, int k)
{
    const rb_status s = check_embed_dims(dt, N, d);
    if (s != RB_OK)
        return s;
    if (B < 0 || k < 1 || k > RB_MAX_K || k > N)
        return RB_ERR_DIMS;
    return RB_OK;
}

rb_status check_weights(rb_weights w)
{
    const float v[3] = {w.w_qual, w.w_lat, w.w_cost};
    for (float x : v)
        if (!isfinite(x) || x < 0.f)
            return RB_ERR_WEIGHTS;
    if (fabs((double)v[0] + (double)v[1] + (double)v[2] - 1.0) > 1e-5)
        return RB_ERR_WEIGHTS;
    return RB_OK;
}

rb_status check_inst(const rb_instances *in, int I)
{
    if (!in)
        return RB_ERR_NULL;
    if (I < 1 || I > RB_MAX_I)
        return RB_ERR_DIMS;
    if (!in->model || !in->prefill_q || !in->decode_q || !in->prefill_rate || !in->decode_rate ||
        !in->price_in || !in->price_out)
        return RB_ERR_NULL;
    return RB_OK;
}

rb::InstArgs inst_args(const rb_instances *in)
{
    rb::InstArgs a;
    a.model = in->model;
    a.p = in->prefill_q;
    a.a = in->decode_q;
    a.P = in->prefill_rate;
    a.D = in->decode_rate;
    a.cin = in->price_in;
    a.cout = in->price_out;
    return a;
}

// Workspace of rb_route_batch beyond the KNN plan: neighbour list,
// predictions and processing order for callers that do not want them back.
struct RouteExtra {
    size_t off_nbr, off_qhat, off_lhat, off_order, bytes;
};

RouteExtra route_extra(size_t base, int B, int k, int M)
{
    RouteExtra e;
    size_t off = base;
    e.off_nbr = off;
    off += align256((size_t)B * k * 4);
    e.off_qhat = off;
    off += align256((size_t)B * M * 4);
    e.off_lhat = off;
    off += align256((size_t)B * M * 4);
    e.off_order = off;
    off += align256((size_t)B * 4);
    e.bytes = off;
    return e;
}

const rb_options k_default_opts = {RB_ORDER_ARRIVAL, RB_KNN_UNIFORM, nullptr, nullptr, nullptr,
                                   0u};

// `flags_ok`: the flag bits the entry point takes.
rb_status check_opts(const rb_options *o, uint32_t flags_ok = RB_FLAG_OVERLAP)
{
    if (o->order != RB_ORDER_ARRIVAL && o->order != RB_ORDER_LPT)
        return RB_ERR_UNSUPPORTED;
    if (o->weighting != RB_KNN_UNIFORM && o->weighting != RB_KNN_INV_DIST)
        return RB_ERR_UNSUPPORTED;
    if (o->flags & ~flags_ok)
        return RB_ERR_UNSUPPORTED;
    if ((o->flags & RB_FLAG_LISTS_ONLY) && (o->flags & RB_FLAG_FROM_LISTS))
        return RB_ERR_UNSUPPORTED;
    return RB_OK;
}

// The greedy loop with options: the LPT order first (into `order`), then the
// loop over it.
hipError_t enqueue_assign(const float *qh, const float *lh, const int32_t *plen, int B, int M,
                          const rb_instances *inst, int I, rb_weights w, const rb_options *o,
                          int32_t *order, int32_t *assign, float *chosen, float *decided,
                          hipStream_t st)
{
    rb::AssignOpts ao;
    ao.order = nullptr;
    ao.budget = o->budget;
    ao.mask = o->instance_mask;
    if (o->order == RB_ORDER_LPT) {
        const hipError_t e = rb::launch_lpt_order(lh, B, M, order, st);
        if (e != hipSuccess)
            return e;
        ao.order = order;
    }
    return rb::launch_assign(qh, lh, plen, B, M, inst_args(inst), I, w.w_qual, w.w_lat, w.w_cost,
                             ao, assign, chosen, decided, st);
}

// The dense score matrix at the current state over each request's candidate
// set (the options' budgets and mask).
hipError_t enqueue_score(const float *qh, const float *lh, const int32_t *plen, int B, int M,
                         const rb_instances *inst, int I, rb_weights w, const rb_options *o,
                         float *score0, hipStream_t st)
{
    rb::AssignOpts ao;
    ao.order = nullptr;
    ao.budget = o->budget;
    ao.mask = o->instance_mask;
    return rb::launch_score(qh, lh, plen, B, M, inst_args(inst), I, w.w_qual, w.w_lat, w.w_cost,
                            ao, score0, st);
}

// The KNN plan on the current device. With `overlap`, the scan leaves one
// compute unit of each XCD free, so that a single-workgroup kernel of another
// stream (the greedy pass, the carry) finds room on whichever XCD it is
// dispatched to instead of waiting for the scan to drain.
// rb_workspace_size covers both plans.
rb_status plan(int B, int N, int d, rb_dtype dt, int k, rb::KnnPlan *p, bool overlap = false)
{
    int cu = 0;
    if (num_cu(&cu) != 0)
        return RB_ERR_HIP;
    if (rb::plan_knn(B, N, d, (int)dt, k, cu, p, overlap ? 1 : 0) != 0)
        return RB_ERR_DIMS;
    return RB_OK;
}

rb_status hip_status(hipError_t e) { return e == hipSuccess ? RB_OK : RB_ERR_HIP; }

rb_status route_batch(const void *queries, const void *bank, const float *bank_norms,
                      rb_dtype dtype, int B, int N, int d, int k, const float *bank_qual,
                      const float *bank_len, int M, const int32_t *prompt_len,
                      const rb_instances *inst, int I, rb_weights w, const rb_options *o,
                      int32_t *assign, float *chosen_score, int32_t *nbr_idx, float *nbr_dist,
                      float *q_hat, float *l_hat, float *score0, void *ws, size_t ws_bytes,
                      void *stream)
{
    rb_status s = check_knn_dims(dtype, B, N, d, k);
    if (s != RB_OK)
        return s;
    if (M < 1 || M > RB_MAX_M)
        return RB_ERR_DIMS;
    if ((s = check_inst(inst, I)) != RB_OK)
        return s;
    if ((s = check_weights(w)) != RB_OK)
        return s;
    if ((s = check_opts(o)) != RB_OK)
        return s;
    if (B == 0)
        return RB_OK;
    if (!queries || !bank || !bank_norms || !bank_qual || !bank_len || !prompt_len || !assign)
        return RB_ERR_NULL;
    if (!aligned(queries, 16) || !aligned(bank, 16))
        return RB_ERR_ALIGN;
    rb::KnnPlan p;
    if ((s = plan(B, N, d, dtype, k, &p, (o->flags & RB_FLAG_OVERLAP) != 0)) != RB_OK)
        return s;
    const RouteExtra ex = route_extra(p.bytes, B, k, M);
    if (!ws || ws_bytes < ex.bytes)
        return RB_ERR_WORKSPACE;
    if (!aligned(ws, 256))
        return RB_ERR_ALIGN;
    uint8_t *wb = (uint8_t *)ws;
    int32_t *nbr = nbr_idx ? nbr_idx : (int32_t *)(wb + ex.off_nbr);
    float *qh = q_hat ? q_hat : (float *)(wb + ex.off_qhat);
    float *lh = l_hat ? l_hat : (float *)(wb + ex.off_lhat);
    int32_t *order = o->order_out ? o->order_out : (int32_t *)(wb + ex.off_order);
    hipStream_t st = (hipStream_t)stream;
    hipError_t e = rb::launch_knn(p, queries, bank, bank_norms, ws, nbr, nbr_dist, bank_qual,
                                  bank_len, M, qh, lh, o->weighting == RB_KNN_INV_DIST, st);
    if (e != hipSuccess)
        return RB_ERR_HIP;
    if (score0 &&
        (e = enqueue_score(qh, lh, prompt_len, B, M, inst, I, w, o, score0, st)) != hipSuccess)
        return RB_ERR_HIP;
    e = enqueue_assign(qh, lh, prompt_len, B, M, inst, I, w, o, order, assign, chosen_score,
                       nullptr, st);
    if (e == hipSuccess && o->order != RB_ORDER_LPT && o->order_out)
        e = rb::launch_iota(o->order_out, B, st);
    return hip_status(e);
}

}  // namespace

extern "C" {

const char *rb_status_string(rb_status s)
{
    switch (s) {
    case RB_OK: return "RB_OK";
    case RB_ERR_NULL: return "RB_ERR_NULL: a required pointer is NULL";
    case RB_ERR_DIMS: return "RB_ERR_DIMS: a size is out of range";
    case RB_ERR_DTYPE: return "RB_ERR_DTYPE: unsupported dtype";
    case RB_ERR_WEIGHTS: return "RB_ERR_WEIGHTS: weights are not on the 3-simplex";
    case RB_ERR_WORKSPACE: return "RB_ERR_WORKSPACE: workspace missing or too small";
    case RB_ERR_UNSUPPORTED: return "RB_ERR_UNSUPPORTED: option not implemented";
    case RB_ERR_HIP: return "RB_ERR_HIP: HIP runtime or launch failure";
    case RB_ERR_ALIGN: return "RB_ERR_ALIGN: pointer not aligned as required";
    case RB_ERR_SCRATCH:
        return "RB_ERR_SCRATCH: these sizes need more workspace than the library's static "
               "RB_SCRATCH_BYTES";
    }
    return "unknown rb_status";
}

rb_status rb_workspace_size(int B, int N, int d, rb_dtype dtype, int k, int M, size_t *bytes)
{
    if (!bytes)
        return RB_ERR_NULL;
    rb_status s = check_knn_dims(dtype, B, N, d, k);
    if (s != RB_OK)
        return s;
    if (M < 1 || M > RB_MAX_M)
        return RB_ERR_DIMS;
    rb::KnnPlan p, q;
    if ((s = plan(B, N, d, dtype, k, &p)) != RB_OK)
        return s;
    if ((s = plan(B, N, d, dtype, k, &q, true)) != RB_OK)
        return s;
    *bytes = route_extra(p.bytes > q.bytes ? p.bytes : q.bytes, B, k, M).bytes;
    return RB_OK;
}

rb_status rb_bank_norms(const void *bank, rb_dtype dtype, int N, int d, float *norms,
                        void *stream)
{
    const rb_status s = check_embed_dims(dtype, N, d);
    if (s != RB_OK)
        return s;
    if (!bank || !norms)
        return RB_ERR_NULL;
    if (!aligned(bank, 16))
        return RB_ERR_ALIGN;
    return hip_status(rb::launch_bank_norms(bank, (int)dtype, N, d, norms, (hipStream_t)stream));
}

rb_status rb_knn_topk(const void *queries, const void *bank, const float *bank_norms,
                      rb_dtype dtype, int B, int N, int d, int k, int32_t *nbr_idx,
                      float *nbr_dist, void *ws, size_t ws_bytes, void *stream)
{
    rb_status s = check_knn_dims(dtype, B, N, d, k);
    if (s != RB_OK)
        return s;
    if (B == 0)
        return RB_OK;
    if (!queries || !bank || !bank_norms || !nbr_idx)
        return RB_ERR_NULL;
    if (!aligned(queries, 16) || !aligned(bank, 16))
        return RB_ERR_ALIGN;
    rb::KnnPlan p;
    if ((s = plan(B, N, d, dtype, k, &p)) != RB_OK)
        return s;
    if (!ws || ws_bytes < p.bytes)
        return RB_ERR_WORKSPACE;
    if (!aligned(ws, 256))
        return RB_ERR_ALIGN;
    return hip_status(rb::launch_knn(p, queries, bank, bank_norms, ws, nbr_idx, nbr_dist, nullptr,
                                     nullptr, 0, nullptr, nullptr, false, (hipStream_t)stream));
}

rb_status rb_predict(const int32_t *nbr_idx, const float *nbr_dist, int B, int k,
                     rb_knn_weighting weighting, const float *bank_qual, const float *bank_len,
                     int N, int M, float *q_hat, float *l_hat, void *stream)
{
    if (B < 0 || k < 1 || k > RB_MAX_K || N < 1 || M < 1 || M > RB_MAX_M)
        return RB_ERR_DIMS;
    if (weighting != RB_KNN_UNIFORM && weighting != RB_KNN_INV_DIST)
        return RB_ERR_UNSUPPORTED;
    if (B == 0)
        return RB_OK;
    const bool inv = weighting == RB_KNN_INV_DIST;
    if (!nbr_idx || !bank_qual || !bank_len || !q_hat || !l_hat || (inv && !nbr_dist))
        return RB_ERR_NULL;
    return hip_status(rb::launch_predict(nbr_idx, nbr_dist, B, k, inv, bank_qual, bank_len, N, M,
                                         q_hat, l_hat, (hipStream_t)stream));
}

rb_status rb_score(const float *q_hat, const float *l_hat, const int32_t *prompt_len, int B,
                   int M, const rb_instances *inst, int I, rb_weights w, float *score0,
                   void *stream)
{
    if (B < 0 || M < 1 || M > RB_MAX_M)
        return RB_ERR_DIMS;
    rb_status s = check_inst(inst, I);
    if (s != RB_OK)
        return s;
    if ((s = check_weights(w)) != RB_OK)
        return s;
    if (B == 0)
        return RB_OK;
    if (!q_hat || !l_hat || !prompt_len || !score0)
        return RB_ERR_NULL;
    return hip_status(enqueue_score(q_hat, l_hat, prompt_len, B, M, inst, I, w, &k_default_opts,
                                    score0, (hipStream_t)stream));
}

rb_status rb_assign(const float *q_hat, const float *l_hat, const int32_t *prompt_len, int B,
                    int M, const rb_instances *inst, int I, rb_weights w, int32_t *assign,
                    float *chosen_score, float *decided, void *stream)
{
    if (B < 0 || M < 1 || M > RB_MAX_M)
        return RB_ERR_DIMS;
    rb_status s = check_inst(inst, I);
    if (s != RB_OK)
        return s;
    if ((s = check_weights(w)) != RB_OK)
        return s;
    if (B == 0)
        return RB_OK;
    if (!q_hat || !l_hat || !prompt_len || !assign)
        return RB_ERR_NULL;
    return hip_status(enqueue_assign(q_hat, l_hat, prompt_len, B, M, inst, I, w, &k_default_opts,
                                     nullptr, assign, chosen_score, decided,
                                     (hipStream_t)stream));
}

rb_status rb_assign_ex(const float *q_hat, const float *l_hat, const int32_t *prompt_len, int B,
                       int M, const rb_instances *inst, int I, rb_weights w,
                       const rb_options *opts, int32_t *assign, float *chosen_score,
                       float *decided, void *stream)
{
    const rb_options *o = opts ? opts : &k_default_opts;
    if (B < 0 || M < 1 || M > RB_MAX_M)
        return RB_ERR_DIMS;
    rb_status s = check_inst(inst, I);
    if (s != RB_OK)
        return s;
    if ((s = check_weights(w)) != RB_OK)
        return s;
    if ((s = check_opts(o)) != RB_OK)
        return s;
    if (B == 0)
        return RB_OK;
    if (!q_hat || !l_hat || !prompt_len || !assign)
        return RB_ERR_NULL;
    if (o->order == RB_ORDER_LPT && !o->order_out)
        return RB_ERR_NULL;
    hipStream_t st = (hipStream_t)stream;
    hipError_t e = enqueue_assign(q_hat, l_hat, prompt_len, B, M, inst, I, w, o, o->order_out,
                                  assign, chosen_score, decided, st);
    if (e == hipSuccess && o->order != RB_ORDER_LPT && o->order_out)
        e = rb::launch_iota(o->order_out, B, st);
    return hip_status(e);
}

rb_status rb_knn_predict(const void *queries, const void *bank, const float *bank_norms,
                         rb_dtype dtype, int B, int N, int d, int k, const float *bank_qual,
                         const float *bank_len, int M, const rb_options *opts, int32_t *nbr_idx,
                         float *nbr_dist, float *q_hat, float *l_hat, void *ws, size_t ws_bytes,
                         void *stream)
{
    const rb_options *o = opts ? opts : &k_default_opts;
    rb_status s = check_knn_dims(dtype, B, N, d, k);
    if (s != RB_OK)
        return s;
    if (M < 1 || M > RB_MAX_M)
        return RB_ERR_DIMS;
    if ((s = check_opts(o, RB_FLAG_OVERLAP | RB_FLAG_LISTS_ONLY | RB_FLAG_FROM_LISTS)) != RB_OK)
        return s;
    if (B == 0)
        return RB_OK;
    // the halves of the lookup: seed and scan to the lists, then merge and average
    const bool lists_only = (o->flags & RB_FLAG_LISTS_ONLY) != 0;
    const bool from_lists = (o->flags & RB_FLAG_FROM_LISTS) != 0;
    if (!from_lists && (!queries || !bank || !bank_norms))
        return RB_ERR_NULL;
    if (!lists_only && (!bank_qual || !bank_len || !q_hat || !l_hat))
        return RB_ERR_NULL;
    if (!from_lists && (!aligned(queries, 16) || !aligned(bank, 16)))
        return RB_ERR_ALIGN;
    rb::KnnPlan p;
    if ((s = plan(B, N, d, dtype, k, &p, (o->flags & RB_FLAG_OVERLAP) != 0)) != RB_OK)
        return s;
    const RouteExtra ex = route_extra(p.bytes, B, k, M);
    if (!ws || ws_bytes < ex.bytes)
        return RB_ERR_WORKSPACE;
    if (!aligned(ws, 256))
        return RB_ERR_ALIGN;
    int32_t *nbr = nbr_idx ? nbr_idx : (int32_t *)((uint8_t *)ws + ex.off_nbr);
    const int phases = lists_only ? rb::KNN_LISTS : from_lists ? rb::KNN_MERGE : rb::KNN_ALL;
    return hip_status(rb::launch_knn(p, queries, bank, bank_norms, ws, nbr, nbr_dist, bank_qual,
                                     bank_len, M, q_hat, l_hat,
                                     o->weighting == RB_KNN_INV_DIST, (hipStream_t)stream,
                                     phases));
}

rb_status rb_route_batch(const void *queries, const void *bank, const float *bank_norms,
                         rb_dtype dtype, int B, int N, int d, int k, const float *bank_qual,
                         const float *bank_len, int M, const int32_t *prompt_len,
                         const rb_instances *inst, int I, rb_weights w, int32_t *assign,
                         float *chosen_score, int32_t *nbr_idx, float *nbr_dist, float *q_hat,
                         float *l_hat, float *score0, void *ws, size_t ws_bytes, void *stream)
{
    return route_batch(queries, bank, bank_norms, dtype, B, N, d, k, bank_qual, bank_len, M,
                       prompt_len, inst, I, w, &k_default_opts, assign, chosen_score, nbr_idx,
                       nbr_dist, q_hat, l_hat, score0, ws, ws_bytes, stream);
}

rb_status rb_route_batch_ex(const void *queries, const void *bank, const float *bank_norms,
                            rb_dtype dtype, int B, int N, int d, int k, const float *bank_qual,
                            const float *bank_len, int M, const int32_t *prompt_len,
                            const rb_instances *inst, int I, rb_weights w,
                            const rb_options *opts, int32_t *assign, float *chosen_score,
                            int32_t *nbr_idx, float *nbr_dist, float *q_hat, float *l_hat,
                            float *score0, void *ws, size_t ws_bytes, void *stream)
{
    return route_batch(queries, bank, bank_norms, dtype, B, N, d, k, bank_qual, bank_len, M,
                       prompt_len, inst, I, w, opts ? opts : &k_default_opts, assign,
                       chosen_score, nbr_idx, nbr_dist, q_hat, l_hat, score0, ws, ws_bytes,
                       stream);
}

rb_status rb_route_batch_noalloc(const void *queries, const void *bank, const float *bank_norms,
                                 rb_dtype dtype, int B, int N, int d, int k,
                                 const float *bank_qual, const float *bank_len, int M,
                                 const int32_t *prompt_len, const rb_instances *inst, int I,
                                 rb_weights w, int32_t *assign, float *chosen_score,
                                 int32_t *nbr_idx, float *nbr_dist, float *q_hat, float *l_hat,
                                 float *score0, void *stream)
{
    // the size checks of rb_route_batch first, so that a too-large batch is
    // refused as such and not as a short workspace
    rb_status s = check_knn_dims(dtype, B, N, d, k);
    if (s != RB_OK)
        return s;
    if (M < 1 || M > RB_MAX_M)
        return RB_ERR_DIMS;
    if (B == 0)
        return route_batch(queries, bank, bank_norms, dtype, B, N, d, k, bank_qual, bank_len, M,
                           prompt_len, inst, I, w, &k_default_opts, assign, chosen_score, nbr_idx,
                           nbr_dist, q_hat, l_hat, score0, nullptr, 0, stream);
    rb::KnnPlan p;
    if ((s = plan(B, N, d, dtype, k, &p)) != RB_OK)
        return s;
    if (route_extra(p.bytes, B, k, M).bytes > (size_t)RB_SCRATCH_BYTES)
        return RB_ERR_SCRATCH;
    void *ws = scratch_ptr();
    if (!ws)
        return RB_ERR_HIP;
    return route_batch(queries, bank, bank_norms, dtype, B, N, d, k, bank_qual, bank_len, M,
                       prompt_len, inst, I, w, &k_default_opts, assign, chosen_score, nbr_idx,
                       nbr_dist, q_hat, l_hat, score0, ws, RB_SCRATCH_BYTES, stream);
}

rb_status rb_profile_scan_events(void *begin, void *end)
{
    rb::set_scan_events((hipEvent_t)begin, (hipEvent_t)end);
    return RB_OK;
}

rb_status rb_advance_state(const rb_instances *inst, int I, float dt_seconds, void *stream)
{
    const rb_status s = check_inst(inst, I);
    if (s != RB_OK)
        return s;
    if (!isfinite(dt_seconds) || dt_seconds < 0.f)
        return RB_ERR_DIMS;
    return hip_status(rb::launch_advance(inst_args(inst), I, dt_seconds, (hipStream_t)stream));
}

}  // extern "C"
