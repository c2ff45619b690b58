// Internal launch interface between the C ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace rb {

// The scan runs 8 waves, two per SIMD, each within half the register file
// (256 registers: 128 accumulators for 2 row tiles x 16 query groups): the
// workgroup covers 256 bank rows per iteration, so every streamed query byte
// serves 256 rows, and each SIMD has a second wave to cover load latency.
constexpr int SCAN_THREADS = 512;   // 8 waves, two per SIMD
constexpr int SCAN_WAVES = 8;
constexpr int SCAN_RT = 2;          // 16-row MFMA tiles per wave per iteration (32 rows)
constexpr int SCAN_KPAD = 4;        // k-steps per row are padded to a multiple of this
// Ring depth of the scan's loads, in k-steps (the loop is unrolled by it):
// bank fragments go to a register ring and streamed query fragments to an LDS
// ring of as many slots, both depth - 1 k-steps ahead of the MFMAs. Four for
// tiles below 256 queries. For a full tile, four only for bf16 rows of whole
// k-steps with less than half the tile resident (the fp32 MFMA steps and the
// lane masks of a partial k-step take the registers, and with half the tile
// resident or more the LDS serves better as resident queries than as ring
// slots).
__host__ __device__ constexpr int scan_ring(int dtype, int ng, int gr, bool ragged)
{
    return ng < 16 || (dtype == 1 && !ragged && gr < ng / 2) ? 4 : 2;
}
constexpr int STAGE_CAP = 128;      // per-wave LDS staging of one iteration's candidates
constexpr size_t LDS_LIMIT = 160 * 1024;
constexpr int MERGE_WAVES = 4;      // queries per merge workgroup, one wave each
constexpr int MERGE_CAP = 2048;     // candidates per query the merge holds in LDS
constexpr int MERGE_MAX_LISTS = 64 * 64;   // 64 lists per lane
constexpr int RB_MAX_K_DEV = 64;    // largest k (the ABI limit)
constexpr int SEED_MAX_GROUPS = 2048;  // S / 16 for S <= 32768
// The query-resident scan (bf16 rows of 384, 512, 768 or 1024 elements, a
// batch that fits its waves' registers): RQ_WAVES waves, blocks of RQ_ROWS
// bank rows, a ring of stages of a block's k-steps in LDS.
constexpr int RQ_WAVES = 8;
constexpr int RQ_ROWS = 32;
constexpr int RQ_SMALL_B_MIN_ROWS = 2048;   // bank rows per compute unit, batches of <= 64
constexpr int RQ_SPLIT_MIN_ROWS = 1024;     // chunk rows from which the scan may go in two passes
// The GEMM-structured scan (bf16 rows, d a multiple of GM_KST, more than 256
// requests): GM_WAVES waves per workgroup, macro tiles of GM_ROWS bank rows by
// a tile of GM_QRY requests, K in stages of GM_KST elements in GM_SLOTS LDS
// slots.
constexpr int GM_WAVES = 8;
constexpr int GM_ROWS = 256;
constexpr int GM_QRY = 256;
constexpr int GM_KST = 64;
constexpr int GM_SLOTS = 2;
constexpr int GM_STAGE = 64;   // per-wave LDS staging of one macro tile's candidates

// How one rb_knn_topk call is split (the tile scan; the query-resident scan
// differs in that one workgroup holds the whole batch, so n_qt = 1; the
// GEMM-structured scan in its request tiles of GM_QRY, one workgroup per
// (chunk, tile) with the chunk in macro tiles of GM_ROWS rows).
//  * seed: S bank rows spread evenly over the bank, scored in groups of 16;
//    per query, the k-th smallest of 128 of the S/16 group minima (each
//    lane's two smallest of its share) bounds the k-th nearest distance from
//    above (k distinct rows lie at or below it).
//  * scan: query tiles of 16*ng queries, whose first gr groups stay in LDS
//    for the whole call while the others stream through it; the
//    bank in n_chunks contiguous row ranges (multiples of 16 rows); one
//    workgroup per (chunk, tile); each of its SCAN_WAVES waves owns 16*rt rows per
//    iteration; the workgroup keeps, per query, one list of the k best
//    candidates that pass the bound.
//  * merge: per query, the k smallest of its W lists (W = n_chunks, times
//    the row halves rs of the query-resident scan).
struct KnnPlan {
    int kind;           // 0 tile scan, 1 query-resident scan, 2 GEMM-structured scan
    int qw, rs, spb;    // query-resident scan: query groups per wave, row halves, stages per block,
    int stages;         //   ring slots
    int dtype;          // 0 fp32, 1 bf16
    int B, N, d, k;
    int nks, nksp;      // 64-byte k-steps per row, padded to SCAN_KPAD
    int ng, gr, rt;     // query groups of 16 per tile (gr of them resident), 16-row tiles per wave
    int n_qt, n_chunks, W;   // request tiles, bank chunks, lists per query the scan leaves
    long rows_per_chunk;
    int S, G;           // seed rows and groups (0 = no seed)
    int rq_split;       // query-resident scan: rows of every chunk in its first pass (0 = one pass)
    int grid;           // scan workgroups
    int ovf_cap;        // candidates per scan wave that the workspace takes past LDS
    size_t lds_bytes;
    size_t off_tau, off_qn, off_gmin, off_ccnt, off_ckey, off_cidx, off_ovf, bytes;
};

// reserve: compute units per XCD to leave free for kernels of other streams.
int plan_knn(int B, int N, int d, int dtype, int k, int num_cu, KnnPlan *p, int reserve = 0);

// Events recorded around the bank-scan kernel when set (per host thread).
void set_scan_events(hipEvent_t begin, hipEvent_t end);

hipError_t launch_bank_norms(const void *bank, int dtype, int N, int d, float *norms,
                             hipStream_t s);
// The halves of launch_knn: the seed and the bank scan (which leave the
// per-chunk lists in the workspace), and the merge of those lists.
enum KnnPhases { KNN_LISTS = 1, KNN_MERGE = 2, KNN_ALL = 3 };
// With q_hat non-null, the merge also averages the labels (inv_dist: with
// inverse-distance weights instead of the plain mean).
hipError_t launch_knn(const KnnPlan &p, const void *queries, const void *bank,
                      const float *bank_norms, void *ws, int32_t *nbr_idx, float *nbr_dist,
                      const float *bank_qual, const float *bank_len, int M, float *q_hat,
                      float *l_hat, bool inv_dist, hipStream_t s, int phases = KNN_ALL);
hipError_t launch_predict(const int32_t *nbr_idx, const float *nbr_dist, int B, int k,
                          bool inv_dist, const float *bank_qual, const float *bank_len, int N,
                          int M, float *q_hat, float *l_hat, hipStream_t s);

struct InstArgs {
    const int32_t *model;
    float *p, *a;
    const float *P, *D, *cin, *cout;
};

// Options of the greedy loop; null pointers are the defaults (arrival order,
// no budgets, every instance available).
struct AssignOpts {
    const int32_t *order;    // [B] request decided at each step
    const float *budget;     // [B] per-request cost budget
    const uint8_t *mask;     // [I] nonzero = available
};

// The dense score matrix; opt's budget and mask restrict each row's
// candidates (its order is not read).
hipError_t launch_score(const float *q_hat, const float *l_hat, const int32_t *plen, int B, int M,
                        const InstArgs &in, int I, float wq, float wl, float wc,
                        const AssignOpts &opt, float *S0, hipStream_t s);

hipError_t launch_lpt_order(const float *l_hat, int B, int M, int32_t *order, hipStream_t s);
// out[i] = i for i < n (the arrival order, when the caller asks for it).
hipError_t launch_iota(int32_t *out, int n, hipStream_t s);
hipError_t launch_assign(const float *q_hat, const float *l_hat, const int32_t *plen, int B,
                         int M, const InstArgs &in, int I, float wq, float wl, float wc,
                         const AssignOpts &opt, int32_t *assign, float *chosen, float *decided,
                         hipStream_t s);
hipError_t launch_advance(const InstArgs &in, int I, float dt, hipStream_t s);

}  // namespace rb
