// Internal launch interface between the C ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace rb {

constexpr int SCAN_THREADS = 256;         // 4 waves
constexpr int SCAN_WAVES = 4;
constexpr int SCAN_WR = 32;               // bank rows per wave per iteration (two 16-row MFMA tiles)
constexpr int SCAN_RT = SCAN_WAVES * SCAN_WR;   // bank rows per workgroup iteration
constexpr int SCAN_DSTRIDE = SCAN_RT + 4; // padded row stride of the distance tile (words)
constexpr size_t LDS_LIMIT = 160 * 1024;
constexpr int MERGE_THREADS = 256;
constexpr int MERGE_MAX_EPT = 32;         // partial entries per merge thread
constexpr int MERGE_MAX_ENTRIES = MERGE_THREADS * MERGE_MAX_EPT;
constexpr int RB_MAX_K_DEV = 64;          // largest k (the ABI limit)

// How one rb_knn_topk call is split: query tiles of qt = 16*ng queries, the
// bank cut into n_chunks contiguous row ranges, one workgroup per
// (chunk, query tile).
struct KnnPlan {
    int dtype;          // 0 fp32, 1 bf16
    int B, N, d, k;
    int ng;             // query groups of 16 per tile (1, 2 or 4)
    int n_qt;           // query tiles
    int nks;            // 64-byte k-steps per row
    int n_chunks;       // bank chunks
    long rows_per_chunk;
    size_t lds_bytes;   // dynamic LDS of the scan kernel
    size_t off_tau, off_pkey, off_pidx, bytes;   // workspace layout
};

int plan_knn(int B, int N, int d, int dtype, int k, int num_cu, KnnPlan *p);

// Events recorded around the bank-scan kernel when set (per host thread).
void set_scan_events(hipEvent_t begin, hipEvent_t end);

hipError_t launch_bank_norms(const void *bank, int dtype, int N, int d, float *norms,
                             hipStream_t s);
hipError_t launch_knn(const KnnPlan &p, const void *queries, const void *bank,
                      const float *bank_norms, void *ws, int32_t *nbr_idx, float *nbr_dist,
                      const float *bank_qual, const float *bank_len, int M, float *q_hat,
                      float *l_hat, hipStream_t s);
hipError_t launch_predict(const int32_t *nbr_idx, int B, int k, const float *bank_qual,
                          const float *bank_len, int N, int M, float *q_hat, float *l_hat,
                          hipStream_t s);

struct InstArgs {
    const int32_t *model;
    float *p, *a;
    const float *P, *D, *cin, *cout;
};

hipError_t launch_score(const float *q_hat, const float *l_hat, const int32_t *plen, int B, int M,
                        const InstArgs &in, int I, float wq, float wl, float wc, float *S0,
                        hipStream_t s);
hipError_t launch_assign(const float *q_hat, const float *l_hat, const int32_t *plen, int B,
                         int M, const InstArgs &in, int I, float wq, float wl, float wc,
                         int32_t *assign, float *chosen, hipStream_t s);
hipError_t launch_advance(const InstArgs &in, int I, float dt, hipStream_t s);

}  // namespace rb
