// Bank-scan instantiations for bf16 embeddings whose d is not a multiple of the 64-byte k-step.
#include "scan.hpp"

namespace rb {

hipError_t launch_scan_bf16_ragged(const KnnPlan &p, const ScanArgs &a, hipStream_t s)
{
    return launch_scan_r<1, true>(p, a, p.grid, s);
}

}  // namespace rb
