// Bank-scan instantiations for bf16 embeddings, d a multiple of the 64-byte k-step.
#include "scan.hpp"

namespace rb {

hipError_t launch_scan_bf16(const KnnPlan &p, const ScanArgs &a, hipStream_t s)
{
    return launch_scan_r<1, false>(p, a, p.grid, s);
}

}  // namespace rb
