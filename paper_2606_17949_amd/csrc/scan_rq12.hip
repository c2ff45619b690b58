// Query-resident bank-scan instantiations: bf16 rows of 384 elements.
#include "scan_rq.hpp"

namespace rb {

hipError_t launch_scan_rq12(const KnnPlan &p, const ScanArgs &a, hipStream_t s)
{
    return launch_rq_nks<12>(p, a, s);
}

}  // namespace rb
