// Query-resident bank-scan instantiations: bf16 rows of 512 elements.
#include "scan_rq.hpp"

namespace rb {

hipError_t launch_scan_rq16(const KnnPlan &p, const ScanArgs &a, hipStream_t s)
{
    return launch_rq_nks<16>(p, a, s);
}

}  // namespace rb
