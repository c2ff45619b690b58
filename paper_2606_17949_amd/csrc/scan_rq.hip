// Query-resident bank-scan instantiations: bf16 rows of 768 elements.
#include "scan_rq.hpp"

namespace rb {

hipError_t launch_scan_rq(const KnnPlan &p, const ScanArgs &a, hipStream_t s)
{
    if (p.nks == RQ_NKS && p.qw == RQ_QW)
        return launch_rq_scan<RQ_NKS, RQ_QW>(a, p.lds_bytes, p.grid, s);
    return hipErrorInvalidValue;
}

}  // namespace rb
