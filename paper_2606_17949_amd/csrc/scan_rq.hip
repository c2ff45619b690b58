// Query-resident bank scan: dispatch on the row length (one translation unit
// per length holds its instantiations).
#include "knn_common.hpp"

namespace rb {

hipError_t launch_scan_rq(const KnnPlan &p, const ScanArgs &a, hipStream_t s)
{
    switch (p.nks) {
    case 12: return launch_scan_rq12(p, a, s);
    case 16: return launch_scan_rq16(p, a, s);
    case 24: return launch_scan_rq24(p, a, s);
    case 32: return launch_scan_rq32(p, a, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace rb
