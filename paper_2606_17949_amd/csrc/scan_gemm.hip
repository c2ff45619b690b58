// GEMM-structured bank-scan launcher.
#include "scan_gemm.hpp"

namespace rb {

hipError_t launch_scan_gemm(const KnnPlan &p, const ScanArgs &a, hipStream_t s)
{
    hipError_t e = hipFuncSetAttribute((const void *)gemm_scan_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)p.lds_bytes);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(gemm_scan_kernel, dim3(p.grid), dim3(GM_WAVES * WAVE), p.lds_bytes, s, a);
    return hipGetLastError();
}

}  // namespace rb
