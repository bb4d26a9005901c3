// launch_direct.hip -- instances of the DIRECT configurations (both B layouts)
// and of the ping-pong kernel (row-major B).
#include "families.h"
#include "kern_direct.h"

namespace gemm {

template <int DT, int BM, int BN, int WM, int WN, int WPE>
static hipError_t launch_direct(const KernelArgs &a, int64_t grid, hipStream_t stream) {
    if (a.b_trans)
        hipLaunchKernelGGL((gemm_lds_kernel<DT, BM, BN, WM, WN, WPE, true>), dim3(unsigned(grid)),
                           dim3(64 * WM * WN), 0, stream, a);
    else
        hipLaunchKernelGGL((gemm_lds_kernel<DT, BM, BN, WM, WN, WPE, false>), dim3(unsigned(grid)),
                           dim3(64 * WM * WN), 0, stream, a);
    return hipGetLastError();
}

template <int DT>
hipError_t launch_direct_family(int32_t cfg, const KernelArgs &a, int64_t grid, hipStream_t s) {
    switch (cfg) {
        case 8: return launch_direct<DT, 256, 256, 2, 2, 1>(a, grid, s);
        case 9: return launch_direct<DT, 128, 256, 2, 2, 1>(a, grid, s);
        case 10: return launch_direct<DT, 256, 256, 2, 4, 2>(a, grid, s);
        case 11: return launch_direct<DT, 256, 256, 4, 2, 2>(a, grid, s);
        case 12: return launch_direct<DT, 128, 256, 2, 4, 2>(a, grid, s);
        case 13:
            if (a.b_trans) return hipErrorInvalidValue;
            hipLaunchKernelGGL((gemm_pingpong_kernel<DT>), dim3(unsigned(grid)), dim3(512), 0, s, a);
            return hipGetLastError();
        default: return hipErrorInvalidValue;
    }
}

template hipError_t launch_direct_family<DT_I8>(int32_t, const KernelArgs &, int64_t, hipStream_t);
template hipError_t launch_direct_family<DT_BF16>(int32_t, const KernelArgs &, int64_t, hipStream_t);

}  // namespace gemm
