// launch_ring.h -- the RING configurations.  Instantiated for one dtype and one
// B layout per translation unit (launch_ring_{i8,bf16}_{row,col}.hip): this
// family has the most instances.
#pragma once

#include "families.h"
#include "kern_ring.h"

namespace gemm {

template <int DT, bool BT, int BM, int BN, int WM, int WN, int WPE, int NB>
static hipError_t launch_ring(const KernelArgs &a, int64_t grid, hipStream_t stream) {
    hipLaunchKernelGGL((gemm_ring_kernel<DT, BM, BN, WM, WN, WPE, BT, NB>), dim3(unsigned(grid)),
                       dim3(64 * WM * WN), 0, stream, a);
    return hipGetLastError();
}

template <int DT, bool BT>
hipError_t launch_ring_family(int32_t cfg, const KernelArgs &a, int64_t grid, hipStream_t s) {
    if (bool(a.b_trans) != BT) return hipErrorInvalidValue;
    switch (cfg) {
        case 16: return launch_ring<DT, BT, 256, 256, 2, 4, 2, 4>(a, grid, s);
        case 17: return launch_ring<DT, BT, 256, 256, 4, 2, 2, 4>(a, grid, s);
        case 18: return launch_ring<DT, BT, 128, 256, 2, 4, 2, 5>(a, grid, s);
        case 19: return launch_ring<DT, BT, 256, 256, 2, 2, 1, 4>(a, grid, s);
        case 20: return launch_ring<DT, BT, 32, 64, 1, 2, 2, 8>(a, grid, s);
        case 21: return launch_ring<DT, BT, 64, 64, 1, 2, 2, 8>(a, grid, s);
        case 22: return launch_ring<DT, BT, 32, 128, 1, 4, 2, 8>(a, grid, s);
        case 23: return launch_ring<DT, BT, 64, 128, 1, 4, 2, 8>(a, grid, s);
        case 24: return launch_ring<DT, BT, 32, 256, 1, 4, 1, 6>(a, grid, s);
        case 25: return launch_ring<DT, BT, 64, 256, 1, 4, 1, 6>(a, grid, s);
        case 28: return launch_ring<DT, BT, 32, 256, 1, 4, 2, 4>(a, grid, s);
        case 29: return launch_ring<DT, BT, 32, 128, 1, 4, 2, 6>(a, grid, s);
        case 30: return launch_ring<DT, BT, 64, 128, 1, 4, 2, 5>(a, grid, s);
        case 31: return launch_ring<DT, BT, 128, 128, 2, 2, 2, 4>(a, grid, s);
        case 32: return launch_ring<DT, BT, 128, 128, 2, 2, 2, 8>(a, grid, s);
        case 33: return launch_ring<DT, BT, 128, 128, 2, 4, 2, 8>(a, grid, s);
        case 34: return launch_ring<DT, BT, 256, 256, 4, 2, 2, 5>(a, grid, s);
        case 35: return launch_ring<DT, BT, 256, 256, 2, 4, 2, 5>(a, grid, s);
        case 36: return launch_ring<DT, BT, 256, 256, 2, 2, 1, 5>(a, grid, s);
        case 37: return launch_ring<DT, BT, 128, 256, 2, 2, 2, 3>(a, grid, s);
        case 38: return launch_ring<DT, BT, 256, 128, 2, 2, 2, 3>(a, grid, s);
        case 39: return launch_ring<DT, BT, 128, 256, 1, 4, 2, 3>(a, grid, s);
        case 40: return launch_ring<DT, BT, 128, 256, 2, 4, 4, 3>(a, grid, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace gemm
