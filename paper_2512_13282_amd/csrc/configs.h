// configs.h -- the tile configurations compiled into the library.
//
// One table, read by the host-side selector (selector.cpp) and by the launch
// code (gemm_launch.hip and the launch_*.hip family units), which instantiates
// exactly these kernels.  Pure C++:
// no HIP headers, so the selector builds and tests on a machine without a GPU.
//
// Tiling levels (paper, Sec. 4.1: instruction tile r x s x t -> per-core kernel
// m_ct x k_ct x n_ct -> whole-array tile -> full GEMM): here the MFMA
// instruction tile -> the wave tile -> the workgroup macro-tile BM x BK x BN
// staged through LDS -> the grid of output tiles.  Each workgroup owns one
// output tile and reduces K in time with the accumulators held in registers
// (output-stationary, Sec. 4.2.1); split-K (several workgroups per tile, each
// on a K slice) is only used where too few output tiles exist to fill the GPU.
#pragma once

#include <stdint.h>

namespace gemm {

enum Dtype : int32_t { DT_I8 = 0, DT_BF16 = 1 };

enum Family : int32_t { FAM_GENERIC = 0, FAM_MACRO = 1, FAM_SKINNY = 2, FAM_DIRECT = 3, FAM_RING = 4,
                        FAM_GEMV = 5 };

struct TileConfig {
    int32_t family;
    int32_t bm, bn;      // workgroup macro-tile (rows of C, cols of C)
    int32_t wm, wn;      // waves along M and N (wave tile = bm/wm x bn/wn)
    int32_t occupancy;   // workgroups resident per CU (LDS and register bound)
    int32_t stages;      // LDS stage buffers
    double  eff_i8;      // sustained fraction of the 2.4 GHz dense MFMA peak, int8
    double  eff_bf16;    // same, bf16 (measured on the 8192^3 GEMM, MI355X; ring_128x128_w4's
                         // int8 figure raised above its 8-slot twin's, which it beats on
                         // mid-size int8 shapes)
    int32_t col_major_b; // also compiled for B stored column-major (N x K)
    const char *name;
};

// K depth of one LDS stage is 128 bytes for both dtypes: 64 bf16 or 128 int8
// elements.  Every MFMA consumes 32 bytes of K per lane pair (bf16 32x32x16,
// int8 32x32x32), so a stage is 4 MFMA k-steps.
constexpr int32_t kStageKBytes = 128;

// The ring family walks K in 64-byte slots (two MFMA k-steps), `stages` of them
// resident in LDS at once.
constexpr int32_t kSlotKBytes = 64;

// Family GENERIC: alignment-agnostic element-wise loads (any lda/ldb/K/N).
// Family MACRO: 16-byte vector loads staged through registers (B transposed
// in registers); large tiles.
// Family SKINNY: same loaders, narrow M tile for M <= 64.
// Family GEMV: M = 1 only, vector-ALU matrix-vector kernels, one per B layout
// (col_major_b = 1 marks the column-major-only one); the efficiencies are the
// vector-ALU multiply-add rate as a fraction of the MFMA peak.
// Family DIRECT: both operands stream global -> LDS directly (buffer loads with
// an LDS destination); B's fragments come from LDS transpose reads, or, for B
// stored column-major, from 16-byte reads like A's.
constexpr TileConfig kConfigs[] = {
    // family       bm   bn  wm wn occ stages eff_i8 eff_bf16 colB name
    {FAM_GENERIC,   64,  64, 2, 2, 2, 2, 0.05, 0.07, 1, "generic_64x64_w4"},
    {FAM_GENERIC,  128, 128, 2, 2, 1, 2, 0.07, 0.10, 1, "generic_128x128_w4"},
    {FAM_MACRO,    256, 256, 2, 2, 1, 2, 0.33, 0.41, 0, "macro_256x256_w4"},
    {FAM_MACRO,    128, 256, 2, 2, 1, 2, 0.27, 0.33, 0, "macro_128x256_w4"},
    {FAM_MACRO,    256, 128, 2, 2, 1, 2, 0.31, 0.33, 0, "macro_256x128_w4"},
    {FAM_MACRO,    128, 128, 2, 2, 2, 2, 0.30, 0.35, 0, "macro_128x128_w4"},
    {FAM_SKINNY,    32, 256, 1, 4, 2, 2, 0.17, 0.22, 0, "skinny_32x256_w4"},
    {FAM_SKINNY,    64, 256, 1, 4, 2, 2, 0.25, 0.32, 0, "skinny_64x256_w4"},
    {FAM_DIRECT,   256, 256, 2, 2, 1, 2, 0.40, 0.44, 1, "direct_256x256_w4"},
    {FAM_DIRECT,   128, 256, 2, 2, 1, 2, 0.39, 0.34, 1, "direct_128x256_w4"},
    {FAM_DIRECT,   256, 256, 2, 4, 1, 2, 0.44, 0.51, 1, "direct_256x256_w8"},
    {FAM_DIRECT,   256, 256, 4, 2, 1, 2, 0.45, 0.51, 1, "direct_256x256_w8t"},
    {FAM_DIRECT,   128, 256, 2, 4, 1, 2, 0.42, 0.36, 1, "direct_128x256_w8"},
    {FAM_DIRECT,   256, 256, 2, 4, 1, 2, 0.30, 0.30, 0, "pingpong_256x256_w8"},
    {FAM_SKINNY,    32, 256, 1, 4, 1, 4, 0.10, 0.12, 0, "stream_32x256_s4"},
    {FAM_SKINNY,    64, 256, 1, 4, 1, 3, 0.15, 0.18, 0, "stream_64x256_s3"},
    {FAM_RING,     256, 256, 2, 4, 1, 4, 0.40, 0.45, 1, "ring_256x256_w8"},
    {FAM_RING,     256, 256, 4, 2, 1, 4, 0.40, 0.45, 1, "ring_256x256_w8t"},
    {FAM_RING,     128, 256, 2, 4, 1, 5, 0.38, 0.34, 1, "ring_128x256_w8"},
    {FAM_RING,     256, 256, 2, 2, 1, 4, 0.38, 0.42, 1, "ring_256x256_w4"},
    {FAM_RING,      32,  64, 1, 2, 2, 8, 0.10, 0.12, 1, "ring_32x64_w2"},
    {FAM_RING,      64,  64, 1, 2, 2, 8, 0.15, 0.18, 1, "ring_64x64_w2"},
    {FAM_RING,      32, 128, 1, 4, 1, 8, 0.12, 0.14, 1, "ring_32x128_w4"},
    {FAM_RING,      64, 128, 1, 4, 1, 8, 0.18, 0.20, 1, "ring_64x128_w4"},
    {FAM_RING,      32, 256, 1, 4, 1, 6, 0.15, 0.18, 1, "ring_32x256_w4"},
    {FAM_RING,      64, 256, 1, 4, 1, 6, 0.22, 0.26, 1, "ring_64x256_w4"},
    {FAM_GEMV,       1, 1024, 1, 4, 4, 1, 0.03, 0.06, 0, "gemv_1024"},
    {FAM_GEMV,       1,  16, 1, 4, 4, 1, 0.03, 0.06, 1, "gemv_bt_16"},
    {FAM_RING,      32, 256, 1, 4, 2, 4, 0.15, 0.18, 1, "ring_32x256_w4_r4"},
    {FAM_RING,      32, 128, 1, 4, 2, 6, 0.12, 0.14, 1, "ring_32x128_w4_r6"},
    {FAM_RING,      64, 128, 1, 4, 2, 5, 0.18, 0.20, 1, "ring_64x128_w4_r5"},
    {FAM_RING,     128, 128, 2, 2, 2, 4, 0.32, 0.34, 1, "ring_128x128_w4"},
    {FAM_RING,     128, 128, 2, 2, 1, 8, 0.30, 0.34, 1, "ring_128x128_w4_r8"},
    {FAM_RING,     128, 128, 2, 4, 1, 8, 0.30, 0.34, 1, "ring_128x128_w8"},
    {FAM_RING,     256, 256, 4, 2, 1, 5, 0.40, 0.45, 1, "ring_256x256_w8t_r5"},
    {FAM_RING,     256, 256, 2, 4, 1, 5, 0.40, 0.45, 1, "ring_256x256_w8_r5"},
    {FAM_RING,     256, 256, 2, 2, 1, 5, 0.38, 0.42, 1, "ring_256x256_w4_r5"},
    {FAM_RING,     128, 256, 2, 2, 2, 3, 0.36, 0.34, 1, "ring_128x256_w4_r3"},
    {FAM_RING,     256, 128, 2, 2, 2, 3, 0.36, 0.34, 1, "ring_256x128_w4_r3"},
    {FAM_RING,     128, 256, 1, 4, 2, 3, 0.36, 0.34, 1, "ring_128x256_w4c_r3"},
    {FAM_RING,     128, 256, 2, 4, 2, 3, 0.36, 0.34, 1, "ring_128x256_w8_r3"},
};
constexpr int32_t kNumConfigs = int32_t(sizeof(kConfigs) / sizeof(kConfigs[0]));

// LDS bytes of one workgroup: `stages` copies of an A stage (bm x 128 B) and a
// B stage (bn x 128 B).  The analog of the paper's L1 budget (Eq. 5) without
// the C term: the output tile lives in registers, not in LDS.
constexpr int64_t lds_bytes(const TileConfig &c) {
    if (c.family == FAM_GEMV) return c.col_major_b ? 4 * int64_t(c.bn) : 4 * 4 * int64_t(c.bn);
    return int64_t(c.stages) * (int64_t(c.bm) + int64_t(c.bn)) * (c.family == FAM_RING ? kSlotKBytes : kStageKBytes);
}

}  // namespace gemm
