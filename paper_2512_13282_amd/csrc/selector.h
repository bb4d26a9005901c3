// selector.h -- shape-driven choice of kernel, tile and split-K (host only).
#pragma once

#include <stdint.h>

#include "configs.h"

namespace gemm {

struct Problem {
    int32_t dtype;
    int64_t M, N, K;
    int64_t lda, ldb, ldc;
    uintptr_t a_addr, b_addr, c_addr;
    int32_t trans_b = 0;   // 1: B stored column-major (N x K, row stride ldb)
};

struct Plan {
    int32_t config;      // index into kConfigs
    int32_t split_k;     // >= 1
    int32_t reduce_in_kernel;  // split-K reduction: REDUCE_SEPARATE, REDUCE_LAST_SLICE,
                               // REDUCE_ATOMIC or REDUCE_ATOMIC_FLAG (launch.h)
    int64_t k_chunk;     // K elements per slice (multiple of the stage depth)
    int64_t tiles_m, tiles_n;
    int64_t grid;
    int64_t workspace_bytes;
    double  traffic_bytes, t_comp_us, t_mem_us, t_total_us;
};

// Chip constants used by the model (AMD's published MI355X figures).
struct Chip {
    int32_t cus = 256;              // 8 XCDs x 32 CUs
    double  clock_hz = 2.4e9;
    double  i8_ops_per_clk_cu = 8192.0;   // dense int8 MFMA
    double  bf16_ops_per_clk_cu = 4096.0; // dense bf16 MFMA
    double  hbm_bytes_per_s = 4.0e12;     // sustained cold-HBM streaming rate the kernels reach
    double  reread_bytes_per_s = 16.0e12; // A/B tile re-reads mostly served by L2/MALL
    double  wg_cold_bytes_per_s = 30.0e9; // one workgroup streaming its own strip of B from HBM
                                          // (measured 26-38 GB/s: its loads in flight over the latency)
    double  launch_us = 5.0;              // per kernel launch on the stream
    double  round_trip_us = 1.5;          // one dependent global-memory round trip of a workgroup
    double  tile_overhead_us = 2.0;       // per round of workgroups: the first loads' latency and
                                          // the C stores, which the K loop does not hide
};

int32_t elem_bytes(int32_t dtype);
int32_t stage_k_elems(int32_t dtype);    // K elements per 128-byte LDS stage

// Whether the 16-byte vector loaders (MACRO / SKINNY) may run this problem.
bool vector_loads_ok(const Problem &p);

// Whether config `cfg` can run problem `p` at all.
bool config_applicable(const Problem &p, int32_t cfg);

// Evaluates the model for one (config, split) candidate.  reduce < 0 picks the
// cheaper split-K reduction by the model, 0 / 1 pins it.
Plan evaluate(const Problem &p, int32_t cfg, int32_t split, const Chip &chip = Chip(),
              int32_t reduce = -1);

// A plan measured fastest on the device for exactly this shape, if any applies
// (*reduce = -1 when the measurement left the reduction to the model).
bool tuned_plan(const Problem &p, int32_t *config, int32_t *split, int32_t *reduce);

// For M <= kNeighbourMaxM without a plan of its own: the plan measured for the nearest
// tuned M (same dtype, B layout, N and K, same number of tile rows), if any, with
// *reduce = -1 (the model picks the reduction).
constexpr int64_t kNeighbourMaxM = 2048;
bool neighbour_plan(const Problem &p, int32_t *config, int32_t *split, int32_t *reduce);

// Best plan: a tuned plan for this exact shape if one applies, else a neighbour's
// tuned plan (M <= kNeighbourMaxM), else the model's.  forced_family < 0 means any family; forced_config
// >= 0 pins the configuration; forced_split > 0 pins the split factor.
// Returns false if nothing applicable exists (only possible when forced).
// forced_reduce >= 0 pins the split-K reduction (0 separate kernel, 1 in-kernel).
bool select_plan(const Problem &p, Plan *out, int32_t forced_family = -1,
                 int32_t forced_config = -1, int32_t forced_split = 0,
                 const Chip &chip = Chip(), int32_t forced_reduce = -1);

}  // namespace gemm
