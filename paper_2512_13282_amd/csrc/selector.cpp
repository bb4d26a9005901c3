// selector.cpp -- the paper's compute/memory balance model, transplanted.
//
// The paper picks its per-core tile by modelling compute time against data
// movement time and searching for the point where the two balance
// (Sec. 4.5.1, Eqs. 1-5; Sec. 4.5.2, Eqs. 6-10):
//   * off-chip reads of A scale as M*K*N*ty(A) / (width of the output tile in N)
//     and reads of B as M*K*N*ty(B) / (height in M) (Eqs. 6-7); C is written
//     once (Eq. 8);
//   * compute time is 2*M*K*N / (eff * peak) (Eq. 9), memory time is traffic /
//     bandwidth (Eq. 10), and the better tile is the one with the smaller
//     maximum of the two.
// On the GPU the same two terms decide between macro-tiles, with two terms
// the NPU does not have: wave quantization (output tiles are spread over 256
// CUs in whole rounds) and split-K partial traffic, which the paper avoids by
// never splitting K across cores (Sec. 4.2.1).  Split-K is therefore only
// chosen where the tile count alone cannot fill the chip.
#include "selector.h"
#include "launch.h"

#include <algorithm>
#include <cmath>

namespace gemm {

int32_t elem_bytes(int32_t dtype) { return dtype == DT_I8 ? 1 : 2; }

int32_t stage_k_elems(int32_t dtype) { return kStageKBytes / elem_bytes(dtype); }

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool vector_loads_ok(const Problem &p) {
    // 16-byte pieces of A rows and B rows must start 16-byte aligned and never
    // straddle the end of a row; buffer offsets are 32-bit, so a 256-row panel
    // of either operand must span less than 2 GiB.  Rows of A and of a
    // column-major B hold K elements, rows of a row-major B hold N.
    const int64_t e = elem_bytes(p.dtype);
    const int64_t max_row_bytes = int64_t(1) << 22;
    const int64_t b_row_elems = p.trans_b ? p.K : p.N;
    return (p.a_addr % 16 == 0) && (p.b_addr % 16 == 0) &&
           ((p.lda * e) % 16 == 0) && ((p.ldb * e) % 16 == 0) &&
           ((p.K * e) % 16 == 0) && ((b_row_elems * e) % 16 == 0) &&
           p.lda * e <= max_row_bytes && p.ldb * e <= max_row_bytes;
}

bool config_applicable(const Problem &p, int32_t cfg) {
    if (cfg < 0 || cfg >= kNumConfigs) return false;
    const TileConfig &c = kConfigs[cfg];
    if (p.trans_b && !c.col_major_b) return false;
    if (c.family == FAM_GEMV) return p.M == 1 && (c.col_major_b != 0) == (p.trans_b != 0) && vector_loads_ok(p);
    if (c.family == FAM_GENERIC) return true;
    return vector_loads_ok(p);
}

Plan evaluate(const Problem &p, int32_t cfg, int32_t split, const Chip &chip, int32_t reduce) {
    const TileConfig &c = kConfigs[cfg];
    const int64_t e = elem_bytes(p.dtype);
    const int64_t bk = stage_k_elems(p.dtype);
    Plan pl{};
    pl.config = cfg;
    pl.tiles_m = ceil_div(p.M, c.bm);
    pl.tiles_n = ceil_div(p.N, c.bn);
    const int64_t nkt = ceil_div(p.K, bk);  // K stages in total
    if (p.K == 0) {
        pl.split_k = 1;
        pl.k_chunk = 0;
    } else {
        int64_t s = std::max<int64_t>(1, std::min<int64_t>(split, nkt));
        pl.k_chunk = ceil_div(nkt, s) * bk;
        pl.split_k = int32_t(ceil_div(p.K, pl.k_chunk));
    }
    pl.grid = pl.tiles_m * pl.tiles_n * pl.split_k;

    // Split-K reduction (REDUCE_* in launch.h).  Last slice: the last slice of each
    // tile reads the tile's partials, sixteen slices per round trip of 256 threads x 4
    // columns, at the end of the kernel.  Separate: one more launch streaming the
    // partial planes.  Atomic (int8 only): a fill launch ahead of the GEMM, the partial
    // tiles added into C, no workspace; the model's choice for int8, where it costs the
    // separate reduction's one extra launch without its partial planes (measured on the
    // skinny shapes: it matches or beats both others).  Atomic with C zeroed by each
    // tile's first slice (ring and GEMV kernels): no fill launch; the int8 choice for
    // those kernels, 2-12 % faster than the fill on the skinny shapes.
    double red_us = 0.0;
    pl.reduce_in_kernel = REDUCE_SEPARATE;
    if (pl.split_k > 1) {
        // Measured on the skinny bf16 shapes: the last-slice reduction beats the separate
        // kernel by 1-2 us at M = 1 and loses by 3-7 us at M = 16 (10-40 us at M = 64):
        // beside its three dependent round trips it issues the tile's device-coherent
        // partial stores, which grow with the tile's valid rows, and one workgroup reads
        // every other slice's partial tile.  The separate kernel is priced as a launch.
        const int64_t rows = std::min<int64_t>(c.bm, p.M), cols = std::min<int64_t>(c.bn, p.N);
        const double in_kernel_us = 2.5 + 0.35 * double(rows) +
                                    double(pl.split_k - 1) * double(rows * cols) * 4.0 / chip.wg_cold_bytes_per_s * 1e6;
        const double separate_us = chip.launch_us;
        int32_t mode = reduce >= 0 ? reduce
                     : p.dtype == DT_I8 ? ((c.family == FAM_RING || c.family == FAM_GEMV) ? REDUCE_ATOMIC_FLAG
                                                                                       : REDUCE_ATOMIC)
                     : (in_kernel_us <= separate_us ? REDUCE_LAST_SLICE : REDUCE_SEPARATE);
        if ((mode == REDUCE_ATOMIC || mode == REDUCE_ATOMIC_FLAG) && p.dtype != DT_I8) mode = REDUCE_SEPARATE;
        if (mode == REDUCE_ATOMIC_FLAG && c.family != FAM_RING && c.family != FAM_GEMV) mode = REDUCE_ATOMIC;
        pl.reduce_in_kernel = mode;
        // atomic: the fill launch; atomic with slice 0's zeros: their round trip, growing
        // with the slices that add into the same lines of C
        red_us = mode == REDUCE_LAST_SLICE ? in_kernel_us
               : mode == REDUCE_ATOMIC_FLAG ? chip.round_trip_us * (1.0 + double(pl.split_k) / 8.0) : separate_us;
    }
    const bool partial_planes =
        pl.split_k > 1 && pl.reduce_in_kernel != REDUCE_ATOMIC && pl.reduce_in_kernel != REDUCE_ATOMIC_FLAG;
    pl.workspace_bytes = partial_planes ? int64_t(pl.split_k) * p.M * p.N * 4 : 0;

    // Compute: whole rounds of resident workgroups (wave quantization).
    const double ops_clk = p.dtype == DT_I8 ? chip.i8_ops_per_clk_cu : chip.bf16_ops_per_clk_cu;
    const double cu_rate = ops_clk * chip.clock_hz;                 // ops/s per CU
    const int64_t slots = int64_t(chip.cus) * c.occupancy;
    const int64_t rounds = ceil_div(pl.grid, slots);
    const double wg_ops = 2.0 * c.bm * c.bn * double(pl.k_chunk);
    const double eff = p.dtype == DT_I8 ? c.eff_i8 : c.eff_bf16;
    const double wg_s = wg_ops / (cu_rate * eff / c.occupancy);
    pl.t_comp_us = double(rounds) * wg_s * 1e6;

    // Memory: compulsory traffic at HBM speed; tile re-reads (Eqs. 6-7 analog)
    // mostly from L2/MALL; split-K partials written and read back once, or added
    // into C once after C is zeroed.  Row-major B read in row pieces narrower than a
    // 128-byte line (64 int8 columns) costs whole lines: each tile's piece is half of a
    // line whose other half a neighbouring workgroup, often on another XCD, fetches again
    // (measured: the unsplit 64-column int8 plans at M = 32-64 run 1.3-1.7x the
    // 128-column ones).
    const double b_line = (!p.trans_b && c.bn * e < 128) ? 128.0 / double(c.bn * e) : 1.0;
    const double a_bytes = double(p.M) * p.K * e, b_bytes = double(p.K) * p.N * e * b_line;
    const double c_bytes = double(p.M) * p.N * 4;
    const double a_reads = a_bytes * double(pl.tiles_n);
    const double b_reads = b_bytes * double(pl.tiles_m);
    const double ws = partial_planes ? 2.0 * double(pl.workspace_bytes)
                                     : (pl.split_k > 1 ? double(pl.split_k + 1) * p.M * p.N * 4 : 0.0);
    pl.traffic_bytes = a_reads + b_reads + c_bytes + ws;
    pl.t_mem_us = ((a_bytes + b_bytes + c_bytes + ws) / chip.hbm_bytes_per_s +
                   (a_reads + b_reads - a_bytes - b_bytes) / chip.reread_bytes_per_s) * 1e6;
    // With one tile row every workgroup streams a strip of B of its own from HBM, beside
    // its slice of A, at a rate one workgroup's loads in flight bound: too few workgroups
    // cannot reach the HBM rate (measured: 112 unsplit workgroups of 32 x 128 at M = 16
    // take 1.4x the time of 224 split ones).
    if (pl.tiles_m == 1 && p.K > 0) {
        const double wg_bytes = double(std::min<int64_t>(pl.k_chunk, p.K)) *
                                (double(std::min<int64_t>(c.bm, p.M)) + double(std::min<int64_t>(c.bn, p.N)) * b_line) * e;
        pl.t_mem_us = std::max(pl.t_mem_us, double(rounds) * wg_bytes / chip.wg_cold_bytes_per_s * 1e6);
    }

    // Each round of workgroups also pays its tiles' prologue and epilogue (measured at
    // 2048^3: 1.3 us of first loads and 2.5 us of C stores around an 8.5 us K loop); two
    // workgroups resident on a CU overlap each other's.
    pl.t_total_us = std::max(pl.t_comp_us, pl.t_mem_us) + double(rounds) * chip.tile_overhead_us / c.occupancy +
                    chip.launch_us + red_us;
    return pl;
}

// Plans measured fastest on the device for specific shapes (tune.py).
struct TunedPlan {
    int32_t dtype;
    int64_t M, N, K;
    int32_t config, split;
    int32_t reduce;      // -1: the model's choice
    int32_t trans_b;     // B layout the plan was measured with (1: column-major)
};
static const TunedPlan kTuned[] = {
#include "tuned_plans.inc"
    {-1, 0, 0, 0, 0, 0, -1, 0},   // sentinel
};

bool tuned_plan(const Problem &p, int32_t *config, int32_t *split, int32_t *reduce) {
    for (const TunedPlan &t : kTuned) {
        if (t.trans_b == p.trans_b && t.dtype == p.dtype && t.M == p.M && t.N == p.N && t.K == p.K &&
            t.config >= 0 && t.config < kNumConfigs && config_applicable(p, t.config)) {
            *config = t.config;
            *split = t.split;
            *reduce = t.reduce;
            return true;
        }
    }
    return false;
}

// A shape with M <= kNeighbourMaxM and no measured plan of its own borrows the plan
// measured for the nearest M at the same dtype, B layout, N and K.  Only plans whose
// tile covers the same number of rows of C at both sizes qualify, so the borrowed plan
// runs the same grid of tiles over the same reads of B as where it was measured (few
// rows: reading B is most of the work and does not depend on M; more: each tile's work
// barely changes); among them the nearest M on a log scale, the larger on a tie.  The split-K reduction is left to the model,
// whose price for it grows with the rows summed (at M = 1-4 the in-kernel sum wins over
// the separate kernel that a plan measured at M = 16 may have used).
bool neighbour_plan(const Problem &p, int32_t *config, int32_t *split, int32_t *reduce) {
    if (p.M < 1 || p.M > kNeighbourMaxM) return false;
    const TunedPlan *best = nullptr;
    double best_d = 0.0;
    for (const TunedPlan &t : kTuned) {
        if (t.dtype != p.dtype || t.trans_b != p.trans_b || t.N != p.N || t.K != p.K) continue;
        if (t.M < 1 || t.M > kNeighbourMaxM || t.config < 0 || t.config >= kNumConfigs) continue;
        const int64_t bm = kConfigs[t.config].bm;
        if ((t.M + bm - 1) / bm != (p.M + bm - 1) / bm || !config_applicable(p, t.config)) continue;
        const double d = std::fabs(std::log(double(t.M) / double(p.M)));
        if (!best || d < best_d - 1e-12 || (d <= best_d + 1e-12 && t.M > best->M)) {
            best = &t;
            best_d = d;
        }
    }
    if (!best) return false;
    *config = best->config;
    *split = best->split;
    *reduce = -1;
    return true;
}

bool select_plan(const Problem &p, Plan *out, int32_t forced_family, int32_t forced_config,
                 int32_t forced_split, const Chip &chip, int32_t forced_reduce) {
    static const int32_t kSplits[] = {1, 2, 3, 4, 6, 8, 12, 16, 24, 32, 48, 64};
    if (forced_family < 0 && forced_config < 0 && forced_split <= 0 && forced_reduce < 0) {
        int32_t cfg, split, reduce;
        if (tuned_plan(p, &cfg, &split, &reduce) || neighbour_plan(p, &cfg, &split, &reduce)) {
            *out = evaluate(p, cfg, split, chip, reduce);
            return true;
        }
    }
    bool found = false;
    Plan best{};
    for (int32_t cfg = 0; cfg < kNumConfigs; ++cfg) {
        if (forced_config >= 0 && cfg != forced_config) continue;
        if (forced_family >= 0 && kConfigs[cfg].family != forced_family) continue;
        if (!config_applicable(p, cfg)) continue;
        // The generic family only runs when nothing vectorised applies, or when forced.
        if (forced_family < 0 && forced_config < 0 && kConfigs[cfg].family == FAM_GENERIC &&
            vector_loads_ok(p))
            continue;
        for (int32_t s : kSplits) {
            if (forced_split > 0 && s != 1) break;
            const int32_t split = forced_split > 0 ? forced_split : s;
            Plan pl = evaluate(p, cfg, split, chip, forced_reduce);
            if (forced_split <= 0 && pl.split_k != split) continue;   // duplicate of a smaller split
            // Ties (memory-bound shapes, where every tile of one size moves the same
            // bytes) go to the plan with the shorter compute time: the faster kernel.
            const bool tie = found && std::abs(pl.t_total_us - best.t_total_us) <= 1e-9 * best.t_total_us;
            if (!found || (!tie && pl.t_total_us < best.t_total_us) ||
                (tie && pl.t_comp_us < best.t_comp_us * (1.0 - 1e-9))) {
                best = pl;
                found = true;
            }
        }
    }
    if (found) *out = best;
    return found;
}

}  // namespace gemm
