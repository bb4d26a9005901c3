/*
 * gemm_mi355x.h -- C ABI of the MI355X (gfx950) dense GEMM library.
 *
 * Operation (paper, Sec. 4.1 "Multi-Level Tiling Method"): an M x K x N GEMM,
 * C = A . B, with A the M x K input (typically activations), B the K x N input
 * (typically weights) and C the M x N output.  Matrices stay in standard
 * row-major order in memory with no pre-tiling (Sec. 1 and Sec. 4.3: the
 * layout transformation into the tiled order the compute units need happens
 * on the fly, inside the kernels), and arbitrary dimensions are supported
 * (Sec. 5.3.1, where the paper zero-pads; here ragged tiles are masked, which
 * gives the same result).
 *
 *   C[i*ldc + j] = sum_{k<K} A[i*lda + k] * B[k*ldb + j],  0 <= i < M, 0 <= j < N
 *
 * The result OVERWRITES C (no alpha/beta; the accumulator starts at zero as
 * in the paper's output-stationary kernel, Sec. 4.2.1).  Elements of C outside
 * the M x N window (row padding beyond N) are never touched.
 *
 * Layout: A, B and C are row-major; lda, ldb, ldc are row strides in ELEMENTS.
 * The *_bt entry points take B stored column-major instead, i.e. as its
 * transpose Bt (N x K, row-major, row stride ldbt >= K), the layout of a
 * PyTorch Linear weight; the paper's preferred and fastest layout (Sec. 4.3,
 * where B in column-major order lets the cores read K-contiguous blocks).
 *
 * Ownership: A, B and C are caller-owned DEVICE pointers on the current HIP
 * device, valid until the work queued on `stream` has completed.  The library
 * keeps no reference after a call returns.  The only memory it allocates is
 * the split-K workspace (partial sums and per-tile arrival counters), one per
 * (device, stream): taken with hipMallocAsync on `stream` at the first split-K
 * call that needs it, grown the same way (the old buffer released with
 * hipFreeAsync on that stream), and kept until the process ends.  Calls on one
 * stream run in order and share it safely; calls on different streams use
 * different workspaces.  A stream handle that is destroyed and re-created with
 * the same value while work of the old one is still running must not be used.
 *
 * Execution: every GEMM call is asynchronous on `stream` (a hipStream_t passed
 * as void*; NULL = the null stream) and never synchronizes the device.
 *
 * Errors: every entry point returns an int status (gemm_status_t) and never
 * throws or aborts.  Argument checks run on the host BEFORE any HIP call:
 *   GEMM_ERR_INVALID_VALUE  M, N or K < 0; lda < K (M, K > 0); ldb < N (K, N > 0;
 *                           ldbt < K for the *_bt calls);
 *                           ldc < N (M, N > 0); a NULL pointer whose operand is
 *                           non-empty; C overlapping A or B in memory.
 *   GEMM_ERR_UNSUPPORTED    a forced plan (gemm_force_plan) that cannot run the
 *                           given shape / alignment.
 *   GEMM_ERR_NO_MEMORY      the split-K workspace could not be allocated (nothing
 *                           is queued; a later call allocates afresh).  Setting
 *                           GEMM_MI355X_TEST_FAIL_WORKSPACE=1 in the environment
 *                           makes every workspace allocation fail this way (a
 *                           test hook; read at each allocation).
 *   GEMM_ERR_HIP            a HIP launch/runtime error.
 *   GEMM_ERR_SCRATCH_LIMIT  (gemm_bf16_f32_noalloc only) the plan's split-K
 *                           partials exceed its fixed scratch.
 * M == 0 or N == 0 is a successful no-op.  K == 0 writes zeros (empty sum).
 * Pointers or strides that are not 16-byte aligned are accepted and routed to
 * an alignment-agnostic kernel (slower, same result).
 */
#ifndef GEMM_MI355X_H
#define GEMM_MI355X_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    GEMM_OK = 0,
    GEMM_ERR_INVALID_VALUE = -1,
    GEMM_ERR_UNSUPPORTED = -2,
    GEMM_ERR_HIP = -3,
    GEMM_ERR_NO_MEMORY = -4,
    GEMM_ERR_SCRATCH_LIMIT = -5  /* gemm_bf16_f32_noalloc: plan needs more than its scratch */
} gemm_status_t;

typedef enum {
    GEMM_DTYPE_I8_I32 = 0,   /* int8 inputs, exact int32 accumulate and output */
    GEMM_DTYPE_BF16_F32 = 1  /* bf16 inputs, fp32 accumulate and output         */
} gemm_dtype_t;

/* Kernel families the selector chooses between (gemm_plan_info.kernel). */
typedef enum {
    GEMM_KERNEL_AUTO = -1,   /* gemm_force_plan: let the selector decide       */
    GEMM_KERNEL_GENERIC = 0, /* any alignment; element-wise masked loads       */
    GEMM_KERNEL_MACRO = 1,   /* 16-byte vector loads, large LDS macro-tiles    */
    GEMM_KERNEL_SKINNY = 2,  /* small M: narrow M tile, wide N, split-K        */
    GEMM_KERNEL_DIRECT = 3,  /* global -> LDS direct loads, LDS transpose reads */
    GEMM_KERNEL_RING = 4,    /* as DIRECT, 64-byte K slots in a deeper LDS ring */
    GEMM_KERNEL_GEMV = 5     /* M = 1: matrix-vector kernels on the vector ALUs */
} gemm_kernel_t;

/* The selector's choice for one call (filled by gemm_plan). */
typedef struct gemm_plan_info {
    int32_t kernel;          /* gemm_kernel_t                                  */
    int32_t config;          /* index of the tile configuration in the family  */
    int32_t bm, bn, bk;      /* workgroup macro-tile (bk in elements)          */
    int32_t waves;           /* wavefronts per workgroup                       */
    int32_t mfma_m, mfma_n, mfma_k;  /* MFMA instruction shape (0: none, GEMV) */
    int32_t split_k;         /* K slices (1 = no split)                        */
    int32_t reduce_in_kernel;/* split-K reduction, GEMM_REDUCE_*: partials summed
                                by a second kernel (0), by the last slice of
                                each tile inside the GEMM kernel (1), or added
                                into C with device atomics, C zeroed by a fill
                                kernel first (2) or by each tile's first slice
                                inside the GEMM kernel (3) (2 and 3: int8 only;
                                the narrowed-output calls of such a plan use 0);
                                0 when split_k == 1                           */
    int64_t k_chunk;         /* K elements per slice                           */
    int64_t grid;            /* workgroups of the main kernel                  */
    int64_t lds_bytes;       /* LDS per workgroup                              */
    int64_t workspace_bytes; /* split-K partials (0 when split_k == 1)         */
    double  model_traffic_bytes; /* modelled global traffic: A and B re-reads
                                    (A ~ MNK/BN, B ~ MNK/BM), C, partials      */
    double  model_t_comp_us; /* modelled MFMA time at the plan's efficiency    */
    double  model_t_mem_us;  /* modelled memory time (sustained HBM rate, L2 re-reads) */
    int32_t source;          /* where the plan came from: GEMM_PLAN_FROM_*      */
    char    name[48];        /* human-readable kernel/config name              */
} gemm_plan_info;

/* Where a plan came from (gemm_plan_info.source). */
enum {
    GEMM_PLAN_FROM_MODEL = 0,     /* the balance model (no measured plan applies)           */
    GEMM_PLAN_FROM_TABLE = 1,     /* the compiled table of measured plans, this exact shape */
    GEMM_PLAN_FROM_NEIGHBOUR = 2, /* the table's plan for the nearest M at this N, K (same
                                     number of tile rows; M <= 2048)                        */
    GEMM_PLAN_FROM_FILE = 3,      /* a plan loaded by gemm_load_plans / GEMM_MI355X_PLANS   */
    GEMM_PLAN_FROM_FORCED = 4     /* gemm_force_plan / gemm_force_reduce                    */
};

/* Split-K reductions (gemm_plan_info.reduce_in_kernel, gemm_force_reduce). */
enum {
    GEMM_REDUCE_SEPARATE = 0,   /* a second kernel sums the slices' partial planes      */
    GEMM_REDUCE_LAST_SLICE = 1, /* the slice of each tile that finishes last sums them  */
    GEMM_REDUCE_ATOMIC = 2,     /* int8, int32 output: C zeroed, then every slice adds
                                   its partial tile into C with device atomics          */
    GEMM_REDUCE_ATOMIC_FLAG = 3 /* as 2, but no fill kernel: the first K slice of each
                                   tile zeroes it, and the others wait for its signal
                                   before adding (RING and GEMV kernels; others use 2) */
};

/* Test and benchmark hook: force the split-K reduction for every later call of
 * `dtype` (a GEMM_REDUCE_* value, or -1 = the selector's choice).  The first two
 * sum the K slices in the same fixed order, so fp32 results do not depend on the
 * choice; the atomic one adds int32 partials in whatever order they arrive, which
 * modulo 2^32 gives the same bits.  A bf16 plan asked for an atomic reduction
 * uses the separate one, as do the int8 -> int8 / int16 calls.  Not thread-safe
 * with respect to concurrent GEMM calls.  Returns GEMM_ERR_INVALID_VALUE for an
 * unknown dtype or mode. */
int gemm_force_reduce(int dtype, int mode);

/* int8 x int8 -> int32.  Exact whenever every true sum fits in int32, which is
 * guaranteed for K <= 131071 (|a*b| <= 2^14); beyond that results wrap modulo
 * 2^32 as the hardware accumulator does. */
int gemm_i8_i32(int64_t M, int64_t N, int64_t K,
                const int8_t *A, int64_t lda,
                const int8_t *B, int64_t ldb,
                int32_t *C, int64_t ldc, void *stream);

/* bf16 x bf16 -> fp32.  A and B hold raw bf16 bit patterns (uint16_t);
 * products are exact and are accumulated in fp32 (order unspecified; split-K
 * partials are summed in a fixed slice order, so results are run-to-run
 * reproducible for a given plan). */
int gemm_bf16_f32(int64_t M, int64_t N, int64_t K,
                  const uint16_t *A, int64_t lda,
                  const uint16_t *B, int64_t ldb,
                  float *C, int64_t ldc, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): gemm_bf16_f32 with the
 * same arguments, plan and result (bit for bit: the same kernels sum in the same
 * order), except that a split-K plan keeps its partial sums and per-tile arrival
 * counters in a fixed 16 MiB array of device memory that the library holds for
 * each GPU it runs on until the process ends (64 KiB of counters, the rest for
 * partials: split_k * M * N * 4 bytes must fit in 16 MiB - 64 KiB).  It never
 * calls hipMalloc, hipFree or an allocating library routine; the counters are
 * cleared by a fill kernel on `stream` at each split-K call.  A plan whose
 * partials do not fit returns GEMM_ERR_SCRATCH_LIMIT before anything is queued.
 * Every call on one GPU shares that GPU's array: calls that overlap in time on
 * one GPU (different streams, or host threads) race on it and must not be
 * issued; calls queued in order on one stream are safe.  Other errors as
 * gemm_bf16_f32. */
int gemm_bf16_f32_noalloc(int64_t M, int64_t N, int64_t K,
                          const uint16_t *A, int64_t lda,
                          const uint16_t *B, int64_t ldb,
                          float *C, int64_t ldc, void *stream);

/* C = A . Bt^T with B stored column-major: C[i*ldc + j] = sum_k A[i*lda + k] *
 * Bt[j*ldbt + k].  Same results, ownership, errors and execution as
 * gemm_i8_i32 / gemm_bf16_f32 (the int8 result is exact, bf16 products are
 * exact with fp32 accumulation). */
int gemm_i8_i32_bt(int64_t M, int64_t N, int64_t K,
                   const int8_t *A, int64_t lda,
                   const int8_t *Bt, int64_t ldbt,
                   int32_t *C, int64_t ldc, void *stream);
int gemm_bf16_f32_bt(int64_t M, int64_t N, int64_t K,
                     const uint16_t *A, int64_t lda,
                     const uint16_t *Bt, int64_t ldbt,
                     float *C, int64_t ldc, void *stream);

/* ---- Reduced-precision outputs ---------------------------------------------
 * The same GEMMs with the output narrowed, the precisions the paper also
 * reports (int8 -> int16 and int8 -> int8, and bf16 -> bf16; Sec. 5.1 and
 * Sec. 5.2.3), which states no rounding or requantisation rule.  The rules here:
 *
 *   gemm_i8_i8 / gemm_i8_i16 : the exact int32 result (wrapping as gemm_i8_i32
 *       documents) divided by 2^shift, rounded to the nearest integer with ties
 *       to even, then saturated to [-128, 127] / [-32768, 32767]; 0 <= shift <= 31.
 *   gemm_bf16_bf16 : the fp32 result of gemm_bf16_f32 rounded to the nearest
 *       bf16, ties to even (raw bf16 bit patterns in C).
 *
 * C is int8_t / int16_t / uint16_t with row stride ldc in ELEMENTS of that type
 * and must be aligned to its element size.  Plans, ownership, workspace,
 * execution and errors are those of the int32 / fp32 calls (the plan does not
 * depend on the output type); a shift outside [0, 31] is GEMM_ERR_INVALID_VALUE.
 * The *_bt forms take B stored column-major (Bt, N x K) as above. */
int gemm_i8_i8(int64_t M, int64_t N, int64_t K,
               const int8_t *A, int64_t lda,
               const int8_t *B, int64_t ldb,
               int8_t *C, int64_t ldc, int shift, void *stream);
int gemm_i8_i16(int64_t M, int64_t N, int64_t K,
                const int8_t *A, int64_t lda,
                const int8_t *B, int64_t ldb,
                int16_t *C, int64_t ldc, int shift, void *stream);
int gemm_bf16_bf16(int64_t M, int64_t N, int64_t K,
                   const uint16_t *A, int64_t lda,
                   const uint16_t *B, int64_t ldb,
                   uint16_t *C, int64_t ldc, void *stream);
int gemm_i8_i8_bt(int64_t M, int64_t N, int64_t K,
                  const int8_t *A, int64_t lda,
                  const int8_t *Bt, int64_t ldbt,
                  int8_t *C, int64_t ldc, int shift, void *stream);
int gemm_i8_i16_bt(int64_t M, int64_t N, int64_t K,
                   const int8_t *A, int64_t lda,
                   const int8_t *Bt, int64_t ldbt,
                   int16_t *C, int64_t ldc, int shift, void *stream);
int gemm_bf16_bf16_bt(int64_t M, int64_t N, int64_t K,
                      const uint16_t *A, int64_t lda,
                      const uint16_t *Bt, int64_t ldbt,
                      uint16_t *C, int64_t ldc, void *stream);

/* Pure host: the plan a GEMM call with these arguments would use (alignment
 * is taken from the three addresses, which are never dereferenced).
 * Returns GEMM_OK, GEMM_ERR_INVALID_VALUE or GEMM_ERR_UNSUPPORTED. */
int gemm_plan(int dtype, int64_t M, int64_t N, int64_t K,
              int64_t lda, int64_t ldb, int64_t ldc,
              uintptr_t a_addr, uintptr_t b_addr, uintptr_t c_addr,
              gemm_plan_info *out);

/* The same for the column-major-B calls (gemm_i8_i32_bt / gemm_bf16_f32_bt). */
int gemm_plan_bt(int dtype, int64_t M, int64_t N, int64_t K,
                 int64_t lda, int64_t ldbt, int64_t ldc,
                 uintptr_t a_addr, uintptr_t bt_addr, uintptr_t c_addr,
                 gemm_plan_info *out);

/* Test and benchmark hook: force the kernel family, tile configuration
 * (-1 = selector's choice within the family) and split-K factor (0 = the
 * selector's) for every later call of `dtype` in this process, or restore
 * automatic selection with kernel = GEMM_KERNEL_AUTO.  Not thread-safe with
 * respect to concurrent GEMM calls.  Returns GEMM_ERR_INVALID_VALUE for an
 * unknown kernel/config or a split factor < 0. */
int gemm_force_plan(int dtype, int kernel, int config, int split_k);

/* Measured plans loaded at run time: the on-device measurement step of the
 * paper's tiling search (Sec. 4.5.2) without rebuilding the library.  `path`
 * names a text file with one plan per line, eight decimal integers separated by
 * blanks -- dtype M N K config split_k reduce trans_b -- the fields of the
 * compiled plan table (reduce: a GEMM_REDUCE_* value, or -1 for the selector's
 * choice; trans_b: 1 for the *_bt calls); '#' starts a comment that runs to the
 * end of the line; a line holds at most 510 characters.  `python -m paper_2512_13282_amd.tune --plans-out FILE`
 * writes this format.  For exactly those shapes and B layouts the loaded plans
 * take precedence over the compiled table and the model, in this process; a
 * call whose operands the plan's configuration cannot run (alignment) uses the
 * selector's plan as before.  A later line, or a later load, for the same shape
 * replaces an earlier one.  The environment variable GEMM_MI355X_PLANS, if set,
 * names a file loaded the same way before the first plan is chosen (a file that
 * does not load is reported once on stderr and ignored).  The path is only read
 * during the call.  Not thread-safe with respect to concurrent GEMM calls.
 * Returns GEMM_OK, or GEMM_ERR_INVALID_VALUE (NULL path, unreadable file, a
 * malformed or out-of-range line: then nothing is loaded). */
int gemm_load_plans(const char *path);

/* Drops every plan loaded by gemm_load_plans or GEMM_MI355X_PLANS.  Returns GEMM_OK. */
int gemm_clear_plans(void);

/* Frees the split-K workspaces the library holds (every device and stream).
 * Synchronizes each device that holds one first, so it must not be called while
 * another thread is issuing GEMM calls; later split-K calls allocate afresh.
 * Returns GEMM_OK, or GEMM_ERR_HIP if a synchronization or free failed. */
int gemm_release_workspace(void);

/* ---- Measurement aid (not part of the GEMM) ------------------------------
 * gemm_probe_mfma runs one workgroup of 8 waves per compute unit that issues
 * only the GEMM's 32x32 MFMA instructions (int8 32x32x32 or bf16 32x32x16,
 * chosen by `dtype`) for `iters` iterations of 32 MFMAs per wave, on operands
 * held in registers: random data shaped like the GEMM inputs (int8 uniform
 * bytes, bf16 approximately N(0,1)) when `random_operands` is non-zero,
 * constants otherwise.  No memory traffic occurs inside the loop, so ops per
 * launch divided by the launch's duration is the MFMA ceiling at the clock the
 * chip sustains under that load; the MI355X clock falls well below its maximum
 * when the multipliers see random data.
 *
 * `clocks` (device, 2 * workgroups int64) receives per workgroup the
 * shader-clock cycles and the constant-rate wall-clock ticks spent in the
 * loop; their ratio times wall_clock_hz is the clock the loop ran at.  `sink`
 * (device, workgroups * threads_per_workgroup uint32) receives values that keep
 * the results live.  With clocks == sink == NULL only `info` is filled.
 * Asynchronous on `stream`.  Returns GEMM_OK, GEMM_ERR_INVALID_VALUE (bad dtype,
 * iters < 1, info NULL, only one of the buffers given) or GEMM_ERR_HIP. */
typedef struct gemm_probe_info {
    int64_t workgroups;            /* one per compute unit                    */
    int64_t threads_per_workgroup;
    double  ops_per_launch;        /* 2 * multiply-adds of all MFMAs          */
    double  wall_clock_hz;         /* rate of the wall-clock ticks in clocks  */
} gemm_probe_info;

int gemm_probe_mfma(int dtype, int random_operands, int32_t iters, int64_t *clocks,
                    unsigned *sink, gemm_probe_info *info, void *stream);

/* ---- Measurement aid (not part of the GEMM) ------------------------------
 * gemm_probe_read reads `bytes` bytes of device memory at `src` once (16 bytes per
 * lane per load, grid-stride over the whole range, 8 workgroups of 256 threads per
 * compute unit) and writes one value per thread to `sink` so that no load is
 * skipped: bytes / duration is what a plain read of that range reaches, the
 * reference for the memory-bound (skinny) GEMMs.  `src` and `bytes` must be
 * multiples of 16; `sink` (device, uint32, `sink_elems` elements) must hold one
 * value per thread: 2048 per compute unit.  Asynchronous on `stream`.  Returns
 * GEMM_OK, GEMM_ERR_INVALID_VALUE (misaligned or negative size, NULL source with
 * bytes > 0, sink NULL or too small) or GEMM_ERR_HIP. */
int gemm_probe_read(const void *src, int64_t bytes, unsigned *sink, int64_t sink_elems, void *stream);

/* Static description of the error code. */
const char *gemm_status_string(int status);

/* Library version string. */
const char *gemm_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GEMM_MI355X_H */
