// kern_small.h -- narrow-M streaming kernels, the matrix-vector kernels (M = 1)
// and the separate split-K reduction.
#pragma once

#include "gemm_common.h"

namespace gemm {

// ---------------------------------------------------------------------------
// Streaming kernel for small M (memory-bound shapes): BM = 32 or 64 rows, BN =
// 256 columns, 4 waves (each a BM x 64 sub-tile), and an NS-deep ring of LDS
// stages so that NS - 1 stages of B stream in while one is consumed.  Same
// LDS layouts, swizzles and fragment reads as gemm_lds_kernel.  Each
// iteration waits only until its own stage has landed (vmcnt counts the loads
// of the younger stages still in flight), then one barrier publishes it and
// retires the buffer the next load overwrites.  Loads of stages past the end
// of the slice are still issued (zero-size resource: they return zero without
// touching memory) so that every iteration counts the same loads.
// ---------------------------------------------------------------------------

template <int DT, int BM, int NS>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
void gemm_stream_kernel(KernelArgs args) {
    using acc_vec = typename Types<DT>::acc_vec;
    using out_t = typename Types<DT>::out_t;
    constexpr int BN = 256, WAVES = 4;
    constexpr int E = Types<DT>::E;
    constexpr int VECE = 16 / E;
    constexpr int BK = kStageKBytes / E;
    constexpr int TM = BM / 32, TN = 2;                    // wave tile BM x 64
    constexpr int A_STAGE = BM * kStageKBytes;
    constexpr int B_PITCH = BN * E;
    constexpr int B_STAGE = BK * B_PITCH;
    constexpr int A_INSTR = A_STAGE / 1024 / WAVES;        // 1 (BM 32) or 2 (BM 64)
    constexpr int B_INSTR = B_STAGE / 1024 / WAVES;        // 8
    constexpr int LPS = A_INSTR + B_INSTR;                 // loads per wave per stage
    constexpr int B_ROWS_PER_KB = 1024 / B_PITCH;
    constexpr int B_CPR = B_PITCH / 16;
    static_assert(A_INSTR >= 1 && A_INSTR * 1024 * WAVES == A_STAGE, "A stage split");
    static_assert((NS - 2) * LPS < 64, "outstanding loads must fit vmcnt");

    __shared__ __attribute__((aligned(1024))) uint8_t a_lds[NS][A_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t b_lds[NS][B_STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    int tm, tn, slice;
    map_tile(args, tm, tn, slice);
    const int64_t M = args.M, N = args.N;
    const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;
    const int64_t k_begin = int64_t(slice) * args.k_chunk;
    int64_t k_end = k_begin + args.k_chunk;
    if (k_end > args.K) k_end = args.K;
    const int nk = k_end > k_begin ? int((k_end - k_begin + BK - 1) / BK) : 0;
    const int64_t lda_b = args.lda * E, ldb_b = args.ldb * E;

    const int64_t a_rows_valid = (M - m0) < BM ? (M - m0) : BM;
    const uint32_t a_bytes = uint32_t(a_rows_valid * lda_b);
    uint32_t a_voff[A_INSTR];
    int a_chunk[A_INSTR];
#pragma unroll
    for (int i = 0; i < A_INSTR; ++i) {
        const int row = (i * WAVES + wave) * 8 + (lane >> 3);
        const int c = (lane & 7) ^ ((row ^ (row >> 3)) & 7);
        a_chunk[i] = c;
        a_voff[i] = uint32_t(row * lda_b + c * 16);
    }
    uint32_t b_voff[B_INSTR];
#pragma unroll
    for (int i = 0; i < B_INSTR; ++i) {
        const int row = (i * WAVES + wave) * B_ROWS_PER_KB + lane / B_CPR;
        const int c = (lane % B_CPR) ^ bswz<DT>(row);
        b_voff[i] = (n0 + int64_t(c) * VECE < N) ? uint32_t(row * ldb_b + c * 16) : kOOB;
    }
    const uint8_t *const a_base = static_cast<const uint8_t *>(args.A) + (m0 * args.lda + k_begin) * E;
    const uint8_t *const b_base = static_cast<const uint8_t *>(args.B) + (k_begin * args.ldb + n0) * E;
    const int64_t k_len = k_end - k_begin;

    // The loads are the ring kernel's inline-assembly form, invisible to the compiler's
    // wait-count tracking (which cannot tell the stage buffers apart and would make every
    // fragment read wait for all loads in flight); the explicit vmcnt wait before each
    // barrier accounts for them.
    const uint32_t wave_u = uint32_t(__builtin_amdgcn_readfirstlane(wave));
    auto load_stage = [&](int kt, auto buf_c) {
        constexpr int BUF = decltype(buf_c)::value;
        const int64_t rem = k_len - int64_t(kt) * BK;
        const i32x4_t ra = ring_rsrc(a_base + int64_t(kt) * kStageKBytes, rem > 0 ? a_bytes : 0u);
        const int64_t rows = rem <= 0 ? 0 : (rem < BK ? rem : BK);
        const i32x4_t rb = ring_rsrc(b_base + int64_t(kt) * BK * ldb_b, uint32_t(rows * ldb_b));
#pragma unroll
        for (int i = 0; i < A_INSTR; ++i) {
            const uint32_t off = int64_t(a_chunk[i]) * VECE < rem ? a_voff[i] : kOOB;
            ring_load16(ra, lds_addr(&a_lds[BUF][0]) + (i * WAVES + wave_u) * 1024, off);
        }
#pragma unroll
        for (int i = 0; i < B_INSTR; ++i)
            ring_load16(rb, lds_addr(&b_lds[BUF][0]) + (i * WAVES + wave_u) * 1024, b_voff[i]);
    };

    const int frag_row = lane & 31;
    const int frag_half = lane >> 5;
    const int wcol0 = wave * 64;
    const int r0 = frag_row;
    const int f0 = (r0 ^ (r0 >> 3)) & 7;
    int a_fo[2][4];
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int st = 0; st < 4; ++st) a_fo[p][st] = r0 * kStageKBytes + 16 * ((2 * st + frag_half) ^ f0 ^ (4 * p));
    const int g16 = lane & 15, lgrp = lane >> 4;
    constexpr int TR_ROWS = DT == DT_BF16 ? 4 : 8;
    constexpr int KSTEP = 32 / E;
    const int tr_row = DT == DT_BF16 ? (g16 >> 2) : (g16 >> 1);
    const int tr_colb = (DT == DT_BF16 ? (g16 & 3) * 8 : (g16 & 1) * 8) + (lgrp & 1) * 16 * E;
    const int tr_khalf = (lgrp >> 1) * (KSTEP / 2);
    const int bz = bswz<DT>(tr_row);
    int b_fo[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int colb = (wcol0 + j * 32) * E + tr_colb;
        b_fo[j] = (tr_khalf + tr_row) * B_PITCH + (((colb >> 4) ^ bz) << 4) + (colb & 15);
    }

    acc_vec acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = acc_vec{};

    auto compute = [&](auto buf_c) {
        constexpr int BUF = decltype(buf_c)::value;
#pragma unroll
        for (int S = 0; S < 4; ++S) {
            u32x4_t fa[TM], fb[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                fa[i] = *reinterpret_cast<const u32x4_t *>(&a_lds[BUF][a_fo[i & 1][S] + 4096 * i]);
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const u32x2_t lo = lds_read_tr<DT>(&b_lds[BUF][b_fo[j] + (S * KSTEP) * B_PITCH]);
                const u32x2_t hi = lds_read_tr<DT>(&b_lds[BUF][b_fo[j] + (S * KSTEP + TR_ROWS) * B_PITCH]);
                fb[j] = u32x4_t{lo[0], lo[1], hi[0], hi[1]};
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = mfma32<DT>(fa[i], fb[j], acc[i][j]);
        }
    };

    // One iteration: stage kt is in buffer BUF; buffer (BUF + NS - 1) % NS receives stage kt + NS - 1.
    auto iteration = [&](int kt, auto buf_c) {
        constexpr int BUF = decltype(buf_c)::value;
        ring_barrier<(NS - 2) * LPS>();                    // own loads of stage kt have landed, then
                                                           // everyone's; buffer BUF-1 retired
        load_stage(kt + NS - 1, std::integral_constant<int, (BUF + NS - 1) % NS>{});
        compute(buf_c);
    };

    if (nk > 0) {
        static_for<0, NS - 1>([&](auto u) { load_stage(decltype(u)::value, u); });
        for (int kt = 0; kt < nk; kt += NS) {
            static_for<0, NS>([&](auto u) {
                if (kt + decltype(u)::value < nk) iteration(kt + decltype(u)::value, u);
            });
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // drain ring loads past the end before exit

    __shared__ int s_last;
    store_tile<DT, BM, BN, TM, TN>(args, acc, tm, tn, slice, m0, n0 + wcol0, lane, s_last);
}

// ---------------------------------------------------------------------------
// Matrix-vector kernels for M = 1 (the paper's stated future work: GEMV).  With
// one row of A there is no reuse to stage through LDS or to feed MFMAs with: the
// work is a single pass over B, bound by HBM bandwidth, so these kernels only
// keep enough 16-byte loads in flight and do the few multiply-adds per byte on
// the vector ALUs.
//
// Row-major B (gemv_kernel): a workgroup owns 1024 columns of one K slice; lane l
// of each wave holds 16 consecutive columns (16 int8 or 2 x 8 bf16 per row), the
// four waves take every fourth row of the slice, and their partial sums meet in
// LDS at the end.
//
// Column-major B (gemv_bt_kernel, B stored N x K): a workgroup owns 16 columns
// (rows of the stored matrix), four per wave; the lanes of a wave split K in
// 16-byte pieces and accumulate with the 4-way int8 dot-product instruction
// (bf16: widened to fp32, fused multiply-adds), then a butterfly over the wave
// sums the lanes.
//
// Split-K uses the partial planes and arrival counters of the tile kernels,
// with the same fixed slice order.
// ---------------------------------------------------------------------------
template <int DT>
using gemv_acc_t = typename std::conditional<DT == DT_I8, int32_t, float>::type;
template <int DT>
using gemv_sum_t = typename std::conditional<DT == DT_I8, uint32_t, float>::type;   // int32 wraps mod 2^32

// Writes `cols` results v[c] of columns n0 + c (one output row) for K slice
// `slice`: straight into C without split-K, else into the slice's partial plane;
// with the in-kernel reduction the workgroup arriving last for this column block
// sums the planes in slice order; with the atomic ones (int8, int32 output) every
// slice adds into C, zeroed beforehand (REDUCE_ATOMIC) or by slice 0, whose credit a
// later slice takes first (REDUCE_ATOMIC_FLAG; `seen` is thread 0's earlier read of
// the tile's counter).  Thread t handles c = t, t + 256, ...
template <int DT, int COLS>
__device__ __forceinline__ void gemv_store(const KernelArgs &args, const gemv_acc_t<DT> *v, int64_t n0,
                                           int tile, int slice, uint32_t seen) {
    using sum_t = gemv_sum_t<DT>;
    const int64_t N = args.N;
    sum_t *ws = static_cast<sum_t *>(args.workspace);
    const int t = int(threadIdx.x);
    if (args.split_k == 1) {
        for (int c = t; c < COLS; c += 256)
            if (n0 + c < N) write_c<DT>(args, n0 + c, v[c]);
        return;
    }
    if constexpr (DT == DT_I8) {
        if (args.reduce_in_kernel == REDUCE_ATOMIC || args.reduce_in_kernel == REDUCE_ATOMIC_FLAG) {
            if (args.reduce_in_kernel == REDUCE_ATOMIC_FLAG && slice != 0) flag_take_credit(args, tile, seen);
            for (int c = t; c < COLS; c += 256)
                if (n0 + c < N)
                    __hip_atomic_fetch_add(&static_cast<uint32_t *>(args.C)[n0 + c], uint32_t(v[c]), __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
            return;
        }
    }
    if (args.reduce_in_kernel == REDUCE_SEPARATE) {
        for (int c = t; c < COLS; c += 256)
            if (n0 + c < N) ws[int64_t(slice) * N + n0 + c] = sum_t(v[c]);
        return;
    }
    for (int c = t; c < COLS; c += 256)
        if (n0 + c < N) store_coherent(&ws[int64_t(slice) * N + n0 + c], sum_t(v[c]));
    __shared__ int s_last;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this thread's partial stores are complete
    __syncthreads();                                   // ... and every thread's
    if (t == 0) {
        const unsigned ticket = __hip_atomic_fetch_add(&args.counters[tile], 1u, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
        s_last = ticket == unsigned(args.split_k - 1);
    }
    __syncthreads();
    if (!s_last) return;
    // Sixteen slices per round trip: the loads of a batch are all issued before any is
    // used, then added in slice order.
    for (int c = t; c < COLS; c += 256) {
        if (n0 + c >= N) continue;
        sum_t s = sum_t(0);
        for (int p0 = 0; p0 < args.split_k; p0 += 16) {
            sum_t v16[16];
#pragma unroll
            for (int u = 0; u < 16; ++u)
                v16[u] = load_coherent(&ws[int64_t(p0 + u < args.split_k ? p0 + u : 0) * N + n0 + c]);
#pragma unroll
            for (int u = 0; u < 16; ++u)
                if (p0 + u < args.split_k) s = (p0 + u == 0) ? v16[u] : s + v16[u];
        }
        write_c<DT>(args, n0 + c, s);
    }
    if (t == 0) __hip_atomic_store(&args.counters[tile], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// 4 x 4 byte transpose: col[j] gets byte j of r0, r1, r2, r3 (in that order, low byte
// first).  Two rounds of byte permutes (v_perm_b32 picks bytes 0-3 from its second source
// and 4-7 from its first): pair rows 0/1 and 2/3 by even and odd byte, then merge.
__device__ __forceinline__ void transpose4x4_bytes(uint32_t r0, uint32_t r1, uint32_t r2, uint32_t r3,
                                                   uint32_t (&col)[4]) {
    const uint32_t t0 = __builtin_amdgcn_perm(r1, r0, 0x06020400u);   // r0.b0 r1.b0 r0.b2 r1.b2
    const uint32_t t1 = __builtin_amdgcn_perm(r1, r0, 0x07030501u);   // r0.b1 r1.b1 r0.b3 r1.b3
    const uint32_t t2 = __builtin_amdgcn_perm(r3, r2, 0x06020400u);
    const uint32_t t3 = __builtin_amdgcn_perm(r3, r2, 0x07030501u);
    col[0] = __builtin_amdgcn_perm(t2, t0, 0x05040100u);
    col[1] = __builtin_amdgcn_perm(t3, t1, 0x05040100u);
    col[2] = __builtin_amdgcn_perm(t2, t0, 0x07060302u);
    col[3] = __builtin_amdgcn_perm(t3, t1, 0x07060302u);
}

template <int DT>
__global__ __launch_bounds__(256) void gemv_kernel(KernelArgs args) {
    using acc_t = gemv_acc_t<DT>;
    constexpr int E = Types<DT>::E;
    constexpr int CB = 1024;                   // columns per workgroup
    constexpr int CPL = 16;                    // columns per lane
    constexpr int PIECES = CPL * E / 16;       // 16-byte pieces per lane and row (1 int8, 2 bf16)
    constexpr int U = 8 / PIECES;              // rows in flight per lane and iteration
    const int lane = int(threadIdx.x) & 63;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);

    int tm, tn, slice;
    map_tile(args, tm, tn, slice);
    (void)tm;
    const int64_t N = args.N;
    const int64_t n0 = int64_t(tn) * CB;
    const int64_t col = n0 + int64_t(lane) * CPL;
    const int64_t k_begin = int64_t(slice) * args.k_chunk;
    int64_t k_end = k_begin + args.k_chunk;
    if (k_end > args.K) k_end = args.K;
    // REDUCE_ATOMIC_FLAG: slice 0 zeroes its 1024 outputs first; the other slices read
    // the credit counter once halfway through their rows.
    const bool flag = DT == DT_I8 && args.split_k > 1 && args.reduce_in_kernel == REDUCE_ATOMIC_FLAG;
    if (flag && slice == 0) flag_zero_tile<1, CB, 256>(args, 0, n0, tn);
    bool poll_pending = flag && slice != 0;
    const int64_t k_poll = k_begin + (k_end - k_begin) / 2;
    uint32_t seen = 0u;
    // N * E is a multiple of 16 bytes, so a 16-byte piece is either wholly inside a row or past its end.
    bool piece_ok[PIECES];
#pragma unroll
    for (int h = 0; h < PIECES; ++h) piece_ok[h] = col + h * (16 / E) < N;

    const uint8_t *const Ab = static_cast<const uint8_t *>(args.A);
    const uint8_t *const Bb = static_cast<const uint8_t *>(args.B);
    const int64_t ldb_b = args.ldb * E;

    acc_t acc[CPL];
#pragma unroll
    for (int j = 0; j < CPL; ++j) acc[j] = acc_t(0);

    // Batches of U rows (this wave's rows k0, k0 + 4, ..., k0 + 4(U-1)); the loads of
    // the next batch are issued before the current one is consumed, so two batches
    // are in flight per lane.
    struct Batch {
        u32x4_t v[U][PIECES];
        acc_t a[U];
    };
    auto load_batch = [&](Batch &bt, int64_t k0) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t k = k0 + 4 * u;
            const bool row_ok = k < k_end;
            const uint8_t *const row = Bb + k * ldb_b + col * E;
#pragma unroll
            for (int h = 0; h < PIECES; ++h)
                bt.v[u][h] = (row_ok && piece_ok[h]) ? *reinterpret_cast<const u32x4_t *>(row + 16 * h)
                                                     : u32x4_t{0u, 0u, 0u, 0u};
            if constexpr (DT == DT_I8) {
                bt.a[u] = row_ok ? acc_t(reinterpret_cast<const int8_t *>(Ab)[k]) : acc_t(0);
            } else {
                const uint32_t bits = row_ok ? uint32_t(reinterpret_cast<const uint16_t *>(Ab)[k]) : 0u;
                bt.a[u] = __uint_as_float(bits << 16);
            }
        }
    };
    auto use_batch = [&](const Batch &bt) {
        if constexpr (DT == DT_I8) {
            // Four rows at a time: each dword of the four rows' pieces (4 columns x 4 rows of
            // bytes) is transposed so that a dword holds one column's four bytes, then one
            // 4-way dot product with the four rows' A values adds them to that column.
            static_assert(U % 4 == 0 && PIECES == 1, "int8 rows come in groups of four");
#pragma unroll
            for (int g = 0; g < U / 4; ++g) {
                const uint32_t ap = (uint32_t(bt.a[4 * g]) & 0xFFu) | ((uint32_t(bt.a[4 * g + 1]) & 0xFFu) << 8) |
                                    ((uint32_t(bt.a[4 * g + 2]) & 0xFFu) << 16) | (uint32_t(bt.a[4 * g + 3]) << 24);
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    uint32_t col[4];
                    transpose4x4_bytes(bt.v[4 * g][0][w], bt.v[4 * g + 1][0][w], bt.v[4 * g + 2][0][w],
                                       bt.v[4 * g + 3][0][w], col);
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc[4 * w + j] = __builtin_amdgcn_sdot4(int(col[j]), int(ap), acc[4 * w + j], false);
                }
            }
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int h = 0; h < PIECES; ++h)
#pragma unroll
                    for (int w = 0; w < 4; ++w) {
                        const unsigned x = bt.v[u][h][w];
                        acc[8 * h + 2 * w] = fmaf(__uint_as_float(x << 16), bt.a[u], acc[8 * h + 2 * w]);
                        acc[8 * h + 2 * w + 1] =
                            fmaf(__uint_as_float(x & 0xffff0000u), bt.a[u], acc[8 * h + 2 * w + 1]);
                    }
        }
    };
    constexpr int64_t STEP = 4 * U;            // rows advanced per batch (four waves interleaved)
    Batch b0, b1;
    int64_t k0 = k_begin + wave;
    if (k0 < k_end) load_batch(b0, k0);
    for (; k0 < k_end; k0 += 2 * STEP) {
        if (poll_pending && k0 >= k_poll) {
            seen = load_coherent(flag_counter(args, tn));
            poll_pending = false;
        }
        if (k0 + STEP < k_end) load_batch(b1, k0 + STEP);
        use_batch(b0);
        if (k0 + STEP >= k_end) break;
        if (k0 + 2 * STEP < k_end) load_batch(b0, k0 + 2 * STEP);
        use_batch(b1);
    }
    if (poll_pending) seen = load_coherent(flag_counter(args, tn));

    // The four waves' partial sums of the same columns, added in wave order.
    __shared__ acc_t red[4][CB];
#pragma unroll
    for (int j = 0; j < CPL; ++j) red[wave][lane * CPL + j] = acc[j];
    __syncthreads();
    acc_t tot[CB / 256];
#pragma unroll
    for (int i = 0; i < CB / 256; ++i) {
        const int c = int(threadIdx.x) + 256 * i;
        tot[i] = ((red[0][c] + red[1][c]) + red[2][c]) + red[3][c];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < CB / 256; ++i) red[0][int(threadIdx.x) + 256 * i] = tot[i];
    __syncthreads();
    gemv_store<DT, CB>(args, red[0], n0, tn, slice, seen);
}

template <int DT>
__global__ __launch_bounds__(256) void gemv_bt_kernel(KernelArgs args) {
    using acc_t = gemv_acc_t<DT>;
    constexpr int E = Types<DT>::E;
    constexpr int VECE = 16 / E;               // K elements per 16-byte piece
    constexpr int R = 4;                       // columns (stored rows) per wave
    constexpr int CB = 4 * R;                  // columns per workgroup
    const int lane = int(threadIdx.x) & 63;
    const int wave = int(threadIdx.x) >> 6;

    int tm, tn, slice;
    map_tile(args, tm, tn, slice);
    (void)tm;
    const int64_t N = args.N;
    const int64_t n0 = int64_t(tn) * CB;
    const int64_t k_begin = int64_t(slice) * args.k_chunk;
    int64_t k_end = k_begin + args.k_chunk;
    if (k_end > args.K) k_end = args.K;
    const uint8_t *const Ab = static_cast<const uint8_t *>(args.A);
    const uint8_t *const Bb = static_cast<const uint8_t *>(args.B);
    const int64_t ldb_b = args.ldb * E;
    bool row_ok[R];
    const uint8_t *brow[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t n = n0 + wave * R + r;
        row_ok[r] = n < N;
        brow[r] = Bb + (row_ok[r] ? n : 0) * ldb_b;
    }

    // REDUCE_ATOMIC_FLAG: slice 0 zeroes its 16 outputs first; the other slices read the
    // credit counter halfway through their K range.
    const bool flag = DT == DT_I8 && args.split_k > 1 && args.reduce_in_kernel == REDUCE_ATOMIC_FLAG;
    if (flag && slice == 0) flag_zero_tile<1, CB, 256>(args, 0, n0, tn);
    uint32_t seen = 0u;

    acc_t acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = acc_t(0);
    // K * E is a multiple of 16 bytes and so are the slice bounds: a piece is wholly in or out.
    auto step = [&](int64_t k) {
        const u32x4_t a = *reinterpret_cast<const u32x4_t *>(Ab + k * E);
        u32x4_t b[R];
#pragma unroll
        for (int r = 0; r < R; ++r)
            b[r] = row_ok[r] ? *reinterpret_cast<const u32x4_t *>(brow[r] + k * E) : u32x4_t{0u, 0u, 0u, 0u};
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                if constexpr (DT == DT_I8) {
                    acc[r] = __builtin_amdgcn_sdot4(int(a[w]), int(b[r][w]), acc[r], false);
                } else {
                    // Both bf16 halves widened exactly to fp32, then two fused multiply-adds.
                    acc[r] = fmaf(__uint_as_float(a[w] << 16), __uint_as_float(b[r][w] << 16), acc[r]);
                    acc[r] = fmaf(__uint_as_float(a[w] & 0xffff0000u), __uint_as_float(b[r][w] & 0xffff0000u), acc[r]);
                }
            }
    };
    // The first half of the whole 64-piece rounds needs no bound check (every lane's piece
    // of them lies below k_end); the counter read goes between the halves.
    const int half = int((k_end - k_begin) / (64 * VECE) / 2);
    int64_t k = k_begin + int64_t(lane) * VECE;
    for (int it = 0; it < half; ++it, k += 64 * VECE) step(k);
    if (flag && slice != 0) seen = load_coherent(flag_counter(args, tn));
    for (; k < k_end; k += 64 * VECE) step(k);
    // Butterfly over the 64 lanes: every lane ends with the wave's sums.
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) acc[r] += __shfl_xor(acc[r], m, 64);
    __shared__ acc_t res[CB];
    if (lane < R) {
        acc_t v = acc[0];
#pragma unroll
        for (int r = 1; r < R; ++r) v = lane == r ? acc[r] : v;
        res[wave * R + lane] = v;
    }
    __syncthreads();
    gemv_store<DT, CB>(args, res, n0, tn, slice, seen);
}

// Sums split-K partials [split][M][N] into C in slice order 0, 1, ... (the
// same fixed order as the in-kernel reduction).
template <int DT>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(KernelArgs a) {
    using sum_t = typename std::conditional<DT == DT_I8, uint32_t, float>::type;   // int32 wraps mod 2^32
    const sum_t *__restrict__ ws = static_cast<const sum_t *>(a.workspace);
    const int64_t total = a.M * a.N;
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total; idx += stride) {
        sum_t s = ws[idx];
        for (int32_t p = 1; p < a.split_k; ++p) s += ws[int64_t(p) * total + idx];
        const int64_t row = idx / a.N, col = idx % a.N;
        write_c<DT>(a, row * a.ldc + col, s);
    }
}

}  // namespace gemm
