// kern_direct.h -- direct-to-LDS kernels: DIRECT (two 128-byte K stages) and
// the ping-pong variant.
#pragma once

#include "gemm_common.h"

namespace gemm {

// ---------------------------------------------------------------------------
// Direct-to-LDS kernel (gfx950): both operands go from global memory straight
// into LDS with buffer_load ... lds, and B's K-contiguous MFMA fragments are
// produced by LDS transpose reads (ds_read_b64_tr_b16 / _b8) instead of an
// in-register transpose.  The K loop then holds only loads, LDS reads, MFMAs
// and one barrier per stage.
//
// LDS, per stage: A as BM rows of 128 K-bytes (16-byte chunks XOR-swizzled by
// swz(c, row)), B untransposed as BK rows (k) of BN*E bytes (chunks swizzled by
// a function of k mod 4 (bf16) or k mod 8 (int8), matched to the row sets the
// transpose reads touch together).
//
// Transpose read, per 16-lane group (lane g within the group): every lane
// supplies the address of one 8-byte piece; lane g receives column g of the
// block formed by the group's pieces -- b16: 4 rows x 16 columns, lane g
// addresses row g/4, columns 4(g%4)..+3; b8: 8 rows x 16 columns, lane g
// addresses row g/2, columns 8(g%2)..+7.
// ---------------------------------------------------------------------------
template <int DT, int BM, int BN, int WM, int WN, int WAVES_PER_EU, bool BT = false>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * WM * WN, 64 * WM * WN),
                          amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void gemm_lds_kernel(KernelArgs args) {
    using acc_vec = typename Types<DT>::acc_vec;
    using out_t = typename Types<DT>::out_t;
    constexpr int E = Types<DT>::E;
    constexpr int VECE = 16 / E;
    constexpr int BK = kStageKBytes / E;                  // K elements per stage
    constexpr int THREADS = 64 * WM * WN;
    constexpr int WAVES = WM * WN;
    constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
    constexpr int A_STAGE = BM * kStageKBytes;            // bytes
    // Row-major B sits in LDS as BK rows (k) of BN*E bytes; column-major B (BT)
    // as BN rows (n) of 128 K-bytes, exactly like A.
    constexpr int B_PITCH = BT ? kStageKBytes : BN * E;   // bytes per B row in LDS
    constexpr int B_STAGE = BN * kStageKBytes;
    constexpr int A_INSTR = A_STAGE / 1024 / WAVES;       // 1 KiB per wave-wide load
    constexpr int B_INSTR = B_STAGE / 1024 / WAVES;
    constexpr int B_ROWS_PER_KB = 1024 / B_PITCH;         // B rows covered by one wave-wide load
    static_assert(A_INSTR >= 1 && A_INSTR * 1024 * WAVES == A_STAGE, "A stage split");
    static_assert(B_INSTR >= 1 && B_INSTR * 1024 * WAVES == B_STAGE, "B stage split");
    static_assert(B_PITCH <= 1024 && 1024 % B_PITCH == 0, "B row pitch");

    // One LDS array per stage buffer and operand: with every access naming a
    // fixed array, the compiler can tell the direct-to-LDS writes of one stage
    // from the fragment reads of the other and does not serialise them.
    __shared__ __attribute__((aligned(1024))) uint8_t a_lds0[A_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t a_lds1[A_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t b_lds0[B_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t b_lds1[B_STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wave_m = wave / WN, wave_n = wave % WN;

    int tm, tn, slice;
    map_tile(args, tm, tn, slice);
    const int64_t M = args.M, N = args.N;
    const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;
    const int64_t k_begin = int64_t(slice) * args.k_chunk;
    int64_t k_end = k_begin + args.k_chunk;
    if (k_end > args.K) k_end = args.K;
    const int nk = k_end > k_begin ? int((k_end - k_begin + BK - 1) / BK) : 0;
    const int64_t lda_b = args.lda * E, ldb_b = args.ldb * E;

    // ---- global source offsets of this lane's 16-byte pieces (constant over K) ----
    // A load i of this wave fills LDS bytes [(i*WAVES + wave) KiB, +1 KiB): lane L
    // writes physical chunk L%8 of row (i*WAVES + wave)*8 + L/8, which holds the
    // logical chunk c = (L%8) ^ f(row).  Rows at or past M are masked by the
    // resource size (rows_valid * lda bytes from the tile's first row).
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
    // B load i fills LDS bytes [(i*WAVES + wave) KiB, +1 KiB) of the B stage: lane L
    // writes physical chunk p = L % B_CPR of row (i*WAVES+wave)*B_ROWS_PER_KB + L / B_CPR,
    // holding logical chunk p ^ bswz(row).  Columns at or past N get an out-of-range
    // offset; K rows past the slice end are masked by the resource size.
    // Column-major B (BT): the same scheme as A over BN rows (n) of the N x K
    // matrix; rows at or past N are masked by the resource size.
    constexpr int B_CPR = B_PITCH / 16;                   // chunks per B row
    static_assert(BT || B_CPR >= 16, "transpose-read swizzle needs rows of at least 16 chunks");
    const int64_t b_rows_valid = (N - n0) < BN ? (N - n0) : BN;
    const uint32_t bt_bytes = uint32_t(b_rows_valid * ldb_b);
    uint32_t b_voff[B_INSTR];
    int b_chunk[B_INSTR];
#pragma unroll
    for (int i = 0; i < B_INSTR; ++i) {
        if constexpr (BT) {
            const int row = (i * WAVES + wave) * 8 + (lane >> 3);
            const int c = (lane & 7) ^ ((row ^ (row >> 3)) & 7);
            b_chunk[i] = c;
            b_voff[i] = uint32_t(row * ldb_b + c * 16);
        } else {
            const int row = (i * WAVES + wave) * B_ROWS_PER_KB + lane / B_CPR;
            const int c = (lane % B_CPR) ^ bswz<DT>(row);
            b_chunk[i] = 0;
            b_voff[i] = (n0 + int64_t(c) * VECE < N) ? uint32_t(row * ldb_b + c * 16) : kOOB;
        }
    }
    const uint8_t *const a_base = static_cast<const uint8_t *>(args.A) + (m0 * args.lda + k_begin) * E;
    const uint8_t *const b_base = static_cast<const uint8_t *>(args.B) +
                                  (BT ? n0 * args.ldb + k_begin : k_begin * args.ldb + n0) * E;
    // B resource of stage kt; `rows` valid K rows bound row-major B only.
    auto b_rsrc = [&](int kt, int64_t rows) {
        if constexpr (BT) return make_rsrc(b_base + int64_t(kt) * kStageKBytes, bt_bytes);
        else return make_rsrc(b_base + int64_t(kt) * BK * ldb_b, uint32_t(rows * ldb_b));
    };
    const int64_t k_len = k_end - k_begin;

    // Issues the loads of stage kt into LDS buffer BUF.  Full stages use the
    // precomputed offsets as they are; only a partial last stage (and stages past
    // the end, which load nothing) pays for the per-chunk K mask.
    auto load_stage = [&](int kt, auto buf_c) {
        constexpr int BUF = decltype(buf_c)::value;
        const int64_t rem = k_len - int64_t(kt) * BK;
        const __amdgpu_buffer_rsrc_t ra = make_rsrc(a_base + int64_t(kt) * kStageKBytes, a_bytes);
        const int64_t rows = rem <= 0 ? 0 : (rem < BK ? rem : BK);
        const __amdgpu_buffer_rsrc_t rb = b_rsrc(kt, rows);
        uint8_t *const as = BUF ? a_lds1 : a_lds0;
        uint8_t *const bs = BUF ? b_lds1 : b_lds0;
        if (rem >= BK) {
#pragma unroll
            for (int i = 0; i < A_INSTR; ++i) {
                load_lds16(ra, as + (i * WAVES + wave) * 1024, a_voff[i]);
                if (i < B_INSTR) load_lds16(rb, bs + (i * WAVES + wave) * 1024, b_voff[i]);
            }
#pragma unroll
            for (int i = A_INSTR; i < B_INSTR; ++i) load_lds16(rb, bs + (i * WAVES + wave) * 1024, b_voff[i]);
        } else {
#pragma unroll
            for (int i = 0; i < A_INSTR; ++i) {
                const uint32_t off = int64_t(a_chunk[i]) * VECE < rem ? a_voff[i] : kOOB;
                load_lds16(ra, as + (i * WAVES + wave) * 1024, off);
            }
#pragma unroll
            for (int i = 0; i < B_INSTR; ++i) {
                // Column-major B masks its K tail per chunk, as A does; row-major B by rows.
                const uint32_t off = (!BT || int64_t(b_chunk[i]) * VECE < rem) ? b_voff[i] : kOOB;
                load_lds16(rb, bs + (i * WAVES + wave) * 1024, off);
            }
        }
    };

    // A full stage's loads issued in two halves, at the start of k-steps 0 and 1:
    // issuing all of them in one burst backs up the vector memory path and
    // stalls the issuing waves (and their MFMAs) for longer than the spread
    // costs in latency.  A partial last stage is loaded whole with part 0.
    auto load_stage_part = [&](int kt, auto buf_c, int part) {
        constexpr int BUF = decltype(buf_c)::value;
        const int64_t rem = k_len - int64_t(kt) * BK;
        if (rem < BK) {
            if (part == 0) load_stage(kt, buf_c);
            return;
        }
        const __amdgpu_buffer_rsrc_t ra = make_rsrc(a_base + int64_t(kt) * kStageKBytes, a_bytes);
        const __amdgpu_buffer_rsrc_t rb = b_rsrc(kt, BK);
        uint8_t *const as = BUF ? a_lds1 : a_lds0;
        uint8_t *const bs = BUF ? b_lds1 : b_lds0;
#pragma unroll
        for (int i = 0; i < (A_INSTR > B_INSTR ? A_INSTR : B_INSTR); ++i) {
            if ((i & 1) != part) continue;
            if (i < A_INSTR) load_lds16(ra, as + (i * WAVES + wave) * 1024, a_voff[i]);
            if (i < B_INSTR) load_lds16(rb, bs + (i * WAVES + wave) * 1024, b_voff[i]);
        }
    };

    // ---- fragment offsets (lane constants; the k-step and tile index only add immediates) ----
    const int frag_row = lane & 31;
    const int frag_half = lane >> 5;
    const int wrow0 = wave_m * (BM / WM);
    const int wcol0 = wave_n * (BN / WN);
    // A tile i, k-step s: row r_i = wrow0 + 32 i + frag_row, chunk 2s + half, swizzled by
    // f(r_i) = f(r_0) ^ 4 (i & 1).  Offset = r_0*128 + 4096 i + 16 ((2s + half) ^ f(r_0) ^ 4(i&1)).
    const int r0 = wrow0 + frag_row;
    const int f0 = (r0 ^ (r0 >> 3)) & 7;
    int a_fo[2][4];
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int st = 0; st < 4; ++st) a_fo[p][st] = r0 * kStageKBytes + 16 * ((2 * st + frag_half) ^ f0 ^ (4 * p));
    // B transpose reads: group = lane/16, g = lane%16.
    // bf16: rows 4*h + g/4 (+8 for the upper K half), byte columns 8*(g%4) (+32 for odd groups)
    // int8: rows 8*h + g/2 (+16 for the upper K half), byte columns 8*(g%2) (+16 for odd groups)
    // The row's swizzle depends only on g (k mod 4 or 8), so tile j, read h, k-step s
    // is b_fo[j] + (s*KSTEP + h*TR_ROWS) * B_PITCH.
    const int grp = lane >> 4, g16 = lane & 15;
    constexpr int TR_ROWS = DT == DT_BF16 ? 4 : 8;        // rows per transpose read
    constexpr int KSTEP = 32 / E;                         // K elements per MFMA
    const int tr_row = DT == DT_BF16 ? (g16 >> 2) : (g16 >> 1);
    const int tr_colb = (DT == DT_BF16 ? (g16 & 3) * 8 : (g16 & 1) * 8) + (grp & 1) * 16 * E;
    const int tr_khalf = (grp >> 1) * (KSTEP / 2);
    const int bz = bswz<DT>(tr_row);
    int b_fo[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int colb = (wcol0 + j * 32) * E + tr_colb;
        b_fo[j] = (tr_khalf + tr_row) * B_PITCH + (((colb >> 4) ^ bz) << 4) + (colb & 15);
    }
    // Column-major B: fragments are 16-byte reads of K-contiguous rows, as for A.
    const int rb0 = wcol0 + frag_row;
    const int fb0 = (rb0 ^ (rb0 >> 3)) & 7;
    int bt_fo[2][4];
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int st = 0; st < 4; ++st) bt_fo[p][st] = rb0 * kStageKBytes + 16 * ((2 * st + frag_half) ^ fb0 ^ (4 * p));

    u32x4_t fa[2][TM], fb[2][TN];
    auto load_frags = [&](auto buf_c, auto s_c, auto slot_c) {
        constexpr int BUF = decltype(buf_c)::value;
        constexpr int S = decltype(s_c)::value;
        constexpr int SLOT = decltype(slot_c)::value;
        const uint8_t *const as = BUF ? a_lds1 : a_lds0;
        const uint8_t *const bs = BUF ? b_lds1 : b_lds0;
#pragma unroll
        for (int i = 0; i < TM; ++i)
            fa[SLOT][i] = *reinterpret_cast<const u32x4_t *>(as + a_fo[i & 1][S] + 4096 * i);
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            if constexpr (BT) {
                fb[SLOT][j] = *reinterpret_cast<const u32x4_t *>(bs + bt_fo[j & 1][S] + 4096 * j);
            } else {
                const u32x2_t lo = lds_read_tr<DT>(bs + b_fo[j] + (S * KSTEP) * B_PITCH);
                const u32x2_t hi = lds_read_tr<DT>(bs + b_fo[j] + (S * KSTEP + TR_ROWS) * B_PITCH);
                fb[SLOT][j] = u32x4_t{lo[0], lo[1], hi[0], hi[1]};
            }
        }
    };

    acc_vec acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = acc_vec{};
#pragma unroll
    for (int i = 0; i < TM; ++i) fa[1][i] = u32x4_t{0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < TN; ++j) fb[1][j] = u32x4_t{0u, 0u, 0u, 0u};

    auto mfma_slot = [&](auto slot_c) {
        constexpr int SLOT = decltype(slot_c)::value;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma32<DT>(fa[SLOT][i], fb[SLOT][j], acc[i][j]);
    };

    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;

    // One stage (buffer BUF holds stage kt, visible).  On entry slot 1 holds the
    // fragments of the previous stage's last k-step, whose MFMAs run here, under
    // the latency of this stage's first LDS reads; on exit slot 1 holds this
    // stage's last k-step and every wave has finished reading buffer BUF.
    auto stage = [&](int kt, auto buf_c) {
        constexpr int BUF = decltype(buf_c)::value;
        using OTHER = std::integral_constant<int, 1 - BUF>;
        load_stage_part(kt + 1, OTHER{}, 0);
        __builtin_amdgcn_sched_barrier(0);
        load_frags(buf_c, I0{}, I0{});
        mfma_slot(I1{});
        __builtin_amdgcn_sched_barrier(0);
        load_stage_part(kt + 1, OTHER{}, 1);
        __builtin_amdgcn_sched_barrier(0);
        load_frags(buf_c, I1{}, I1{});
        mfma_slot(I0{});
        __builtin_amdgcn_sched_barrier(0);
        load_frags(buf_c, I2{}, I0{});
        mfma_slot(I1{});
        __builtin_amdgcn_sched_barrier(0);
        load_frags(buf_c, I3{}, I1{});
        mfma_slot(I0{});
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    };

    if (nk > 0) {
        load_stage(0, I0{});
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    }
    int kt = 0;
    for (; kt + 1 < nk; kt += 2) {
        stage(kt, I0{});
        stage(kt + 1, I1{});
    }
    if (kt < nk) stage(kt, I0{});
    mfma_slot(I1{});

    __shared__ int s_last;
    store_tile<DT, BM, BN, TM, TN>(args, acc, tm, tn, slice, m0 + wrow0, n0 + wcol0, lane, s_last);
}

// ---------------------------------------------------------------------------
// Ping-pong direct-to-LDS kernel: 256 x 256 macro-tile, 8 waves, two wave
// groups that alternate between a compute phase and a memory phase.
//
// Waves w and w + 4 share a SIMD.  Group 0 (waves 0-3) owns output rows 0-127
// of the tile, group 1 rows 128-255; each wave a 128 x 64 sub-tile.  A "unit"
// is half a stage (two MFMA k-steps).  Group 1 runs one phase behind group 0,
// so in every phase one wave per SIMD issues a dense run of 16 MFMAs from
// fragments already in registers while the other reads its next unit's
// fragments from LDS and issues its share of the next stage's global -> LDS
// loads.  Phases are separated by workgroup barriers.  Stage s sits in LDS
// buffer s % 2 and is read in phases 4s .. 4s+3; the loads of stage s+1 are
// issued in phases 4s (group 0) and 4s+1 (group 1) and waited for at the end
// of phase 4s+3, so a load has three phases to land.  Every wave executes
// the same barrier sequence; only the work between barriers depends on the
// group.
// ---------------------------------------------------------------------------
template <int DT>
__global__ __attribute__((amdgpu_flat_work_group_size(512, 512), amdgpu_waves_per_eu(2, 2)))
void gemm_pingpong_kernel(KernelArgs args) {
    using acc_vec = typename Types<DT>::acc_vec;
    using out_t = typename Types<DT>::out_t;
    constexpr int BM = 256, BN = 256, WAVES = 8;
    constexpr int E = Types<DT>::E;
    constexpr int VECE = 16 / E;
    constexpr int BK = kStageKBytes / E;
    constexpr int TM = 4, TN = 2;                          // 128 x 64 per wave
    constexpr int A_STAGE = BM * kStageKBytes;
    constexpr int B_PITCH = BN * E;
    constexpr int B_STAGE = BK * B_PITCH;
    constexpr int A_INSTR = A_STAGE / 1024 / WAVES;        // 4
    constexpr int B_INSTR = B_STAGE / 1024 / WAVES;        // 4
    constexpr int B_ROWS_PER_KB = 1024 / B_PITCH;
    constexpr int B_CPR = B_PITCH / 16;

    __shared__ __attribute__((aligned(1024))) uint8_t a_lds0[A_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t a_lds1[A_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t b_lds0[B_STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t b_lds1[B_STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int grp = wave >> 2;
    const int wave_m = grp, wave_n = wave & 3;

    int tm, tn, slice;
    map_tile(args, tm, tn, slice);
    const int64_t M = args.M, N = args.N;
    const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;
    const int64_t k_begin = int64_t(slice) * args.k_chunk;
    int64_t k_end = k_begin + args.k_chunk;
    if (k_end > args.K) k_end = args.K;
    const int nk = k_end > k_begin ? int((k_end - k_begin + BK - 1) / BK) : 0;
    const int64_t lda_b = args.lda * E, ldb_b = args.ldb * E;

    // global -> LDS source offsets (see gemm_lds_kernel)
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

    auto load_stage = [&](int kt, auto buf_c) {
        constexpr int BUF = decltype(buf_c)::value;
        const int64_t rem = k_len - int64_t(kt) * BK;
        const __amdgpu_buffer_rsrc_t ra = make_rsrc(a_base + int64_t(kt) * kStageKBytes, a_bytes);
        const int64_t rows = rem <= 0 ? 0 : (rem < BK ? rem : BK);
        const __amdgpu_buffer_rsrc_t rb = make_rsrc(b_base + int64_t(kt) * BK * ldb_b, uint32_t(rows * ldb_b));
        uint8_t *const as = BUF ? a_lds1 : a_lds0;
        uint8_t *const bs = BUF ? b_lds1 : b_lds0;
        if (rem >= BK) {
#pragma unroll
            for (int i = 0; i < A_INSTR; ++i) {
                load_lds16(ra, as + (i * WAVES + wave) * 1024, a_voff[i]);
                load_lds16(rb, bs + (i * WAVES + wave) * 1024, b_voff[i]);
            }
        } else {
#pragma unroll
            for (int i = 0; i < A_INSTR; ++i) {
                const uint32_t off = int64_t(a_chunk[i]) * VECE < rem ? a_voff[i] : kOOB;
                load_lds16(ra, as + (i * WAVES + wave) * 1024, off);
                load_lds16(rb, bs + (i * WAVES + wave) * 1024, b_voff[i]);
            }
        }
    };

    // fragment offsets (see gemm_lds_kernel)
    const int frag_row = lane & 31;
    const int frag_half = lane >> 5;
    const int wrow0 = wave_m * (BM / 2);
    const int wcol0 = wave_n * (BN / 4);
    const int r0 = wrow0 + frag_row;
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

    u32x4_t fa[2][TM], fb[2][TN];                          // one unit: two k-steps
    auto load_unit = [&](auto buf_c, auto h_c) {
        constexpr int BUF = decltype(buf_c)::value;
        constexpr int H = decltype(h_c)::value;
        const uint8_t *const as = BUF ? a_lds1 : a_lds0;
        const uint8_t *const bs = BUF ? b_lds1 : b_lds0;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            constexpr int dummy = 0; (void)dummy;
            const int S = 2 * H + ks;
#pragma unroll
            for (int i = 0; i < TM; ++i)
                fa[ks][i] = *reinterpret_cast<const u32x4_t *>(as + a_fo[i & 1][S] + 4096 * i);
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const u32x2_t lo = lds_read_tr<DT>(bs + b_fo[j] + (S * KSTEP) * B_PITCH);
                const u32x2_t hi = lds_read_tr<DT>(bs + b_fo[j] + (S * KSTEP + TR_ROWS) * B_PITCH);
                fb[ks][j] = u32x4_t{lo[0], lo[1], hi[0], hi[1]};
            }
        }
    };

    acc_vec acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = acc_vec{};

    auto compute_unit = [&]() {
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = mfma32<DT>(fa[ks][i], fb[ks][j], acc[i][j]);
        __builtin_amdgcn_s_setprio(0);
    };

    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;

    // Four phases of stage s (LDS buffer BUF = s % 2).
    auto stage_phases = [&](int s, auto buf_c) {
        using OTHER = std::integral_constant<int, 1 - decltype(buf_c)::value>;
        // phase 4s
        if (grp == 0) {
            if (s + 1 < nk) load_stage(s + 1, OTHER{});
            load_unit(buf_c, I0{});
        } else if (s > 0) {
            compute_unit();
        }
        phase_barrier();
        // phase 4s+1
        if (grp == 0) {
            compute_unit();
        } else {
            if (s + 1 < nk) load_stage(s + 1, OTHER{});
            load_unit(buf_c, I0{});
        }
        phase_barrier();
        // phase 4s+2
        if (grp == 0) load_unit(buf_c, I1{});
        else compute_unit();
        phase_barrier();
        // phase 4s+3
        if (grp == 0) compute_unit();
        else load_unit(buf_c, I1{});
        stage_barrier();
    };

    if (nk > 0) {
        load_stage(0, I0{});
        stage_barrier();
        for (int s = 0; s < nk; s += 2) {
            stage_phases(s, I0{});
            if (s + 1 < nk) stage_phases(s + 1, I1{});
        }
        if (grp == 1) compute_unit();                       // group 1's last unit
    }

    __shared__ int s_last;
    store_tile<DT, BM, BN, TM, TN>(args, acc, tm, tn, slice, m0 + wrow0, n0 + wcol0, lane, s_last);
}

}  // namespace gemm
