// kern_ring.h -- RING: direct-to-LDS loads into a ring of 64-byte K slots.
#pragma once

#include "gemm_common.h"

namespace gemm {

// ---------------------------------------------------------------------------
// Ring kernel (gfx950): the direct-to-LDS data path of gemm_lds_kernel with a
// deeper prefetch.  K is walked in 64-byte slots (32 bf16 or 64 int8 elements,
// two MFMA k-steps) held in an NB-deep ring of LDS buffers, so that a slot's
// global -> LDS loads are issued NB - 1 slots before the slot is consumed
// instead of one 128-byte stage before; the double buffering of inputs
// (paper, Sec. 4.2.1) generalised to NB buffers.  Measured on the 8192^3 GEMM,
// the one-stage lead of the two-buffer kernel leaves the MFMAs waiting on the
// L2 for about a quarter of the time.
//
// Per slot s (buffer s % NB):
//   phase A: read the k-step 1 fragments of slot s, run the k-step 0 MFMAs
//            (fragments read during slot s - 1);
//   wait until this wave's loads of slot s + 1 have landed, barrier: slot s + 1
//            is visible, and every wave holds all of slot s in registers, so
//            buffer s % NB is free;
//   phase B: run the k-step 1 MFMAs of slot s, read the k-step 0 fragments of
//            slot s + 1, and issue the first half of the loads of slot s + NB into
//            buffer s % NB (phase A of slot s + 1 issues the other half).
// The barrier sits between two runs of MFMAs whose operands are already in
// registers, so the matrix pipes stay fed across it.  Within a phase, the MFMAs,
// LDS reads and global loads are issued in a fixed interleaved order.
//
// LDS, per slot: A as BM rows of 64 K-bytes, the 16-byte chunk c of row r at
// chunk c ^ ring_swz(r); B row-major as 64 / E rows (k) of BN * E bytes, chunk c
// of row k at c ^ ring_bswz(k) (gemm_lds_kernel's swizzle for rows of at least
// 256 bytes, measured conflict-free functions for the narrower rows), or
// column-major (BT) like A.  Every slot of every iteration issues the same
// number of loads (slots past the end of the K range get an empty resource and
// load zeros without touching memory), so the wait before each barrier is a
// fixed count of this wave's loads still allowed in flight.
// ---------------------------------------------------------------------------
template <int DT, int BM, int BN, int WM, int WN, int WAVES_PER_EU, bool BT, int NB>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * WM * WN, 64 * WM * WN),
                          amdgpu_waves_per_eu(WAVES_PER_EU, WAVES_PER_EU)))
void gemm_ring_kernel(KernelArgs args) {
    using acc_vec = typename Types<DT>::acc_vec;
    constexpr int E = Types<DT>::E;
    constexpr int VECE = 16 / E;
    constexpr int BKS = kSlotKBytes / E;                  // K elements per slot
    constexpr int WAVES = WM * WN;
    constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
    constexpr int A_SLOT = BM * kSlotKBytes;              // bytes
    constexpr int B_PITCH = BT ? kSlotKBytes : BN * E;    // bytes per B row in LDS
    constexpr int B_SLOT = BN * kSlotKBytes;
    // A moves in 16-byte pieces per lane (1 KiB per wave-wide load) when its slot
    // splits evenly into such loads over the waves, else in 4-byte pieces (256 B per
    // load); B always moves in 16-byte pieces.
    constexpr int A_W = (A_SLOT % (1024 * WAVES) == 0) ? 16 : 4;
    constexpr int A_LOAD = 64 * A_W;                      // bytes per wave-wide A load
    constexpr int A_INSTR = A_SLOT / A_LOAD / WAVES;
    constexpr int A_ROWS_PER_LOAD = A_LOAD / kSlotKBytes;
    constexpr int B_INSTR = B_SLOT / 1024 / WAVES;
    constexpr int LPS = A_INSTR + B_INSTR;                // loads per wave per slot
    constexpr int B_ROWS_PER_KB = 1024 / B_PITCH;
    constexpr int B_CPR = B_PITCH / 16;                   // 16-byte chunks per B row
    // Row-major B rows are swizzled for conflict-free transpose reads (ring_bswz, by row width).
    constexpr int NREAD = TM + (BT ? TN : 2 * TN);        // LDS reads per k-step
    static_assert(NB >= 3 && NB <= 8, "ring depth");
    static_assert(TM >= 1 && TN >= 1, "wave tile of at least one 32 x 32 MFMA tile");
    static_assert(A_INSTR >= 1 && A_INSTR * A_LOAD * WAVES == A_SLOT, "A slot split");
    static_assert(B_INSTR >= 1 && B_INSTR * 1024 * WAVES == B_SLOT, "B slot split");
    static_assert(B_PITCH <= 1024 && 1024 % B_PITCH == 0, "B row pitch");
    static_assert((NB - 1) * LPS < 64, "loads in flight must fit vmcnt");

    // The ring: NB buffers, each an A part then a B part.
    __shared__ __attribute__((aligned(1024))) uint8_t ring_lds[NB][A_SLOT + B_SLOT];
    auto abuf = [&](auto j_c) -> uint8_t * { return ring_lds[decltype(j_c)::value]; };
    auto bbuf = [&](auto j_c) -> uint8_t * { return abuf(j_c) + A_SLOT; };

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wave_m = wave / WN, wave_n = wave % WN;
    const uint32_t wave_u = uint32_t(__builtin_amdgcn_readfirstlane(wave));   // uniform copy for LDS addresses

    int tm, tn, slice;
    map_tile(args, tm, tn, slice);
    const int64_t M = args.M, N = args.N;
    const int64_t m0 = int64_t(tm) * BM, n0 = int64_t(tn) * BN;
    const int64_t k_begin = int64_t(slice) * args.k_chunk;
    int64_t k_end = k_begin + args.k_chunk;
    if (k_end > args.K) k_end = args.K;
    const int ns = k_end > k_begin ? int((k_end - k_begin + BKS - 1) / BKS) : 0;
    const int64_t k_len = k_end - k_begin;
    const int64_t lda_b = args.lda * E, ldb_b = args.ldb * E;

    // ---- global source offsets of this lane's 16-byte pieces (constant over K) ----
    // A load i of this wave fills bytes [(i*WAVES + wave) KiB, +1 KiB) of the A slot:
    // lane L writes physical chunk L%4 of row (i*WAVES + wave)*16 + L/4, which holds
    // logical chunk (L%4) ^ ga(row).  Rows at or past M are masked by the resource size.
    const int64_t a_rows_valid = (M - m0) < BM ? (M - m0) : BM;
    const uint32_t a_bytes = uint32_t(a_rows_valid * lda_b);
    uint32_t a_voff[A_INSTR];
    int a_chunk[A_INSTR];
#pragma unroll
    for (int i = 0; i < A_INSTR; ++i) {
        // Lane L writes A_W bytes at byte L * A_W of the load's block of A_ROWS_PER_LOAD rows.
        const int row = (i * WAVES + wave) * A_ROWS_PER_LOAD + (lane * A_W) / kSlotKBytes;
        const int byte = (lane * A_W) % kSlotKBytes;
        const int c = (byte >> 4) ^ ring_swz(row);
        a_chunk[i] = c;
        a_voff[i] = uint32_t(row * lda_b + c * 16 + (byte & 15));
    }
    // Row-major B: load i fills B-slot bytes [(i*WAVES + wave) KiB, +1 KiB): lane L writes
    // physical chunk p = L % B_CPR of row (i*WAVES + wave)*B_ROWS_PER_KB + L / B_CPR, holding
    // logical chunk p ^ bswz(row); columns at or past N get an out-of-range offset, K rows
    // past the slice end are masked by the resource size.  Column-major B: as A, over BN
    // rows (n) of the N x K matrix.
    const int64_t b_rows_valid = (N - n0) < BN ? (N - n0) : BN;
    const uint32_t bt_bytes = uint32_t(b_rows_valid * ldb_b);
    uint32_t b_voff[B_INSTR];
    int b_chunk[B_INSTR];
#pragma unroll
    for (int i = 0; i < B_INSTR; ++i) {
        if constexpr (BT) {
            const int row = (i * WAVES + wave) * 16 + (lane >> 2);
            const int c = (lane & 3) ^ ring_swz(row);
            b_chunk[i] = c;
            b_voff[i] = uint32_t(row * ldb_b + c * 16);
        } else {
            const int row = (i * WAVES + wave) * B_ROWS_PER_KB + lane / B_CPR;
            const int c = (lane % B_CPR) ^ ring_bswz<DT, B_CPR>(row);
            b_chunk[i] = 0;
            b_voff[i] = (n0 + int64_t(c) * VECE < N) ? uint32_t(row * ldb_b + c * 16) : kOOB;
        }
    }
    const uint8_t *const a_base = static_cast<const uint8_t *>(args.A) + (m0 * args.lda + k_begin) * E;
    const uint8_t *const b_base = static_cast<const uint8_t *>(args.B) +
                                  (BT ? n0 * args.ldb + k_begin : k_begin * args.ldb + n0) * E;

    // Issues load L (A loads first, then B loads) of slot kt into ring buffer J.  A
    // partial last slot masks its K tail per chunk (A, and column-major B) or by rows
    // (row-major B, through the resource size); slots past the end load nothing.
    auto load_one = [&](int kt, auto j_c, auto l_c) {
        constexpr int L = decltype(l_c)::value;
        const int64_t rem = k_len - int64_t(kt) * BKS;
        if constexpr (L < A_INSTR) {
            const i32x4_t ra = ring_rsrc(a_base + int64_t(kt) * kSlotKBytes, rem > 0 ? a_bytes : 0u);
            const uint32_t off = (rem >= BKS || int64_t(a_chunk[L]) * VECE < rem) ? a_voff[L] : kOOB;
            const uint32_t dst = lds_addr(abuf(j_c)) + (L * WAVES + wave_u) * A_LOAD;
            if constexpr (A_W == 16) ring_load16(ra, dst, off);
            else ring_load4(ra, dst, off);
        } else {
            constexpr int I = L - A_INSTR;
            i32x4_t rb;
            uint32_t off = b_voff[I];
            if constexpr (BT) {
                rb = ring_rsrc(b_base + int64_t(kt) * kSlotKBytes, rem > 0 ? bt_bytes : 0u);
                off = (rem >= BKS || int64_t(b_chunk[I]) * VECE < rem) ? off : kOOB;
            } else {
                const int64_t rows = rem <= 0 ? 0 : (rem < BKS ? rem : BKS);
                rb = ring_rsrc(b_base + int64_t(kt) * BKS * ldb_b, uint32_t(rows * ldb_b));
            }
            ring_load16(rb, lds_addr(bbuf(j_c)) + (I * WAVES + wave_u) * 1024, off);
        }
    };
    auto load_slot = [&](int kt, auto j_c) {
        static_for<0, LPS>([&](auto l_c) { load_one(kt, j_c, l_c); });
    };

    // ---- fragment offsets (lane constants; the k-step and tile index only add immediates) ----
    const int frag_row = lane & 31;
    const int frag_half = lane >> 5;
    const int wrow0 = wave_m * (BM / WM);
    const int wcol0 = wave_n * (BN / WN);
    // A tile i, k-step S: row r_i = wrow0 + 32 i + frag_row, logical chunk 2S + half;
    // ga(r_i) = ga(r_0) (ga has period 32), so the offset is a_fo[S] + 2048 i.
    const int r0 = wrow0 + frag_row;
    int a_fo[2];
#pragma unroll
    for (int S = 0; S < 2; ++S) a_fo[S] = r0 * kSlotKBytes + 16 * ((2 * S + frag_half) ^ ring_swz(r0));
    const int rb0 = wcol0 + frag_row;
    int bt_fo[2];
#pragma unroll
    for (int S = 0; S < 2; ++S) bt_fo[S] = rb0 * kSlotKBytes + 16 * ((2 * S + frag_half) ^ ring_swz(rb0));
    // Row-major B transpose reads: as in gemm_lds_kernel.
    const int grp = lane >> 4, g16 = lane & 15;
    constexpr int TR_ROWS = DT == DT_BF16 ? 4 : 8;        // rows per transpose read
    constexpr int KSTEP = 32 / E;                         // K elements per MFMA
    const int tr_row = DT == DT_BF16 ? (g16 >> 2) : (g16 >> 1);
    const int tr_colb = (DT == DT_BF16 ? (g16 & 3) * 8 : (g16 & 1) * 8) + (grp & 1) * 16 * E;
    const int tr_khalf = (grp >> 1) * (KSTEP / 2);
    const int bz = BT ? 0 : ring_bswz<DT, B_CPR>(tr_row);
    int b_fo[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int colb = (wcol0 + j * 32) * E + tr_colb;
        b_fo[j] = (tr_khalf + tr_row) * B_PITCH + (((colb >> 4) ^ bz) << 4) + (colb & 15);
    }

    u32x4_t fa[2][TM], fb[2][TN];
    // LDS read R of k-step S of ring buffer J into register set SET: reads 0 .. TM-1
    // are A's fragments; then B's, one 16-byte read per fragment (column-major B) or
    // two 8-byte transpose reads (row-major B).
    auto read_one = [&](auto j_c, auto s_c, auto set_c, auto r_c) {
        constexpr int S = decltype(s_c)::value;
        constexpr int SET = decltype(set_c)::value;
        constexpr int R = decltype(r_c)::value;
        const uint8_t *const as = abuf(j_c);
        const uint8_t *const bs = bbuf(j_c);
        if constexpr (R < TM) {
            fa[SET][R] = *reinterpret_cast<const u32x4_t *>(as + a_fo[S] + 2048 * R);
        } else if constexpr (BT) {
            constexpr int J = R - TM;
            fb[SET][J] = *reinterpret_cast<const u32x4_t *>(bs + bt_fo[S] + 2048 * J);
        } else {
            constexpr int J = (R - TM) / 2, H = (R - TM) % 2;
            const u32x2_t v = lds_read_tr<DT>(bs + b_fo[J] + (S * KSTEP + H * TR_ROWS) * B_PITCH);
            fb[SET][J][2 * H] = v[0];
            fb[SET][J][2 * H + 1] = v[1];
        }
    };
    auto load_frags = [&](auto j_c, auto s_c, auto set_c) {
        static_for<0, NREAD>([&](auto r_c) { read_one(j_c, s_c, set_c, r_c); });
    };

    acc_vec acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = acc_vec{};

    // One phase, in a fixed order: MFMA q of register set MS (q = 0 .. TM*TN-1), then,
    // after even q, the next of this phase's global loads [L0, L1) of slot lkt into
    // buffer LJ, then LDS reads 2q and 2q+1 of k-step RS of buffer RJ into set RSET.
    // The loads leave one at a time between MFMAs rather than in a burst that backs
    // up the vector memory path and stalls the issuing waves, and the reads go out
    // early enough for their latency to hide under the MFMAs that follow.
    constexpr int NQ = TM * TN;
    auto phase = [&](auto ms_c, auto rj_c, auto rs_c, auto rset_c, int lkt, auto lj_c, auto l0_c, auto l1_c) {
        constexpr int MS = decltype(ms_c)::value;
        constexpr int L0 = decltype(l0_c)::value, L1 = decltype(l1_c)::value;
        static_for<0, NQ>([&](auto q_c) {
            constexpr int Q = decltype(q_c)::value;
            acc[Q / TN][Q % TN] = mfma32<DT>(fa[MS][Q / TN], fb[MS][Q % TN], acc[Q / TN][Q % TN]);
            constexpr int L = L0 + Q / 2;
            if constexpr (Q % 2 == 0 && L < L1) load_one(lkt, lj_c, std::integral_constant<int, L>{});
            if constexpr (2 * Q < NREAD) read_one(rj_c, rs_c, rset_c, std::integral_constant<int, 2 * Q>{});
            if constexpr (2 * Q + 1 < NREAD) read_one(rj_c, rs_c, rset_c, std::integral_constant<int, 2 * Q + 1>{});
            __builtin_amdgcn_sched_barrier(0);
        });
        // Reads beyond two per MFMA (none for the configurations compiled here).
        static_for<2 * NQ, NREAD>([&](auto r_c) { read_one(rj_c, rs_c, rset_c, r_c); });
        static_for<L0 + (NQ + 1) / 2, L1>([&](auto l_c) { load_one(lkt, lj_c, l_c); });
    };

    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    // The loads of slot s + NB (into buffer s % NB, free after the barrier of slot s) are
    // split between phase B of slot s (loads 0 .. LB-1) and phase A of slot s + 1 (the
    // rest); both come before the barrier of slot s + 1, which waits for slot s + 2.
    constexpr int LB = (LPS + 1) / 2;
    using LBC = std::integral_constant<int, LB>;
    using LPSC = std::integral_constant<int, LPS>;

    auto slot = [&](int kt, auto j_c) {
        constexpr int J = decltype(j_c)::value;
        using NEXT = std::integral_constant<int, (J + 1) % NB>;
        using PREV = std::integral_constant<int, (J + NB - 1) % NB>;
        // phase A: MFMAs of k-step 0 (set 0); read k-step 1 of this slot into set 1;
        // finish the loads of slot kt - 1 + NB into buffer J - 1.
        phase(I0{}, j_c, I1{}, I1{}, kt - 1 + NB, PREV{}, LBC{}, LPSC{});
        ring_barrier<(NB - 2) * LPS>();
        __builtin_amdgcn_sched_barrier(0);
        // phase B: MFMAs of k-step 1 (set 1); start the loads of slot kt + NB into
        // buffer J; read k-step 0 of the next slot into set 0.
        phase(I1{}, NEXT{}, I0{}, I0{}, kt + NB, j_c, I0{}, LBC{});
    };

    // REDUCE_ATOMIC_FLAG: slice 0 zeroes its tile of C before loading anything; every
    // other slice reads the tile's credit counter (every wave, so that the test stays
    // uniform) at the last ring turn that starts at least kFlagLeadSlots slots before
    // its end (at the first turn if the slice is shorter than that).
    constexpr int kFlagLeadSlots = 8;
    const bool flag = DT == DT_I8 && args.split_k > 1 && args.reduce_in_kernel == REDUCE_ATOMIC_FLAG;
    const int flag_tile = tm * args.tiles_n + tn;
    if (flag && slice == 0) flag_zero_tile<BM, BN, 64 * WAVES>(args, m0, n0, flag_tile);
    const int poll_kt = (flag && slice != 0) ? (ns > kFlagLeadSlots ? (ns - kFlagLeadSlots) / NB * NB : 0) : -1;
    uint32_t seen = 0u;

    if (ns > 0) {
        // Prologue: slots 0 .. NB-2 whole and the first LB loads of slot NB-1 (phase A
        // of slot 0 issues the rest, as every phase A does), then slot 0 is waited for.
        static_for<0, NB - 1>([&](auto u) { load_slot(decltype(u)::value, u); });
        static_for<0, LB>([&](auto l_c) { load_one(NB - 1, std::integral_constant<int, NB - 1>{}, l_c); });
        ring_barrier<(NB - 2) * LPS + LB>();
        load_frags(I0{}, I0{}, I0{});
        for (int kt = 0; kt < ns; kt += NB) {
            if (kt == poll_kt) seen = load_coherent(flag_counter(args, flag_tile));
            static_for<0, NB>([&](auto u) {
                if (kt + decltype(u)::value < ns) slot(kt + decltype(u)::value, u);
            });
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // drain ring loads past the end before exit

    // The ring is drained and every wave is past its last fragment read when
    // store_tile first synchronises, so it lends the last-slice flag a word.
    store_tile<DT, BM, BN, TM, TN>(args, acc, tm, tn, slice, m0 + wrow0, n0 + wcol0, lane,
                                   *reinterpret_cast<int *>(ring_lds[0]), seen);
}

}  // namespace gemm
