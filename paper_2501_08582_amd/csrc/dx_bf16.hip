// Backward data gradient with weight recompute, bf16 on gfx950.
//
//   dX[L x C] = dY[L x R] . W',   W' = select(M, W + s.B.A, 0)
//
// (dX step of the SP-LoRA backward list in Section 2.2; the merged weight is
// recomputed instead of stored, Algorithm 2 / Section 2.3.)  GEMM over K = R.
//
// Same structure as the forward: each of the 4 waves owns 64 input features
// (n) of the 256 x 256 tile and rebuilds W'[k][n] for its columns in
// registers, in the B-operand layout of the main MFMA (rank-r MFMA with its
// k rows taken in the order pi, see the forward kernel).  Differences:
//   * W is stored [k][n] (k = R), so the raw W values a lane needs -- eight
//     consecutive k of one column n -- come from two LDS transpose loads; the
//     W slab is four per-wave blocks (the 64 k rows of that wave's 64
//     columns, tr64 layout), each filled by its own wave's copies;
//   * the k-rows of the rank-r product are B[k][:], read from a B slab copied
//     contiguously into LDS each K-step; A[:, n] is resident in registers;
//   * the mask bits a lane needs run along k for a fixed n, so they are read
//     from the transposed bitmap M^T (built once per backward call).
// The schedule is the forward's: four sub-steps of 16 k per K-step, each
// MFMA slot carrying a fixed share of the next sub-step's operand reads and
// merge arithmetic, one barrier per K-step before the last sub-step, which
// interleaves the copies of stage kt+2 and the first sub-step of stage kt+1.
// For a power-of-two scale the merge is folded as in the forward: the
// resident A operand is pre-scaled by s, the rank-r MFMA accumulates onto W
// (read, for the next stage, as soon as the wave's own W copies landed), and
// a merge piece is the rounding and the select.
// Works on ranks that are multiples of 8, up to 64 per pass (the launcher pads
// other ranks with a zero-filled copy of B and splits larger ones in two).
#include "gemm_common.hpp"
#include "kernels.hpp"

#include <cmath>
#include <type_traits>

namespace lors {
namespace {

constexpr int NT = 256;
constexpr int BM = 256;  // tokens per tile
constexpr int BN = 256;  // input features per whole tile (64 per wave)
constexpr int BK = 64;   // output features (rows of W) per K-step
constexpr int GROUP_M = 4;
constexpr int kEarly = 12;  // copies of a stage issued right after the barrier; the rest a sub-step later

// B slab [k][rank]: 64 rows of PITCH = 32*RKP bytes (ranks padded to 16*RKP;
// RKP = RK, except 4 for RK = 3 so that a row holds a power of two of 16-byte
// chunks).  Chunk q of row k is stored at chunk q ^ bswz(k): the merge reads
// one chunk of 16 consecutive rows per 16 lanes, and with rows 32*RKP bytes
// apart those rows would fall on only 8 / RKP of the 16 bank groups; the XOR
// spreads them over all 16 (a 256-byte bank window holds 8 / RKP rows, and
// bswz takes 2*RKP distinct values over 16 consecutive rows).
// TM: tokens per tile, NF: 32-column blocks per wave -- BM and 2 for a whole
// tile; a thin tile of a short last wave has half the columns (NF = 1) and
// TM = 256, 128 or 64 tokens.
// W slab: 4 per-wave blocks of [64 k][32 NF n]; with NF = 2 a block has
// 128-byte rows in the tr64 layout, with NF = 1 64-byte rows unswizzled (the
// four rows a 32-lane transpose read covers are then 256 consecutive bytes,
// one per bank).
template <int RK, int TM, int NF>
struct Layout {
    static constexpr int FT = 128 * NF;            // input features per tile
    static constexpr int WROW = 64 * NF;           // bytes per row of a wave's W block
    static constexpr int WBW = BK * WROW;          // one wave's W block
    static constexpr int WB = 4 * WBW;             // W slab
    static constexpr int MB = FT * 2 * 4;          // M^T words [n][kb]
    static constexpr int DB = TM * kRow64;         // dY slab: TM rows of 64 k
    static constexpr int RKP = RK == 3 ? 4 : RK;
    static constexpr int PITCH = 32 * RKP;
    static constexpr int BB = BK * PITCH;          // B slab: 2 KiB per 16 ranks
    static constexpr int D = 0, W = DB, B = DB + WB, M = DB + WB + BB;
    static constexpr int STAGE = DB + WB + BB + MB;
    static constexpr int LUT = 2 * STAGE;          // select table: 16 x 8 B
    static constexpr int SINK = LUT + 256;         // 1 KiB target of padding copies
    static constexpr int TOTAL = SINK + 1024;
    static constexpr int NBC = BB / 1024;          // 1 KiB copies per B slab
    static constexpr int NB = (NBC + 3) / 4;       // B-slab copies per wave
    static constexpr int ND = TM / 32;             // dY-slab copies per wave
    static constexpr int NWC = WBW / 1024;         // W-block copies per wave
    static constexpr int NMC = NF;                 // M^T copies per wave
    static constexpr int COPIES = ND + NWC + NB + NMC;  // copies per wave per stage
    static constexpr int EARLY = COPIES < kEarly ? COPIES : kEarly;
    static_assert(COPIES - EARLY <= 8, "the late copies fit the eight merge slots");
    // physical chunk of logical chunk q in B-slab row k
    static __device__ __forceinline__ int bswz(int k, int q) { return q ^ ((k / (8 / RKP)) & (2 * RKP - 1)); }
};

#define SLOT_END() __builtin_amdgcn_sched_barrier(0)

// RAGGED: some tile reaches past L, C or R (copies check every lane and read
// the zero page outside the tensors); otherwise copies use uniform bases plus
// fixed per-lane offsets.
// PASS2: the second pass of a rank above 64 (ranks 64.. of B and A): W is
// taken as zero and the product is added onto dX.  ldb: row stride of B.
// r: the rank the kernel works on, a multiple of 8 (B's columns ra .. r-1
// are zero); ra: the rows of A that exist (A rows ra .. r-1 are read as zero).
// TM, NF < (BM, 2): a thin tile of TM tokens and 128 NF input features
// (whole-tile shapes, one pass), as in the forward kernel.
template <int RK, bool RAGGED, bool PASS2, bool FOLD, int TM, int NF>
__global__ __launch_bounds__(NT, 1) void dx_kernel(
    const uint16_t* __restrict__ dY, const uint16_t* __restrict__ W,
    const uint32_t* __restrict__ Mt, const uint16_t* __restrict__ Bm,
    const uint16_t* __restrict__ Am, uint16_t* __restrict__ dX, int64_t L, int R, int C, int r,
    int ra, float s, int tiles_m, int tiles_n, int ldb, float* __restrict__ z0, int64_t nz0,
    float* __restrict__ z1, int64_t nz1, int n_full, int split, float* __restrict__ part) {
    using Lay = Layout<RK, TM, NF>;
    constexpr int MBW = TM / 32;  // 32-token blocks per wave
    static_assert((TM == BM && NF == 2) || (!RAGGED && !PASS2), "thin tiles: fixed-offset copies, one pass");
    static_assert(Lay::TOTAL <= 160 * 1024, "LDS budget");
    static_assert(4 * TM * 64 * NF <= 2 * Lay::STAGE, "output staging fits the stage buffers");
    // the prologue parks the merge's A block in stage 1: in its dY region,
    // clear of the W slabs that PASS2 zeroes once (a thin tile's dY region is
    // smaller, but it has no second pass and may use the whole stage)
    static_assert(16 * RK * kRowBytes <= (PASS2 ? Lay::DB : Lay::STAGE), "A block fits stage 1");
    __shared__ __attribute__((aligned(1024))) uint8_t smem[Lay::TOTAL];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31;
    const int h = lane >> 5;

    // z0, z1: dB and dA of the combined backward, cleared here for the fp32
    // atomics of the weight-gradient kernel that follows on the same stream
    // (one launch fewer; plain stores, grid-stride)
    if (z0 != nullptr) {
        const int64_t stride = (int64_t)gridDim.x * NT;
        for (int64_t t = (int64_t)blockIdx.x * NT + tid; t < nz0 + nz1; t += stride) {
            if (t < nz0) z0[t] = 0.f;
            else z1[t - nz0] = 0.f;
        }
    }

    // tile and K-steps: ids past n_full are pieces of split tiles (their
    // partial sums go to `part`, see the epilogue).  Thin tiles: the grid
    // covers logical tiles n_full .. n_full+split-1, each cut into BM/TM
    // token parts of each of its 2/NF feature parts (see thin_coords), with
    // every K-step.
    int tm, tn;
    int kbeg, nk;
    int64_t m0;
    int n0;
    if constexpr (TM == BM && NF == 2) {
        work_coords(blockIdx.x, tiles_m, tiles_n, GROUP_M, n_full, split, (R + BK - 1) / BK, tm, tn, kbeg, nk);
        m0 = (int64_t)tm * BM;
        n0 = tn * BN;
    } else {
        int u;
        thin_coords(blockIdx.x, tiles_m, tiles_n, GROUP_M, n_full, split, (BM / TM) * (2 / NF), tm, tn, u);
        kbeg = 0;
        nk = (R + BK - 1) / BK;
        m0 = (int64_t)tm * BM + (int64_t)(u % (BM / TM)) * TM;
        n0 = tn * BN + (u / (BM / TM)) * Lay::FT;
    }
    const int kofs = kbeg * BK;
    const int wprT = (R + 31) >> 5;  // words per row of M^T
    const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
    const uint8_t* zsrc = (const uint8_t*)g_zero_page + 16 * lane;
    // B-slab copy q of this wave lands at slab byte 1024*(4q + wave) + 16*lane,
    // i.e. row brow[q], physical chunk p; it carries logical chunk
    // bswz(brow, p) -- ranks 8*that .. +7 of B row k0 + brow[q] (rows of B are
    // ldb elements apart in memory), zeros for ranks at or past r
    int brow[Lay::NB], bcol[Lay::NB];
    bool bval[Lay::NB];
#pragma unroll
    for (int q = 0; q < Lay::NB; ++q) {
        const int blk = 4 * q + wave;
        const int off = 1024 * blk + 16 * lane;
        brow[q] = off / Lay::PITCH;
        const int lq = Lay::bswz(brow[q], (off % Lay::PITCH) / 16);
        bcol[q] = 16 * lq;
        bval[q] = blk < Lay::NBC && 8 * lq < r;
    }

    // M^T is a plain bitmap whatever the caller's layout.
    if (tid < 16) *(u32x2*)(smem + Lay::LUT + 8 * tid) = select_lut16_entry<false>((uint32_t)tid);


    // ---- slab copies.  Copies 0..ND-1: dY slab rows 8*(ND*wave + q) + lane/8
    // (64 k per row); copies ND..ND+NWC-1: this wave's W block, its 32 NF
    // columns (NF = 2: rows 8q + lane/8 in the tr64 layout; NF = 1: rows
    // 16q + lane/4, 16-byte chunk lane % 4); then the B slab and the M^T
    // words.
    uint32_t offD[Lay::ND], offW[Lay::NWC];
#pragma unroll
    for (int q = 0; q < Lay::ND; ++q) {
        const int rd = 8 * (Lay::ND * wave + q) + (lane >> 3);
        offD[q] = (uint32_t)((rd * R + 8 * ((lane & 7) ^ ((rd >> 1) & 7))) * 2);
    }
#pragma unroll
    for (int q = 0; q < Lay::NWC; ++q) {
        if constexpr (NF == 2) {
            const int rw = 8 * q + (lane >> 3);
            offW[q] = (uint32_t)((rw * C + 64 * wave + 8 * ((lane & 7) ^ tr64_swz(rw))) * 2);
        } else {
            const int rw = 16 * q + (lane >> 2);
            offW[q] = (uint32_t)((rw * C + 32 * wave + 8 * (lane & 3)) * 2);
        }
    }
    // M^T words of a K-step: with whole tiles the tile's columns hold them
    // as one contiguous run of 2 words per column (see mt_index), so copy q
    // of a wave moves 256 consecutive bytes of it
    uint32_t offM[Lay::NMC];
#pragma unroll
    for (int q = 0; q < Lay::NMC; ++q) offM[q] = (uint32_t)((64 * (Lay::NMC * wave + q) + lane) * 4);
    const uint16_t* Dt = uniform_ptr(dY + m0 * R);
    const uint16_t* Wn = uniform_ptr(W + n0);
    const uint32_t* Mn = uniform_ptr(Mt + 2 * (int64_t)n0);

    auto copy_j = [&](int j, int k0, uint32_t sb) {
        k0 += kofs;
        if (j < Lay::ND) {
            const int q = j, blk = Lay::ND * wave + q;
            const uint32_t dst = sb + Lay::D + 1024 * blk;
            if constexpr (!RAGGED) {
                copy16s_to_lds(uniform_ptr(Dt + k0), offD[q], dst);
            } else {
                const int row = 8 * blk + (lane >> 3);
                const int lc = (lane & 7) ^ ((row >> 1) & 7);
                const bool ok = m0 + row < L && k0 + 8 * lc < R;
                copy16_to_lds(ok ? (const void*)(Dt + (int64_t)row * R + k0 + 8 * lc) : (const void*)zsrc, dst);
            }
        } else if (j < Lay::ND + Lay::NWC) {
            if (PASS2) return;  // W is zero: its slabs were cleared once
            const int q = j - Lay::ND;
            const uint32_t dst = sb + Lay::W + Lay::WBW * wave + 1024 * q;
            if constexpr (!RAGGED) {
                copy16s_to_lds(uniform_ptr(Wn + (int64_t)k0 * C), offW[q], dst);
            } else {
                const int row = 8 * q + (lane >> 3);
                const int col = 64 * wave + 8 * ((lane & 7) ^ tr64_swz(row));
                const bool ok = k0 + row < R && n0 + col < C;
                copy16_to_lds(ok ? (const void*)(Wn + (int64_t)(k0 + row) * C + col) : (const void*)zsrc, dst);
            }
        } else if (j < Lay::ND + Lay::NWC + Lay::NB) {
            // the swizzled B slab of rows k0 .. k0+63; every wave issues NB
            // copies, those past the slab go to the sink
            const int q = j - Lay::ND - Lay::NWC, blk = 4 * q + wave;
            const bool real = blk < Lay::NBC;
            const bool ok = bval[q] && (!RAGGED || k0 + brow[q] < R);
            const void* src = (const uint8_t*)Bm + ((int64_t)k0 + brow[q]) * (2 * (int64_t)ldb) + bcol[q];
            copy16_to_lds(ok ? src : (const void*)zsrc, real ? sb + Lay::B + 1024 * blk : lds0 + Lay::SINK);
        } else {
            const int q = j - Lay::ND - Lay::NWC - Lay::NB;
            const uint32_t dst = sb + Lay::M + 256 * (Lay::NMC * wave + q);
            if constexpr (!RAGGED) {
                copy4s_to_lds(uniform_ptr(Mn + (int64_t)(k0 >> 5) * C), offM[q], dst);
            } else {
                const int e = 64 * (Lay::NMC * wave + q) + lane;
                const int n = e >> 1, gw = (k0 >> 5) + (e & 1);
                const bool ok = n0 + n < C && gw < wprT;
                copy4_to_lds(ok ? (const void*)(Mt + mt_index(n0 + n, gw, C, wprT)) : (const void*)zsrc, dst);
            }
        }
    };

    // Rows of the merge A operand: lane (rho = l32, h) reads B row pi(rho).
    const int rho = l32;
    const int pik = 16 * (rho >> 4) + 8 * ((rho >> 2) & 1) + 4 * ((rho >> 3) & 1) + (rho & 3);
    const int ncol0 = 32 * NF * wave + l32;
    // transpose-read offsets of the raw W fragments in this wave's W block,
    // sub-step 0 (sub-step c4 is 16 rows further): group g of 16 lanes reads
    // rows 8(g/2) + 4t + 0..3, columns 32nb + 16(g%2) + 0..15
    int offWt[NF][2];
    {
        const int g = lane >> 4, jj = lane & 15;
#pragma unroll
        for (int nb = 0; nb < NF; ++nb)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const int row = 8 * (g >> 1) + 4 * t + (jj >> 2), col = 32 * nb + 16 * (g & 1) + 4 * (jj & 3);
                offWt[nb][t] = Lay::W + Lay::WBW * wave + (NF == 2 ? tr64_elem_off(row, col) : row * Lay::WROW + 2 * col);
            }
    }
    auto doff = [&](int mb, int c4) { return Lay::D + slab64_off(32 * mb + l32, 2 * c4 + h); };

    f32x16 acc[MBW][NF];
#pragma unroll
    for (int i = 0; i < MBW; ++i)
#pragma unroll
        for (int j = 0; j < NF; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    bf16x8 da[MBW], db[MBW];  // dY fragments of alternate sub-steps
    u32x4 wa[NF], wb[NF];     // W' fragments of alternate sub-steps
    f32x16 T[NF];             // rank-r block of the current 32-wide k half
    uint32_t mw[NF][2];       // M^T words [nb][kb] of the current K-step
    u32x4 raw[NF], sel[NF];
    u32x4 rwa[NF], rwb[NF];   // folded merge: W of the two sub-steps of a k half
    bf16x8 bfr[RK];           // B[32kb + pi(rho)][16c + 8h .. +7]
    bf16x8 afr[NF][RK];       // A[16c + 8h .. +7][n] (scaled by s when the merge is folded)

    // MFMA slot i of a sub-step: token block i/2, feature block i%2 (the
    // slots of token and feature blocks a thin tile lacks are empty)
    auto mm = [&](int i, const bf16x8 (&df)[MBW], const u32x4 (&wf)[NF]) {
        const int mb = i >> 1, nb = i & 1;
        if (mb < MBW && nb < NF) acc[mb][nb] = mfma_32x32x16(df[mb], as_bf16x8(wf[nb]), acc[mb][nb]);
    };
    // ranks 16c + 8h .. +7 of B row 32kb + pik; the slab holds zeros for
    // ranks at or past r, so the read needs no per-lane test (a lane-dependent
    // branch would split the loop body and undo its per-slot schedule)
    auto read_bfr = [&](const uint8_t* sb, int kb) {
        const int k = 32 * kb + pik;
#pragma unroll
        for (int c = 0; c < RK; ++c)
            bfr[c] = *(const bf16x8*)(sb + Lay::B + k * Lay::PITCH + 16 * Lay::bswz(k, 2 * c + h));
    };
    auto read_mw = [&](const uint8_t* sb) {
#pragma unroll
        for (int nb = 0; nb < NF; ++nb) {
            const u32x2 v = *(const u32x2*)(sb + Lay::M + 8 * (ncol0 + 32 * nb));
            mw[nb][0] = v[0];
            mw[nb][1] = v[1];
        }
    };
    auto read_rs = [&](const uint8_t* sb, int c4) {
#pragma unroll
        for (int nb = 0; nb < NF; ++nb) {
            const u32x2 lo = lds_tr_read(sb + offWt[nb][0] + 16 * c4 * Lay::WROW);
            const u32x2 hi = lds_tr_read(sb + offWt[nb][1] + 16 * c4 * Lay::WROW);
            raw[nb][0] = lo[0];
            raw[nb][1] = lo[1];
            raw[nb][2] = hi[0];
            raw[nb][3] = hi[1];
            sel[nb] = read_sel16(smem + Lay::LUT, mw[nb][c4 >> 1], 8 * (2 * (c4 & 1) + h));
        }
    };
    auto read_d2 = [&](bf16x8 (&df)[MBW], const uint8_t* sb, int c4, int p) {
        if (2 * p < MBW) df[2 * p] = *(const bf16x8*)(sb + doff(2 * p, c4));
        if (2 * p + 1 < MBW) df[2 * p + 1] = *(const bf16x8*)(sb + doff(2 * p + 1, c4));
    };
    auto merge_piece = [&](u32x4 (&wf)[NF], int p, int cp) {
        const int nb = p >> 2, q = p & 3;
        if (nb < NF)
            wf[nb][q] = merge_pair(raw[nb][q], T[nb][8 * cp + 2 * q], T[nb][8 * cp + 2 * q + 1], s, sel[nb][q]);
    };
    // folded merge (see the forward kernel): raw W of sub-step c4, its select
    // masks, the unpack of a W pair into the rank-r accumulator, the merge
    auto read_raw = [&](u32x4 (&rw)[NF], const uint8_t* sb, int c4) {
#pragma unroll
        for (int nb = 0; nb < NF; ++nb) {
            const u32x2 lo = lds_tr_read(sb + offWt[nb][0] + 16 * c4 * Lay::WROW);
            const u32x2 hi = lds_tr_read(sb + offWt[nb][1] + 16 * c4 * Lay::WROW);
            rw[nb][0] = lo[0];
            rw[nb][1] = lo[1];
            rw[nb][2] = hi[0];
            rw[nb][3] = hi[1];
        }
    };
    auto read_sel = [&](int c4) {
#pragma unroll
        for (int nb = 0; nb < NF; ++nb) {
            sel[nb] = read_sel16(smem + Lay::LUT, mw[nb][c4 >> 1], 8 * (2 * (c4 & 1) + h));
        }
    };
    auto unpack = [&](const u32x4 (&rw)[NF], int cp, int p) {
        const int nb = p >> 2, q = p & 3;
        if (nb < NF) {
            T[nb][8 * cp + 2 * q] = __uint_as_float(rw[nb][q] << 16);
            T[nb][8 * cp + 2 * q + 1] = __uint_as_float(rw[nb][q] & 0xFFFF0000u);
        }
    };
    auto merge_fold = [&](u32x4 (&wf)[NF], int p, int cp) {
        const int nb = p >> 2, q = p & 3;
        if (nb < NF) wf[nb][q] = pack_bf16x2(T[nb][8 * cp + 2 * q], T[nb][8 * cp + 2 * q + 1]) & sel[nb][q];
    };
    // late_*: the copies EARLY.. of the stage in the other buffer, issued in
    // the merge slots of the first sub-step of a K-step (see the main loop)
    auto substep = [&](const bf16x8 (&dc)[MBW], const u32x4 (&wc)[NF], bf16x8 (&dn)[MBW], u32x4 (&wn)[NF],
                       const uint8_t* sb, int c4n, auto rank_tag, int late_k = 0, uint32_t late_sq = 0,
                       bool late_on = false) {
        constexpr bool RANK = decltype(rank_tag)::value;
        mm(0, dc, wc); read_rs(sb, c4n); SLOT_END();
        mm(1, dc, wc); if constexpr (RANK) read_bfr(sb, 1); SLOT_END();
        mm(2, dc, wc); read_d2(dn, sb, c4n, 0); SLOT_END();
        mm(3, dc, wc); read_d2(dn, sb, c4n, 1); SLOT_END();
        mm(4, dc, wc); read_d2(dn, sb, c4n, 2); SLOT_END();
        mm(5, dc, wc); read_d2(dn, sb, c4n, 3); SLOT_END();
        mm(6, dc, wc); SLOT_END();
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            mm(7 + p, dc, wc);
            merge_piece(wn, p, c4n & 1);
            if (late_on && Lay::EARLY + p < Lay::COPIES) copy_j(Lay::EARLY + p, late_k, late_sq);
            SLOT_END();
        }
        mm(15, dc, wc);
        if constexpr (RANK) rank_mfma2<RK>(T, bfr, afr);  // after the merge pieces read T
        SLOT_END();
    };
    // the sub-steps with the folded merge (schedule as in the forward)
    auto substep_fold = [&](const bf16x8 (&dc)[MBW], const u32x4 (&wc)[NF], bf16x8 (&dn)[MBW], u32x4 (&wn)[NF],
                            const uint8_t* sb, const uint8_t* snext, int c4n, int late_k = 0,
                            uint32_t late_sq = 0, bool late_on = false) {
        const int cp = c4n & 1;
        mm(0, dc, wc); read_sel(c4n); if (c4n == 1) read_raw(rwa, sb, 2); SLOT_END();
        mm(1, dc, wc); if (c4n == 1) { read_bfr(sb, 1); read_raw(rwb, sb, 3); } SLOT_END();
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            mm(2 + i, dc, wc);
            read_d2(dn, sb, c4n, i);
            if (c4n == 1) { unpack(rwa, 0, 2 * i); unpack(rwa, 0, 2 * i + 1); }
            if (c4n == 3 && i == 3) {
                wait_vmcnt<Lay::NB + Lay::NMC>();  // this wave's W copies of the next stage
                read_raw(rwa, snext, 0);
                read_raw(rwb, snext, 1);
            }
            SLOT_END();
        }
        mm(6, dc, wc); SLOT_END();
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            mm(7 + p, dc, wc);
            merge_fold(wn, p, cp);
            if (c4n == 1) unpack(rwb, 1, p);
            if (c4n == 3) { unpack(rwb, 1, p); unpack(rwa, 0, p); }
            if (late_on && Lay::EARLY + p < Lay::COPIES) copy_j(Lay::EARLY + p, late_k, late_sq);
            SLOT_END();
        }
        mm(15, dc, wc);
        if (c4n == 1) rank_mfma2_acc<RK>(T, bfr, afr);  // after the merge pieces read T
        SLOT_END();
    };

    if constexpr (PASS2) {  // W taken as zero: clear both W slabs once, never copy them
        for (int i = tid; i < 2 * (Lay::WB / 16); i += NT)
            *(u32x4*)(smem + (i / (Lay::WB / 16)) * Lay::STAGE + Lay::W + 16 * (i % (Lay::WB / 16))) = zero_u32x4();
        __syncthreads();
    }

    // ---- prologue.  The A block of the merge goes to stage 1's dY region
    // while stage 0 is copied; once both landed, the A block is read into
    // registers and stage 1 is copied over it (the first K-step's barrier
    // waits for stage 1), so the two round trips to memory overlap.
    // A[:, n0 .. n0+255] (16*RK rows) -> stage 1's dY region
#pragma unroll
    for (int q = 0; q < 2 * RK; ++q) {
        const int blk = 4 * q + wave;
        const int row = 2 * blk + h;
        const int lc = swz_chunk(row, lane & 31);
        const int gn = n0 + 8 * lc;
        copy16_to_lds((row < ra && gn < C) ? (const void*)(Am + (int64_t)row * C + gn) : (const void*)zsrc,
                      lds0 + Lay::STAGE + 1024 * blk);
    }
#pragma unroll
    for (int j = 0; j < Lay::COPIES; ++j) copy_j(j, 0, lds0);
    stage_barrier<0>();
    // the merge's B operand A[16c + 8h + e][n] into registers via transpose loads
#pragma unroll
    for (int nb = 0; nb < NF; ++nb)
#pragma unroll
        for (int c = 0; c < RK; ++c)
            afr[nb][c] = frag_from_tr(lds_tr_read(smem + Lay::STAGE + tr_frag_off(lane, 16 * c, 32 * NF * wave + 32 * nb, 0)),
                                      lds_tr_read(smem + Lay::STAGE + tr_frag_off(lane, 16 * c, 32 * NF * wave + 32 * nb, 1)));
    if constexpr (FOLD) {  // s.A, exact for a power-of-two s
#pragma unroll
        for (int nb = 0; nb < NF; ++nb)
#pragma unroll
            for (int c = 0; c < RK; ++c) {
                u32x4 v = __builtin_bit_cast(u32x4, afr[nb][c]);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    v[e] = pack_bf16x2(s * __uint_as_float(v[e] << 16), s * __uint_as_float(v[e] & 0xFFFF0000u));
                afr[nb][c] = as_bf16x8(v);
            }
    }
    lds_barrier();
#pragma unroll
    for (int j = 0; j < Lay::COPIES; ++j) copy_j(j, nk > 1 ? BK : 0, lds0 + Lay::STAGE);
    read_mw(smem);
    read_bfr(smem, 0);
    if constexpr (FOLD) {
        read_raw(rwa, smem, 0);
        read_raw(rwb, smem, 1);
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            unpack(rwa, 0, p);
            unpack(rwb, 1, p);
        }
        rank_mfma2_acc<RK>(T, bfr, afr);
        read_sel(0);
    } else {
        rank_mfma2<RK>(T, bfr, afr);
        read_rs(smem, 0);
    }
#pragma unroll
    for (int p = 0; p < 4; ++p) read_d2(da, smem, 0, p);
#pragma unroll
    for (int p = 0; p < 8; ++p) {
        if constexpr (FOLD) merge_fold(wa, p, 0);
        else merge_piece(wa, p, 0);
    }

    // ---- main loop (branch-free, see the forward kernel)
    for (int kt = 0; kt < nk; ++kt) {
        const int st = kt & 1;
        const uint8_t* sb = smem + st * Lay::STAGE;
        const uint8_t* sn = smem + (st ^ 1) * Lay::STAGE;
        // copies EARLY.. of stage kt+1 (buffer st^1, free since the last
        // barrier; the barrier below waits for them); at kt = 0 the prologue
        // issued all of stage 1
        const int k1 = (kt + 1 < nk ? kt + 1 : nk - 1) * BK;
        if constexpr (FOLD) {
            substep_fold(da, wa, db, wb, sb, sn, 1, k1, lds0 + (st ^ 1) * Lay::STAGE, kt > 0);
            substep_fold(db, wb, da, wa, sb, sn, 2);
            substep_fold(da, wa, db, wb, sb, sn, 3);
        } else {
            substep(da, wa, db, wb, sb, 1, std::true_type{}, k1, lds0 + (st ^ 1) * Lay::STAGE, kt > 0);
            substep(db, wb, da, wa, sb, 2, std::false_type{});
            substep(da, wa, db, wb, sb, 3, std::false_type{});
        }
        stage_barrier<0>();
        const int k2 = (kt + 2 < nk ? kt + 2 : nk - 1) * BK;
        const uint32_t sq = lds0 + st * Lay::STAGE;
        // one copy per MFMA slot: a copy issued behind an MFMA stalls the
        // wave while that MFMA runs, a second one would stall the next
        auto early = [&](int j) {
            if (j < Lay::EARLY) copy_j(j, k2, sq);
        };
        mm(0, db, wb); read_mw(sn); read_bfr(sn, 0); early(0); SLOT_END();
        mm(1, db, wb); early(1); SLOT_END();
        mm(2, db, wb); read_d2(da, sn, 0, 0); early(2); SLOT_END();
        mm(3, db, wb); read_d2(da, sn, 0, 1); early(3); SLOT_END();
        mm(4, db, wb);
        if constexpr (FOLD) read_sel(0);
        else read_rs(sn, 0);
        early(4); SLOT_END();
        mm(5, db, wb); read_d2(da, sn, 0, 2); early(5); SLOT_END();
        mm(6, db, wb); read_d2(da, sn, 0, 3);
        if constexpr (FOLD) rank_mfma2_acc<RK>(T, bfr, afr);
        else rank_mfma2<RK>(T, bfr, afr);
        early(6); SLOT_END();
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            mm(7 + p, db, wb);
            if constexpr (FOLD) merge_fold(wa, p, 0);
            else merge_piece(wa, p, 0);
            early(7 + p);
            SLOT_END();
        }
        mm(15, db, wb);
        SLOT_END();
    }
    // ---- epilogue: round to bf16, stage the wave's TM x 32 NF block in LDS
    // (rows of 32 NF outputs), then 16-byte stores of whole rows.
    wait_vmcnt<0>();
    lds_barrier();  // every wave's copies landed and every read of the stages done
    if (TM == BM && NF == 2 && (int)blockIdx.x >= n_full) {
        // a piece of a split tile: its unrounded fp32 partial sums go to slice
        // blockIdx.x - n_full of `part` (256 tokens x 256 features); the
        // reduction launch adds the pieces in order and rounds once
        float* dst = part + (int64_t)((int)blockIdx.x - n_full) * (BM * BN);
#pragma unroll
        for (int nb = 0; nb < NF; ++nb)
#pragma unroll
            for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    dst[(32 * mb + 8 * (v >> 2) + 4 * h + (v & 3)) * BN + ncol0 + 32 * nb] = acc[mb][nb][v];
        return;
    }
    constexpr int OW = 32 * NF;   // outputs per staged row
    constexpr int CH = OW / 8;    // 16-byte chunks per row
    uint16_t* ol = (uint16_t*)(smem + wave * (TM * OW * 2));
#pragma unroll
    for (int nb = 0; nb < NF; ++nb)
#pragma unroll
        for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                ol[(32 * mb + 8 * (v >> 2) + 4 * h + (v & 3)) * OW + 32 * nb + l32] = bf16_bits(acc[mb][nb][v]);
#pragma unroll 4
    for (int it = 0; it < TM * CH / 64; ++it) {
        const int row = (64 / CH) * it + lane / CH, ch = lane % CH;
        const u32x4 v = *(const u32x4*)(ol + row * OW + 8 * ch);
        const int64_t gm = m0 + row;
        const int gn = n0 + OW * wave + 8 * ch;
        if (gm < L && gn < C) {
            if constexpr (PASS2)
                *(u32x4*)(dX + gm * C + gn) = add_bf16x8(*(const u32x4*)(dX + gm * C + gn), v);
            else
                *(u32x4*)(dX + gm * C + gn) = v;
        }
    }
}

// s.A is exact in bf16 for a power-of-two s; the folded merge needs that
bool power_of_two(float s) {
    int e = 0;
    const float m = std::frexp(s, &e);
    return m == 0.5f || m == -0.5f;
}

// z0, z1: dB (R x rank) and dA (rank x C) to clear, or null
template <int RK, bool RAGGED, bool PASS2, bool FOLD, int TM, int NF>
void launch_tm(const LayerArgs& a, hipStream_t st, int ldb, int ra, int grid, int tiles_m, int tiles_n, int n_full,
               int split, float* part, float* z0, int64_t nz0, float* z1, int64_t nz1) {
    hipLaunchKernelGGL((dx_kernel<RK, RAGGED, PASS2, FOLD, TM, NF>), dim3(grid), dim3(NT), 0, st, (const uint16_t*)a.dY,
                       (const uint16_t*)a.W, a.Mt, (const uint16_t*)a.B, (const uint16_t*)a.A, (uint16_t*)a.dX, a.L,
                       (int)a.R, (int)a.C, (int)a.r, ra, a.scale, tiles_m, tiles_n, ldb, z0, nz0, z1, nz1, n_full,
                       split, part);
}

#ifndef LORS_THIN_TILES

template <int RK, bool PASS2>
hipError_t launch_rk(const LayerArgs& a, hipStream_t st, int ldb, int ra, bool clear) {
    const int tiles_m = (int)((a.L + BM - 1) / BM);
    const int tiles_n = (int)((a.C + BN - 1) / BN);
    const int tiles = tiles_m * tiles_n;
    // fixed-offset copies: whole tiles and K-steps, and per-lane byte
    // offsets (256 dY rows of R, 64 W rows of C, 256 M^T rows) inside 32 bits
    const bool ragged = !dx_whole_tiles(a.L, a.R, a.C);
    const bool fold = !ragged && power_of_two(a.scale);  // whole tiles with a power-of-two scale
    // A short last wave on a whole-tile shape runs as thin tiles (the same
    // bits, no workspace); on other shapes it is cut over K when the caller
    // gave room for the pieces' partial sums (one pass only: ranks up to 64).
    const ThinPlan tp = (!ragged && !PASS2) ? thin_plan(tiles) : ThinPlan{tiles, 0, 1};
    TailSplit sp{tiles, 1, tiles};
    if (tp.q == 1 && a.split_ws != nullptr && !PASS2 && ldb <= 64)
        sp = tail_split(tiles, (a.R + BK - 1) / BK, a.split_budget);
    float* part = sp.split > 1 ? (float*)a.split_ws : nullptr;
    // with thin tiles the whole-tile grid is exactly the first n_full tiles
    // (work_coords regroups ids over the tiles it is told the grid holds)
    const int grid = tp.q > 1 ? tp.n_full : sp.grid;
    const int n_full = tp.q > 1 ? tp.n_full : sp.n_full;
    // clear: dB (R x rank) and dA (rank x C) of the caller's problem, by the
    // first launch of this call
    const bool clear_here = clear && grid > 0;
    float* z0 = clear_here ? a.dB : nullptr;
    float* z1 = clear_here ? a.dA : nullptr;
    const int64_t nz0 = clear_here ? a.R * a.r_grad : 0, nz1 = clear_here ? a.r_grad * a.C : 0;
    if (grid > 0) {
        if (ragged)
            launch_tm<RK, true, PASS2, false, BM, 2>(a, st, ldb, ra, grid, tiles_m, tiles_n, n_full, sp.split, part, z0,
                                                  nz0, z1, nz1);
        else if (fold)
            launch_tm<RK, false, PASS2, true, BM, 2>(a, st, ldb, ra, grid, tiles_m, tiles_n, n_full, sp.split, part, z0,
                                                  nz0, z1, nz1);
        else
            launch_tm<RK, false, PASS2, false, BM, 2>(a, st, ldb, ra, grid, tiles_m, tiles_n, n_full, sp.split, part,
                                                   z0, nz0, z1, nz1);
    }
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && tp.q > 1)
        e = launch_dx_thin_bf16(a, st, ldb, ra, tp.n_full, tp.tail, tp.q, clear && !clear_here);
    if (e == hipSuccess && sp.split > 1)
        e = launch_split_reduce_bf16(part, sp.n_full, sp.split, tiles_m, tiles_n, GROUP_M, a.L, (int)a.C, nullptr,
                                     a.dX, st);
    return e;
}

// a.r: the (padded) rank of this pass; ra: the rows of A that exist
// The first pass clears dB and dA when the caller asks for it (a.clear_grads).
hipError_t launch_ranks(const LayerArgs& a, hipStream_t st, bool pass2, int ldb, int ra) {
    const bool c = a.clear_grads && !pass2;
    switch ((a.r + 15) / 16) {
        case 1: return pass2 ? launch_rk<1, true>(a, st, ldb, ra, false) : launch_rk<1, false>(a, st, ldb, ra, c);
        case 2: return pass2 ? launch_rk<2, true>(a, st, ldb, ra, false) : launch_rk<2, false>(a, st, ldb, ra, c);
        case 3: return pass2 ? launch_rk<3, true>(a, st, ldb, ra, false) : launch_rk<3, false>(a, st, ldb, ra, c);
        case 4: return pass2 ? launch_rk<4, true>(a, st, ldb, ra, false) : launch_rk<4, false>(a, st, ldb, ra, c);
        default: return hipErrorInvalidValue;
    }
}

#else  // LORS_THIN_TILES

// thin tiles of one feature half (NF = 1) and TM tokens: 2 BM / TM per tile
template <int RK, bool FOLD, int TM>
hipError_t launch_thin_tm(const LayerArgs& a, hipStream_t st, int ldb, int ra, int first, int tail, bool clear) {
    const int tiles_m = (int)((a.L + BM - 1) / BM);
    const int tiles_n = (int)((a.C + BN - 1) / BN);
    float* z0 = clear ? a.dB : nullptr;
    float* z1 = clear ? a.dA : nullptr;
    const int64_t nz0 = clear ? a.R * a.r_grad : 0, nz1 = clear ? a.r_grad * a.C : 0;
    launch_tm<RK, false, false, FOLD, TM, 1>(a, st, ldb, ra, tail * (2 * BM / TM), tiles_m, tiles_n, first, tail, nullptr,
                                          z0, nz0, z1, nz1);
    return hipGetLastError();
}

template <int RK, bool FOLD>
hipError_t launch_thin_q(const LayerArgs& a, hipStream_t st, int ldb, int ra, int first, int tail, int q,
                         bool clear) {
    switch (q) {  // q thin tiles per tile: two feature halves, each cut into q/2 token parts
        case 2: return launch_thin_tm<RK, FOLD, BM>(a, st, ldb, ra, first, tail, clear);
        case 4: return launch_thin_tm<RK, FOLD, BM / 2>(a, st, ldb, ra, first, tail, clear);
        case 8: return launch_thin_tm<RK, FOLD, BM / 4>(a, st, ldb, ra, first, tail, clear);
        default: return hipErrorInvalidValue;
    }
}

template <int RK>
hipError_t launch_thin_rk(const LayerArgs& a, hipStream_t st, int ldb, int ra, int first, int tail, int q,
                          bool clear) {
    return power_of_two(a.scale) ? launch_thin_q<RK, true>(a, st, ldb, ra, first, tail, q, clear)
                                 : launch_thin_q<RK, false>(a, st, ldb, ra, first, tail, q, clear);
}

#endif  // LORS_THIN_TILES

}  // namespace

#ifdef LORS_THIN_TILES

hipError_t launch_dx_thin_bf16(const LayerArgs& a, hipStream_t st, int ldb, int ra, int first, int tail, int q,
                               bool clear) {
    if (tail <= 0) return hipSuccess;
    // a.r: this pass's rank, a multiple of 8 up to 64 (see launch_dx_bf16)
    if (!dx_whole_tiles(a.L, a.R, a.C) || a.r < 8 || a.r > 64 || a.r % 8 != 0) return hipErrorInvalidValue;
    switch ((a.r + 15) / 16) {
        case 1: return launch_thin_rk<1>(a, st, ldb, ra, first, tail, q, clear);
        case 2: return launch_thin_rk<2>(a, st, ldb, ra, first, tail, q, clear);
        case 3: return launch_thin_rk<3>(a, st, ldb, ra, first, tail, q, clear);
        case 4: return launch_thin_rk<4>(a, st, ldb, ra, first, tail, q, clear);
        default: return hipErrorInvalidValue;
    }
}

#else

hipError_t launch_dx_bf16(const LayerArgs& a, hipStream_t st) {
    if (a.L == 0 || a.dX == nullptr) return hipSuccess;
    if (a.Mt == nullptr || a.r < 1 || a.r > 128) return hipErrorInvalidValue;
    // The B slab is copied in whole 16-byte chunks of its rows.  A rank that
    // is not a multiple of 8 works on a copy of B whose rows are padded with
    // zero columns to rp = roundup8(r); the missing A rows are read as zero.
    LayerArgs ap = a;
    const int rp = (int)((a.r + 7) / 8 * 8);
    if (rp != a.r) {
        if (a.b_pad == nullptr) return hipErrorInvalidValue;
        const hipError_t e = launch_pad_cols_bf16(a.B, a.R, a.r, rp, a.b_pad, st);
        if (e != hipSuccess) return e;
        ap.B = a.b_pad;
        ap.r = rp;
    }
    if (rp <= 64) return launch_ranks(ap, st, false, rp, (int)a.r);
    // Ranks above 64: two passes over the ranks [0, 64) and [64, r), the
    // second with W taken as zero and its product added onto dX (the mask
    // distributes over the sum; one more bf16 rounding of dX).
    LayerArgs a1 = ap;
    a1.r = 64;
    const hipError_t e = launch_ranks(a1, st, false, rp, 64);
    if (e != hipSuccess) return e;
    LayerArgs a2 = ap;
    a2.r = rp - 64;
    a2.B = (const uint16_t*)ap.B + 64;
    a2.A = (const uint16_t*)a.A + 64 * a.C;
    return launch_ranks(a2, st, true, rp, (int)a.r - 64);
}

#endif  // LORS_THIN_TILES

}  // namespace lors
