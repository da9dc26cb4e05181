// Fused forward of the sparsity-preserved LoRA linear, bf16 on gfx950.
//
//   Y[L x R] = X[L x C] . W'^T,   W' = select(M, W + s.B.A, 0)
//
// (Eq. 3 of Section 2.2 and Algorithm 1, with the listing's scale factor.)
// W' never reaches HBM, and never even reaches LDS: each of the 4 waves owns
// 64 output features (n) of the 256 x 256 tile and rebuilds exactly those 64
// rows of W' in registers, in the operand layout of the main MFMA.
//
// Merge: the rank-r product T = B.A for a 32(k) x 32(n) block is one
// 32x32x16 MFMA per 16 ranks whose A operand is A^T with its 32 rows taken in
// the order pi(8i + 4h + q) = 16(i/2) + 8h + 4(i%2) + q.  With that order the
// 16 accumulator values a lane holds are, in register order, the k values
// 16c + 8h + {0..7} for c = 0, 1 -- exactly two 32x32x16 B-operand fragments.
// Each lane then adds its W values (one 16-byte LDS read per fragment), picks
// the select masks for its eight k from a 16-entry table indexed by the two
// nibbles of the mask byte (128 bytes on distinct LDS banks, so the reads of
// a wave never conflict), rounds once to bf16, and feeds the MFMA directly.
//
// Schedule.  A K-step (64 k) is four sub-steps of 16 k.  While the 16 MFMAs
// of sub-step c run, the wave reads the X fragments of sub-step c+1 and
// builds its W' fragments; every MFMA slot carries a fixed share of that work
// (sched_barrier fences), so the matrix pipe never waits for a burst of
// merge arithmetic.  The rank-r product of the second half of a K-step is
// formed during sub-step 0.  One barrier per K-step, before sub-step 3:
// after it the next stage is visible and the current one is free, so
// sub-step 3 interleaves the first twelve copies of stage kt+2 and the first
// sub-step of stage kt+1 with its MFMAs (those copies have more than a
// K-step to land); the remaining copies of stage kt+2 go out in the merge
// slots of the first sub-step of the next K-step, three sub-steps ahead of
// the barrier that waits for them.  A wave stalls on a burst of
// asynchronous copies, so spreading them keeps the matrix pipe fed.  X, W, A
// and mask slabs travel HBM -> LDS with global_load_lds; accumulators
// (256 x 64 per wave) live in AGPRs.
//
// Folded merge (FOLD, for a scale s that is a power of two): s.B is then
// exact in bf16, so the resident B operand is pre-scaled and the rank-r MFMA
// accumulates onto W itself -- its accumulator starts as the W values of the
// two sub-steps of a k half, unpacked to fp32 -- and a merge piece is only the
// rounding and the select.  W + s.B.A is still formed in fp32 and rounded
// once (the terms are added in another order).  The W slab rows a wave
// unpacks are the rows its own copies fill, so the next stage's W is read
// before the barrier, as soon as the wave's own W copies have landed.
#include "gemm_common.hpp"
#include "kernels.hpp"

#include <cmath>
#include <type_traits>

namespace lors {
namespace {

constexpr int NT = 256;
constexpr int BM = 256;   // tokens per tile
constexpr int BN = 256;   // output features per whole tile (64 per wave)
constexpr int BK = 64;    // input features per K-step
constexpr int GROUP_M = 4;
constexpr int kEarly = 12;  // copies of a stage issued right after the barrier; the rest a sub-step later

// TM: tokens per tile, NF: 32-feature blocks per wave -- BM and 2 for a whole
// tile; a thin tile of a short last wave has half the features (NF = 1) and
// TM = 256, 128 or 64 tokens
template <int RK, int TM, int NF>
struct Layout {
    static constexpr int FT = 128 * NF;           // output features per tile
    static constexpr int XB = TM * kRow64;        // X slab: TM rows of 64 k
    static constexpr int WB = FT * kRow64;        // W slab: FT rows of 64 k
    static constexpr int MB = FT * 2 * 4;         // 2 mask words per row of W
    static constexpr int AB = 16 * RK * kRow64;   // A slab: 16*RK rows of 64 k
    static constexpr int X = 0, W = XB, A = XB + WB, M = XB + WB + AB;
    static constexpr int STAGE = XB + WB + AB + MB;
    static constexpr int LUT = 2 * STAGE;         // select table: 16 x 8 B
    static constexpr int SINK = LUT + 256;        // 1 KiB target of padding copies
    static constexpr int TOTAL = SINK + 1024;
    static constexpr int NX = TM / 32;            // X-slab copies per wave
    static constexpr int NWC = 4 * NF;            // W-slab copies per wave
    static constexpr int NAW = (2 * RK + 3) / 4;  // A-slab copies per wave
    static constexpr int NMC = NF;                // mask copies per wave
    static constexpr int COPIES = NX + NWC + NAW + NMC;  // copies per wave per stage
    static constexpr int EARLY = COPIES < kEarly ? COPIES : kEarly;
    static_assert(COPIES - EARLY <= 8, "the late copies fit the eight merge slots");
};

#define SLOT_END() __builtin_amdgcn_sched_barrier(0)

// A^T slab (rank rows j of 64 k) in the tr64 layout: chunk c of row j is
// stored at chunk c ^ tr64_swz(j), because the merge reads it with transposed
// 4-row fragments (the X/W slabs' row-pair XOR would leave those reads 2-way
// conflicted).

// RAGGED: some tile reaches past L, R or C (copies then check every lane and
// read the zero page outside the tensors); otherwise every slab row and
// K-chunk is in range and copies use a uniform base plus fixed offsets.
// PASS2: the second pass of a rank above 64 (ranks 64.. of B and A): W is
// taken as zero and the product is added onto Y.  ldb: row stride of B.
// TM, NF < (BM, 2): a thin tile of TM tokens and 128 NF features
// (whole-tile shapes, one pass); each wave then holds TM x 32 NF
// accumulators, merges 32 NF rows of W', and the MFMA slots, X reads and
// merge pieces of the missing token and feature blocks drop out of the
// schedule.
template <int RK, bool TWO_FOUR, bool RAGGED, bool PASS2, bool FOLD, int TM, int NF>
__global__ __launch_bounds__(NT, 1) void fwd_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
    const uint32_t* __restrict__ Mp, const uint16_t* __restrict__ Bm,
    const uint16_t* __restrict__ Am, const uint16_t* __restrict__ bias,
    uint16_t* __restrict__ Y, int64_t L, int R, int C, int r, float s, int tiles_m,
    int tiles_n, int ldb, int n_full, int split, float* __restrict__ part) {
    using Lay = Layout<RK, TM, NF>;
    constexpr int MBW = TM / 32;  // 32-token blocks per wave
    static_assert((TM == BM && NF == 2) || (!RAGGED && !PASS2), "thin tiles: fixed-offset copies, one pass");
    static_assert(Lay::TOTAL <= 160 * 1024, "LDS budget");
    static_assert(4 * TM * 64 * NF <= 2 * Lay::STAGE, "output staging fits the stage buffers");
    __shared__ __attribute__((aligned(1024))) uint8_t smem[Lay::TOTAL];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31;
    const int h = lane >> 5;

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
        work_coords(blockIdx.x, tiles_m, tiles_n, GROUP_M, n_full, split, (C + BK - 1) / BK, tm, tn, kbeg, nk);
        m0 = (int64_t)tm * BM;
        n0 = tn * BN;
    } else {
        int u;
        thin_coords(blockIdx.x, tiles_m, tiles_n, GROUP_M, n_full, split, (BM / TM) * (2 / NF), tm, tn, u);
        kbeg = 0;
        nk = (C + BK - 1) / BK;
        m0 = (int64_t)tm * BM + (int64_t)(u % (BM / TM)) * TM;
        n0 = tn * BN + (u / (BM / TM)) * Lay::FT;
    }
    const int kofs = kbeg * BK;
    const int wpr = (C + 31) >> 5;
    const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
    const uint8_t* zsrc = (const uint8_t*)g_zero_page + 16 * (lane & 7);

    // ---- select table (visible to all waves after the first stage barrier)
    // and the resident B operand of the merge: column n = 64 wave + 32 nb + l32,
    // ranks 16c + 8h .. +7
    if (tid < 16) *(u32x2*)(smem + Lay::LUT + 8 * tid) = select_lut16_entry<TWO_FOUR>((uint32_t)tid);
    const bool b_vec = (r & 7) == 0 && (ldb & 7) == 0;
    bf16x8 bfr[NF][RK];
#pragma unroll
    for (int nb = 0; nb < NF; ++nb) {
        const int gn = n0 + 32 * NF * wave + 32 * nb + l32;
#pragma unroll
        for (int c = 0; c < RK; ++c) {
            u32x4 v = zero_u32x4();
            const int j0 = 16 * c + 8 * h;
            if (gn < R) {
                const uint16_t* src = Bm + (int64_t)gn * ldb + j0;
                if (b_vec) {
                    if (j0 < r) v = *(const u32x4*)src;
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        v[e >> 1] |= (j0 + e < r ? (uint32_t)src[e] : 0u) << ((e & 1) * 16);
                }
            }
            if constexpr (FOLD) {  // s.B, exact for a power-of-two s
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    v[e] = pack_bf16x2(s * __uint_as_float(v[e] << 16), s * __uint_as_float(v[e] & 0xFFFF0000u));
            }
            bfr[nb][c] = as_bf16x8(v);
        }
    }

    // ---- slab copies.  Copy q < NX of a wave fills X slab rows
    // 8*(NX*wave + q) + lane/8, copy NX + q (q < NWC) W slab rows
    // 8*(NWC*wave + q) + lane/8; lane l covers physical chunk l % 8 of its
    // row.  (With whole tiles NX = NWC = 8 and the two share their offsets.)
    uint32_t offX[Lay::NX], offW[Lay::NWC];
#pragma unroll
    for (int q = 0; q < Lay::NX; ++q) {
        const int row = 8 * (Lay::NX * wave + q) + (lane >> 3);
        const int lc = (lane & 7) ^ ((row >> 1) & 7);
        offX[q] = (uint32_t)((row * C + 8 * lc) * 2);
    }
#pragma unroll
    for (int q = 0; q < Lay::NWC; ++q) {
        const int row = 8 * (Lay::NWC * wave + q) + (lane >> 3);
        const int lc = (lane & 7) ^ ((row >> 1) & 7);
        offW[q] = (uint32_t)((row * C + 8 * lc) * 2);
    }
    // A slab: copy q of wave w is slab block 4q + w (rows 8 blk .. +7) when
    // that block exists; rows at or past r read zeros
    const uint16_t* aptr[Lay::NAW];
#pragma unroll
    for (int q = 0; q < Lay::NAW; ++q) {
        const int row = 8 * (4 * q + wave) + (lane >> 3);
        const int lc = (lane & 7) ^ tr64_swz(row);
        aptr[q] = Am + (int64_t)row * C + 8 * lc;
    }
    // mask words [row n][kb]: NMC 256-byte copies per wave
    uint32_t offM[Lay::NMC];
#pragma unroll
    for (int q = 0; q < Lay::NMC; ++q) {
        const int e = 64 * (Lay::NMC * wave + q) + lane;
        offM[q] = (uint32_t)(((e >> 1) * wpr + (e & 1)) * 4);
    }
    const uint16_t* Xt = uniform_ptr(X + m0 * C);
    const uint16_t* Wt = uniform_ptr(W + (int64_t)n0 * C);
    const uint32_t* Mt = uniform_ptr(Mp + (int64_t)n0 * wpr);

    // copy j of the stage at K offset k0 into the stage at LDS address sb
    auto copy_j = [&](int j, int k0, uint32_t sb) {
        k0 += kofs;
        if (j < Lay::NX + Lay::NWC) {
            const bool isx = j < Lay::NX;
            const int q = isx ? j : j - Lay::NX;
            if (PASS2 && !isx) return;  // W is zero: its slabs were cleared once
            const int blk = isx ? Lay::NX * wave + q : Lay::NWC * wave + q;
            const uint32_t dst = sb + (isx ? Lay::X : Lay::W) + 1024 * blk;
            if constexpr (!RAGGED) {
                copy16s_to_lds(uniform_ptr((isx ? Xt : Wt) + k0), isx ? offX[q] : offW[q], dst);
            } else {
                const int row = 8 * blk + (lane >> 3);
                const int lc = (lane & 7) ^ ((row >> 1) & 7);
                const bool ok = (isx ? m0 + row < L : n0 + row < R) && k0 + 8 * lc < C;
                const uint16_t* src = (isx ? Xt : Wt) + (int64_t)row * C + k0 + 8 * lc;
                copy16_to_lds(ok ? (const void*)src : (const void*)zsrc, dst);
            }
        } else if (j < Lay::NX + Lay::NWC + Lay::NAW) {
            // every wave issues NAW copies; those past the A slab go to the sink
            const int q = j - Lay::NX - Lay::NWC, blk = 4 * q + wave;
            const bool has = blk < 2 * RK;
            const int row = 8 * blk + (lane >> 3);
            const int lc = (lane & 7) ^ tr64_swz(row);
            const bool ok = has && row < r && (!RAGGED || k0 + 8 * lc < C);
            copy16_to_lds(ok ? (const void*)(aptr[q] + k0) : (const void*)zsrc,
                          has ? sb + Lay::A + 1024 * blk : lds0 + Lay::SINK);
        } else {
            const int q = j - Lay::NX - Lay::NWC - Lay::NAW;
            const uint32_t dst = sb + Lay::M + 256 * (Lay::NMC * wave + q);
            if constexpr (!RAGGED) {
                copy4s_to_lds(uniform_ptr(Mt + (k0 >> 5)), offM[q], dst);
            } else {
                const int e = 64 * (Lay::NMC * wave + q) + lane;
                const bool ok = n0 + (e >> 1) < R && (k0 >> 5) + (e & 1) < wpr;
                const uint32_t* src = Mt + (int64_t)(e >> 1) * wpr + (k0 >> 5) + (e & 1);
                copy4_to_lds(ok ? (const void*)src : (const void*)zsrc, dst);
            }
        }
    };

    // ---- per-lane LDS offsets
    // A^T operand of the merge, k rows in the order pi (see header): group g
    // of 16 lanes reads 4 rows j and 16 permuted k columns per transpose load.
    int offAt[2][2];  // [kb][t] for rank chunk 0 (add 16*128*c for chunk c)
    {
        const int g = lane >> 4, jj = lane & 15;
        const int sig = ((jj & 3) == 1) ? 2 : ((jj & 3) == 2) ? 1 : (jj & 3);
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const int row = 8 * (g >> 1) + 4 * t + (jj >> 2);
                const int col = 32 * kb + 16 * (g & 1) + 4 * sig;
                offAt[kb][t] = Lay::A + tr64_elem_off(row, col);
            }
    }
    const int nrow0 = 32 * NF * wave + l32;
    auto xoff = [&](int mb, int c4) { return Lay::X + slab64_off(32 * mb + l32, 2 * c4 + h); };
    auto woff = [&](int nb, int c4) { return Lay::W + slab64_off(nrow0 + 32 * nb, 2 * c4 + h); };

    f32x16 acc[MBW][NF];
#pragma unroll
    for (int i = 0; i < MBW; ++i)
#pragma unroll
        for (int j = 0; j < NF; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    bf16x8 xa[MBW], xb[MBW];  // X fragments of alternate sub-steps
    u32x4 wa[NF], wb[NF];     // W' fragments of alternate sub-steps
    f32x16 T[NF];             // rank-r block of the current 32-wide k half
    uint32_t mw[NF][2];       // mask words [nb][kb] of the current K-step
    u32x4 raw[NF], sel[NF];   // W and select masks of the sub-step being merged
    u32x4 rwa[NF], rwb[NF];   // folded merge: W of the two sub-steps of a k half
    bf16x8 afr[RK];

    // MFMA slot i of a sub-step: token block i/2, feature block i%2 (the
    // slots of token and feature blocks a thin tile lacks are empty)
    auto mm = [&](int i, const bf16x8 (&xf)[MBW], const u32x4 (&wf)[NF]) {
        const int mb = i >> 1, nb = i & 1;
        if (mb < MBW && nb < NF) acc[mb][nb] = mfma_32x32x16(xf[mb], as_bf16x8(wf[nb]), acc[mb][nb]);
    };
    auto read_afr = [&](const uint8_t* sb, int kb) {
#pragma unroll
        for (int c = 0; c < RK; ++c)
            afr[c] = frag_from_tr(lds_tr_read(sb + offAt[kb][0] + 16 * kRow64 * c),
                                  lds_tr_read(sb + offAt[kb][1] + 16 * kRow64 * c));
    };
    auto read_mw = [&](const uint8_t* sb) {
#pragma unroll
        for (int nb = 0; nb < NF; ++nb) {
            const u32x2 v = *(const u32x2*)(sb + Lay::M + 8 * (nrow0 + 32 * nb));
            mw[nb][0] = v[0];
            mw[nb][1] = v[1];
        }
    };
    // raw W and select masks of sub-step c4 of the stage at sb
    auto read_rs = [&](const uint8_t* sb, int c4) {
#pragma unroll
        for (int nb = 0; nb < NF; ++nb) {
            raw[nb] = *(const u32x4*)(sb + woff(nb, c4));
            sel[nb] = read_sel16(smem + Lay::LUT, mw[nb][c4 >> 1], 8 * (2 * (c4 & 1) + h));
        }
    };
    auto read_x2 = [&](bf16x8 (&xf)[MBW], const uint8_t* sb, int c4, int p) {
        if (2 * p < MBW) xf[2 * p] = *(const bf16x8*)(sb + xoff(2 * p, c4));
        if (2 * p + 1 < MBW) xf[2 * p + 1] = *(const bf16x8*)(sb + xoff(2 * p + 1, c4));
    };
    // merge piece p (0..7): pair p % 4 of fragment nb = p / 4, T half cp
    auto merge_piece = [&](u32x4 (&wf)[NF], int p, int cp) {
        const int nb = p >> 2, q = p & 3;
        if (nb < NF)
            wf[nb][q] = merge_pair(raw[nb][q], T[nb][8 * cp + 2 * q], T[nb][8 * cp + 2 * q + 1], s, sel[nb][q]);
    };
    // folded merge: W of sub-step c4 (raw bf16 pairs), select masks of c4
    auto read_raw = [&](u32x4 (&rw)[NF], const uint8_t* sb, int c4) {
#pragma unroll
        for (int nb = 0; nb < NF; ++nb) rw[nb] = *(const u32x4*)(sb + woff(nb, c4));
    };
    auto read_sel = [&](int c4) {
#pragma unroll
        for (int nb = 0; nb < NF; ++nb) {
            sel[nb] = read_sel16(smem + Lay::LUT, mw[nb][c4 >> 1], 8 * (2 * (c4 & 1) + h));
        }
    };
    // pair p of rw, as fp32, into the accumulator half cp of the rank-r block
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
    // an ordinary sub-step: MFMAs on (xc, wc) while preparing (xn, wn) for
    // sub-step c4n of the stage at sb; optionally the rank-r block of k half 1
    // late_*: the copies EARLY.. of the stage in the other buffer, issued in
    // the merge slots of the first sub-step of a K-step (see the main loop)
    auto substep = [&](const bf16x8 (&xc)[MBW], const u32x4 (&wc)[NF], bf16x8 (&xn)[MBW], u32x4 (&wn)[NF],
                       const uint8_t* sb, int c4n, auto rank_tag, int late_k = 0, uint32_t late_sq = 0,
                       bool late_on = false) {
        constexpr bool RANK = decltype(rank_tag)::value;
        mm(0, xc, wc); read_rs(sb, c4n); SLOT_END();
        mm(1, xc, wc); if constexpr (RANK) read_afr(sb, 1); SLOT_END();
        mm(2, xc, wc); read_x2(xn, sb, c4n, 0); SLOT_END();
        mm(3, xc, wc); read_x2(xn, sb, c4n, 1); SLOT_END();
        mm(4, xc, wc); read_x2(xn, sb, c4n, 2); SLOT_END();
        mm(5, xc, wc); read_x2(xn, sb, c4n, 3); SLOT_END();
        mm(6, xc, wc); SLOT_END();
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            mm(7 + p, xc, wc);
            merge_piece(wn, p, c4n & 1);
            if (late_on && Lay::EARLY + p < Lay::COPIES) copy_j(Lay::EARLY + p, late_k, late_sq);
            SLOT_END();
        }
        mm(15, xc, wc);
        if constexpr (RANK) rank_mfma2<RK>(T, afr, bfr);  // after the merge pieces read T
        SLOT_END();
    };
    // The same sub-step with the folded merge.  The accumulator T holds, per
    // k half, W + s.B.A of its two sub-steps (cp = 0, 1):
    //   sub-step 1 (RANK): merges sub-step 1 from T's cp 1 and refills it, pair
    //     by pair, with W of sub-step 3; W of sub-step 2 goes to cp 0 (free
    //     since the previous K-step's last merge); then the rank-r MFMAs of
    //     k half 1 accumulate onto both;
    //   sub-step 2: merges sub-step 2 from cp 0;
    //   sub-step 3: merges sub-step 3 from cp 1 and refills T with W of the
    //     next stage's sub-steps 0 and 1, read once this wave's own W copies
    //     of that stage have landed (no barrier needed: each wave copies the
    //     W rows it merges); the rank-r MFMAs of that k half run after the
    //     barrier.
    auto substep_fold = [&](const bf16x8 (&xc)[MBW], const u32x4 (&wc)[NF], bf16x8 (&xn)[MBW], u32x4 (&wn)[NF],
                            const uint8_t* sb, const uint8_t* snext, int c4n, int late_k = 0,
                            uint32_t late_sq = 0, bool late_on = false) {
        const int cp = c4n & 1;
        mm(0, xc, wc); read_sel(c4n); if (c4n == 1) read_raw(rwa, sb, 2); SLOT_END();
        mm(1, xc, wc); if (c4n == 1) { read_afr(sb, 1); read_raw(rwb, sb, 3); } SLOT_END();
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            mm(2 + i, xc, wc);
            read_x2(xn, sb, c4n, i);
            if (c4n == 1) { unpack(rwa, 0, 2 * i); unpack(rwa, 0, 2 * i + 1); }
            if (c4n == 3 && i == 3) {
                wait_vmcnt<Lay::NAW + Lay::NMC>();  // this wave's W copies of the next stage
                read_raw(rwa, snext, 0);
                read_raw(rwb, snext, 1);
            }
            SLOT_END();
        }
        mm(6, xc, wc); SLOT_END();
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            mm(7 + p, xc, wc);
            merge_fold(wn, p, cp);
            if (c4n == 1) unpack(rwb, 1, p);
            if (c4n == 3) { unpack(rwb, 1, p); unpack(rwa, 0, p); }
            if (late_on && Lay::EARLY + p < Lay::COPIES) copy_j(Lay::EARLY + p, late_k, late_sq);
            SLOT_END();
        }
        mm(15, xc, wc);
        if (c4n == 1) rank_mfma2_acc<RK>(T, afr, bfr);  // after the merge pieces read T
        SLOT_END();
    };

    if constexpr (PASS2) {  // W taken as zero: clear both W slabs once, never copy them
        for (int i = tid; i < 2 * (Lay::WB / 16); i += NT)
            *(u32x4*)(smem + (i / (Lay::WB / 16)) * Lay::STAGE + Lay::W + 16 * (i % (Lay::WB / 16))) = zero_u32x4();
        __syncthreads();
    }

    // ---- prologue: stages 0 and 1 in flight, then sub-step 0 of stage 0
#pragma unroll
    for (int j = 0; j < Lay::COPIES; ++j) copy_j(j, 0, lds0);
#pragma unroll
    for (int j = 0; j < Lay::COPIES; ++j) copy_j(j, nk > 1 ? BK : 0, lds0 + Lay::STAGE);
    // stage 0 landed everywhere (stage 1's copies, the last issued, may still
    // fly: the first K-step's barrier waits for them)
    stage_barrier<PASS2 ? Lay::COPIES - Lay::NWC : Lay::COPIES>();
    read_mw(smem);
    read_afr(smem, 0);
    if constexpr (FOLD) {
        read_raw(rwa, smem, 0);
        read_raw(rwb, smem, 1);
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            unpack(rwa, 0, p);
            unpack(rwb, 1, p);
        }
        rank_mfma2_acc<RK>(T, afr, bfr);
        read_sel(0);
    } else {
        rank_mfma2<RK>(T, afr, bfr);
        read_rs(smem, 0);
    }
#pragma unroll
    for (int p = 0; p < 4; ++p) read_x2(xa, smem, 0, p);
#pragma unroll
    for (int p = 0; p < 8; ++p) {
        if constexpr (FOLD) merge_fold(wa, p, 0);
        else merge_piece(wa, p, 0);
    }

    // ---- main loop (no data-dependent branches: at the tail the copies
    // repeat the last K-slab into the buffer just consumed, and the reads of
    // the "next" stage after the last K-step are never used)
    for (int kt = 0; kt < nk; ++kt) {
        const int st = kt & 1;
        const uint8_t* sb = smem + st * Lay::STAGE;
        const uint8_t* sn = smem + (st ^ 1) * Lay::STAGE;
        // copies EARLY.. of stage kt+1 (buffer st^1, free since the last
        // barrier; the barrier below waits for them); at kt = 0 the prologue
        // issued all of stage 1
        const int k1 = (kt + 1 < nk ? kt + 1 : nk - 1) * BK;
        if constexpr (FOLD) {
            substep_fold(xa, wa, xb, wb, sb, sn, 1, k1, lds0 + (st ^ 1) * Lay::STAGE, kt > 0);
            substep_fold(xb, wb, xa, wa, sb, sn, 2);
            substep_fold(xa, wa, xb, wb, sb, sn, 3);
        } else {
            substep(xa, wa, xb, wb, sb, 1, std::true_type{}, k1, lds0 + (st ^ 1) * Lay::STAGE, kt > 0);
            substep(xb, wb, xa, wa, sb, 2, std::false_type{});
            substep(xa, wa, xb, wb, sb, 3, std::false_type{});
        }
        // sub-step 3: stage kt+1 landed everywhere, stage kt free
        stage_barrier<0>();
        const int k2 = (kt + 2 < nk ? kt + 2 : nk - 1) * BK;
        const uint32_t sq = lds0 + st * Lay::STAGE;
        // one copy per MFMA slot: a copy issued behind an MFMA stalls the
        // wave while that MFMA runs, a second one would stall the next
        auto early = [&](int j) {
            if (j < Lay::EARLY) copy_j(j, k2, sq);
        };
        mm(0, xb, wb); read_mw(sn); read_afr(sn, 0); early(0); SLOT_END();
        mm(1, xb, wb); early(1); SLOT_END();
        mm(2, xb, wb); read_x2(xa, sn, 0, 0); early(2); SLOT_END();
        mm(3, xb, wb); read_x2(xa, sn, 0, 1); early(3); SLOT_END();
        mm(4, xb, wb);
        if constexpr (FOLD) read_sel(0);
        else read_rs(sn, 0);
        early(4); SLOT_END();
        mm(5, xb, wb); read_x2(xa, sn, 0, 2); early(5); SLOT_END();
        mm(6, xb, wb); read_x2(xa, sn, 0, 3);
        if constexpr (FOLD) rank_mfma2_acc<RK>(T, afr, bfr);
        else rank_mfma2<RK>(T, afr, bfr);
        early(6); SLOT_END();
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            mm(7 + p, xb, wb);
            if constexpr (FOLD) merge_fold(wa, p, 0);
            else merge_piece(wa, p, 0);
            early(7 + p);
            SLOT_END();
        }
        mm(15, xb, wb);
        SLOT_END();
    }
    // ---- epilogue: (+bias), round to bf16, stage the wave's TM x 32 NF block
    // in LDS (rows of 32 NF outputs), then 16-byte stores of whole rows.
    wait_vmcnt<0>();
    lds_barrier();  // every wave's copies landed and every read of the stages done
    if (TM == BM && NF == 2 && (int)blockIdx.x >= n_full) {
        // a piece of a split tile: its unrounded fp32 partial sums go to slice
        // blockIdx.x - n_full of `part` (256 tokens x 256 features); the
        // reduction launch adds the pieces in order, adds the bias and rounds
        float* dst = part + (int64_t)((int)blockIdx.x - n_full) * (BM * BN);
#pragma unroll
        for (int nb = 0; nb < NF; ++nb)
#pragma unroll
            for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    dst[(32 * mb + 8 * (v >> 2) + 4 * h + (v & 3)) * BN + nrow0 + 32 * nb] = acc[mb][nb][v];
        return;
    }
    constexpr int OW = 32 * NF;   // outputs per staged row
    constexpr int CH = OW / 8;    // 16-byte chunks per row
    uint16_t* ol = (uint16_t*)(smem + wave * (TM * OW * 2));
#pragma unroll
    for (int nb = 0; nb < NF; ++nb) {
        const int gn = n0 + nrow0 + 32 * nb;
        const float bv = (bias != nullptr && gn < R) ? bf16_bits_to_f32(bias[gn]) : 0.f;
#pragma unroll
        for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                ol[(32 * mb + 8 * (v >> 2) + 4 * h + (v & 3)) * OW + 32 * nb + l32] = bf16_bits(acc[mb][nb][v] + bv);
    }
#pragma unroll 4
    for (int it = 0; it < TM * CH / 64; ++it) {
        const int row = (64 / CH) * it + lane / CH, ch = lane % CH;
        const u32x4 v = *(const u32x4*)(ol + row * OW + 8 * ch);
        const int64_t gm = m0 + row;
        const int gn = n0 + OW * wave + 8 * ch;
        if (gm < L && gn < R) {
            if constexpr (PASS2)
                *(u32x4*)(Y + gm * R + gn) = add_bf16x8(*(const u32x4*)(Y + gm * R + gn), v);
            else
                *(u32x4*)(Y + gm * R + gn) = v;
        }
    }
}

// s.B is exact in bf16 for a power-of-two s (B's exponent shifts); the folded
// merge needs that.
bool power_of_two(float s) {
    int e = 0;
    const float m = std::frexp(s, &e);
    return m == 0.5f || m == -0.5f;
}

#ifndef LORS_THIN_TILES

template <int RK, bool TWO_FOUR, bool RAGGED, bool PASS2, bool FOLD>
void launch_whole(const LayerArgs& a, hipStream_t st, int ldb, int grid, int tiles_m, int tiles_n, int n_full,
                  int split, float* part) {
    hipLaunchKernelGGL((fwd_kernel<RK, TWO_FOUR, RAGGED, PASS2, FOLD, BM, 2>), dim3(grid), dim3(NT), 0, st,
                       (const uint16_t*)a.X, (const uint16_t*)a.W, a.M, (const uint16_t*)a.B,
                       (const uint16_t*)a.A, (const uint16_t*)a.bias, (uint16_t*)a.Y, a.L, (int)a.R, (int)a.C,
                       (int)a.r, a.scale, tiles_m, tiles_n, ldb, n_full, split, part);
}

template <int RK, bool TWO_FOUR, bool PASS2>
hipError_t launch_fmt(const LayerArgs& a, hipStream_t st, int ldb) {
    const int tiles_m = (int)((a.L + BM - 1) / BM);
    const int tiles_n = (int)((a.R + BN - 1) / BN);
    const int tiles = tiles_m * tiles_n;
    // the fixed-offset copies need every tile and K-step in range and the
    // per-lane byte offsets (256 slab rows of C bf16 or of the mask) inside
    // 32 bits
    const bool ragged = !fwd_whole_tiles(a.L, a.R, a.C);
    const bool fold = !ragged && power_of_two(a.scale);  // whole tiles with a power-of-two scale
    // A short last wave on a whole-tile shape runs as thin tiles (the same
    // bits, no workspace); on other shapes it is cut over K when the caller
    // gave room for the pieces' partial sums (one pass only: ranks up to 64).
    const ThinPlan tp = (!ragged && !PASS2) ? thin_plan(tiles) : ThinPlan{tiles, 0, 1};
    TailSplit sp{tiles, 1, tiles};
    if (tp.q == 1 && a.split_ws != nullptr && !PASS2 && a.r <= 64)
        sp = tail_split(tiles, (a.C + BK - 1) / BK, a.split_budget);
    float* part = sp.split > 1 ? (float*)a.split_ws : nullptr;
    // with thin tiles the whole-tile grid is exactly the first n_full tiles
    // (work_coords regroups ids over the tiles it is told the grid holds)
    const int grid = tp.q > 1 ? tp.n_full : sp.grid;
    const int n_full = tp.q > 1 ? tp.n_full : sp.n_full;
    if (grid > 0) {
        if (ragged)
            launch_whole<RK, TWO_FOUR, true, PASS2, false>(a, st, ldb, grid, tiles_m, tiles_n, n_full, sp.split,
                                                           part);
        else if (fold)
            launch_whole<RK, TWO_FOUR, false, PASS2, true>(a, st, ldb, grid, tiles_m, tiles_n, n_full, sp.split,
                                                           part);
        else
            launch_whole<RK, TWO_FOUR, false, PASS2, false>(a, st, ldb, grid, tiles_m, tiles_n, n_full, sp.split,
                                                            part);
    }
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && tp.q > 1) e = launch_fwd_thin_bf16(a, st, ldb, tp.n_full, tp.tail, tp.q);
    if (e == hipSuccess && sp.split > 1)
        e = launch_split_reduce_bf16(part, sp.n_full, sp.split, tiles_m, tiles_n, GROUP_M, a.L, (int)a.R, a.bias,
                                     a.Y, st);
    return e;
}

template <int RK>
hipError_t launch_rk(const LayerArgs& a, hipStream_t st, bool pass2, int ldb) {
    if (a.two_four && a.sparse_mfma) return launch_fwd24_bf16(a, st);  // structured-sparse MFMA
    if (pass2) return a.two_four ? launch_fmt<RK, true, true>(a, st, ldb) : launch_fmt<RK, false, true>(a, st, ldb);
    return a.two_four ? launch_fmt<RK, true, false>(a, st, ldb) : launch_fmt<RK, false, false>(a, st, ldb);
}

hipError_t launch_ranks(const LayerArgs& a, hipStream_t st, bool pass2, int ldb) {
    switch ((a.r + 15) / 16) {
        case 1: return launch_rk<1>(a, st, pass2, ldb);
        case 2: return launch_rk<2>(a, st, pass2, ldb);
        case 3: return launch_rk<3>(a, st, pass2, ldb);
        case 4: return launch_rk<4>(a, st, pass2, ldb);
        default: return hipErrorInvalidValue;
    }
}

#else  // LORS_THIN_TILES

// thin tiles of one feature half (NF = 1) and TM tokens: 2 BM / TM per tile
template <int RK, bool TWO_FOUR, bool FOLD, int TM>
hipError_t launch_thin_tm(const LayerArgs& a, hipStream_t st, int ldb, int first, int tail) {
    const int tiles_m = (int)((a.L + BM - 1) / BM);
    const int tiles_n = (int)((a.R + BN - 1) / BN);
    hipLaunchKernelGGL((fwd_kernel<RK, TWO_FOUR, false, false, FOLD, TM, 1>), dim3(tail * (2 * BM / TM)), dim3(NT), 0, st,
                       (const uint16_t*)a.X, (const uint16_t*)a.W, a.M, (const uint16_t*)a.B,
                       (const uint16_t*)a.A, (const uint16_t*)a.bias, (uint16_t*)a.Y, a.L, (int)a.R, (int)a.C,
                       (int)a.r, a.scale, tiles_m, tiles_n, ldb, first, tail, (float*)nullptr);
    return hipGetLastError();
}

template <int RK, bool TWO_FOUR, bool FOLD>
hipError_t launch_thin_q(const LayerArgs& a, hipStream_t st, int ldb, int first, int tail, int q) {
    switch (q) {  // q thin tiles per tile: two feature halves, each cut into q/2 token parts
        case 2: return launch_thin_tm<RK, TWO_FOUR, FOLD, BM>(a, st, ldb, first, tail);
        case 4: return launch_thin_tm<RK, TWO_FOUR, FOLD, BM / 2>(a, st, ldb, first, tail);
        case 8: return launch_thin_tm<RK, TWO_FOUR, FOLD, BM / 4>(a, st, ldb, first, tail);
        default: return hipErrorInvalidValue;
    }
}

template <int RK>
hipError_t launch_thin_rk(const LayerArgs& a, hipStream_t st, int ldb, int first, int tail, int q) {
    const bool fold = power_of_two(a.scale);
    if (a.two_four)
        return fold ? launch_thin_q<RK, true, true>(a, st, ldb, first, tail, q)
                    : launch_thin_q<RK, true, false>(a, st, ldb, first, tail, q);
    return fold ? launch_thin_q<RK, false, true>(a, st, ldb, first, tail, q)
                : launch_thin_q<RK, false, false>(a, st, ldb, first, tail, q);
}

#endif  // LORS_THIN_TILES

}  // namespace

#ifndef LORS_THIN_TILES

hipError_t launch_fwd_bf16(const LayerArgs& a, hipStream_t st) {
    if (a.L == 0) return hipSuccess;
    if (a.r <= 64) return launch_ranks(a, st, false, (int)a.r);
    if (a.r > 128) return hipErrorInvalidValue;  // the problem check caps r at 128
    // Ranks above 64: the mask distributes over the sum, so
    //   W' = select(M, W + s.B1.A1, 0) + select(M, s.B2.A2, 0)
    // for ranks [0, 64) and [64, r): two passes of the register-merge
    // kernel, the second with W taken as zero, no bias, and its product added
    // onto Y (one more bf16 rounding of Y).
    LayerArgs a1 = a;
    a1.r = 64;
    const hipError_t e = launch_ranks(a1, st, false, (int)a.r);
    if (e != hipSuccess) return e;
    LayerArgs a2 = a;
    a2.r = a.r - 64;
    a2.B = (const uint16_t*)a.B + 64;
    a2.A = (const uint16_t*)a.A + 64 * a.C;
    a2.bias = nullptr;
    return launch_ranks(a2, st, true, (int)a.r);
}

#else

hipError_t launch_fwd_thin_bf16(const LayerArgs& a, hipStream_t st, int ldb, int first, int tail, int q) {
    if (tail <= 0) return hipSuccess;
    if (!fwd_whole_tiles(a.L, a.R, a.C) || a.r < 1 || a.r > 64) return hipErrorInvalidValue;
    switch ((a.r + 15) / 16) {
        case 1: return launch_thin_rk<1>(a, st, ldb, first, tail, q);
        case 2: return launch_thin_rk<2>(a, st, ldb, first, tail, q);
        case 3: return launch_thin_rk<3>(a, st, ldb, first, tail, q);
        case 4: return launch_thin_rk<4>(a, st, ldb, first, tail, q);
        default: return hipErrorInvalidValue;
    }
}

#endif  // LORS_THIN_TILES

}  // namespace lors
