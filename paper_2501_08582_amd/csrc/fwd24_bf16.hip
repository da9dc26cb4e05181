// Fused forward with a 2:4 mask on gfx950's structured-sparse MFMA.
//
//   Y[L x R] = X[L x C] . W'^T,   W' = select(M, W + s.B.A, 0),  M 2:4 along C
//
// (Eq. 3 of Section 2.2 and Algorithm 1; the 2:4 pattern of Section 3.1.)
// v_smfmac_f32_32x32x32_bf16 multiplies a 32 x 32 A operand that is 2:4
// sparse along K, given as its 16 kept values per row plus 2-bit positions,
// by a dense 32 x 32 B operand: half the matrix-core work of the dense
// product.  The sparse operand must be A, so the roles of the dense forward
// are swapped: W' (rows n) is A and X (columns = tokens) is B, and the
// accumulators hold Y^T blocks, transposed on their way out through LDS.
//
// Operand layouts (32-k step, lane l = 32h + l32):
//   B (X):  row l32 of the token block, k = 16h .. 16h+15 (two 16-byte LDS
//           reads, chunks 2h and 2h+1 of the step);
//   A (W'): row l32 of the feature block, groups 2h, 2h+1, 4+2h, 5+2h of the
//           step (k = 8h .. 8h+7 and 16+8h .. 16+8h+7), two kept bf16 per
//           group in ascending position; the index operand holds the group
//           codes p0 | p1 << 2 in nibble j for the lane's j-th group.
// Those two k ranges are exactly the W' fragments the dense forward builds
// for two consecutive 16-k sub-steps, so the merge is the dense one (rank-r
// MFMA in permuted order, + W, rounded once to bf16) without the select
// masks; a byte permute per group then keeps the two elements the mask
// code names, and the code nibbles themselves are the packed 2:4 mask words
// (one 32-bit word = the eight groups of a 32-k step).  Masked elements never
// enter the product, which is the select semantics of the dense path.
//
// Schedule: a K-step (64 k) is two half-steps of 16 sparse MFMAs; each
// half-step prepares the next one (rank-r product, W' compression, X reads)
// in fixed slots.  The first half-step reads everything the K-step still
// needs from its stage (including all X operands of the second half), so the
// one barrier per K-step, before the second half-step, frees the stage: the
// second half-step issues the copies of stage kt+2 into it and prepares the
// first half of stage kt+1.  Slabs, copies and stage layout are those of the
// dense forward.
#include "gemm_common.hpp"
#include "kernels.hpp"

namespace lors {
namespace {

constexpr int NT = 256;
constexpr int BM = 256;  // tokens per tile
constexpr int BN = 256;  // output features per tile (64 per wave)
constexpr int BK = 64;   // input features per K-step
constexpr int GROUP_M = 4;

constexpr int XB = BM * kRow64;  // 32 KiB
constexpr int WB = BN * kRow64;  // 32 KiB
constexpr int MB = BN * 2 * 4;   // 2 mask words per row of W: 2 KiB

template <int RK>
struct Layout {
    static constexpr int AB = 16 * RK * kRow64;
    static constexpr int X = 0, W = XB, A = XB + WB, M = XB + WB + AB;
    static constexpr int STAGE = XB + WB + AB + MB;
    static constexpr int PLUT = 2 * STAGE;  // 256 x 8 B: byte permute selectors of a mask byte
    static constexpr int SINK = PLUT + 2048;
    static constexpr int TOTAL = SINK + 1024;
    static constexpr int NAW = (2 * RK + 3) / 4;
    static constexpr int COPIES = 16 + NAW + 2;
    static_assert(COPIES - 16 <= 8, "the late copies fit the even slots of a half-step");
};

#define SLOT_END() __builtin_amdgcn_sched_barrier(0)

typedef __bf16 bf16x16 __attribute__((ext_vector_type(16)));

// byte-permute selector keeping bf16 elements p0 < p1 (code p0 | p1 << 2) of
// a group held in two dwords (elements 0, 1 low; 2, 3 high)
__device__ __forceinline__ uint32_t group_selector(uint32_t code) {
    return 0x01000100u + (code & 3u) * 0x0202u + (code >> 2) * 0x02020000u;
}

// W + s.T for one bf16 pair, rounded once (no select: compression drops the
// masked elements)
__device__ __forceinline__ uint32_t merge_pair_all(uint32_t raw, float t0, float t1, float s) {
    return pack_bf16x2(fmaf(s, t0, __uint_as_float(raw << 16)), fmaf(s, t1, __uint_as_float(raw & 0xFFFF0000u)));
}

// T = sum over c of mfma(a[c], b[c]) into VGPRs (one feature block of the
// rank-r product; see rank_mfma2), with the matrix-result -> VALU wait states.
template <int RK>
__device__ __forceinline__ void rank_mfma1(f32x16& T, const bf16x8 (&a)[RK], const bf16x8 (&b)[RK]) {
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(T) : "v"(a[0]), "v"(b[0]));
#pragma unroll
    for (int c = 1; c < RK; ++c)
        asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+&v"(T) : "v"(a[c]), "v"(b[c]));
    if constexpr (RK == 1)
        asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 2" : "+v"(T) : "v"(a[0]));
    else if constexpr (RK == 2)
        asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 2" : "+v"(T) : "v"(a[0]), "v"(a[1]));
    else if constexpr (RK == 3)
        asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 2" : "+v"(T) : "v"(a[0]), "v"(a[1]), "v"(a[2]));
    else {
        static_assert(RK == 4, "ranks up to 64");
        asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 2" : "+v"(T) : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]));
    }
}

template <int RK, bool RAGGED>
__global__ __launch_bounds__(NT, 1) void fwd24_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
    const uint32_t* __restrict__ Mp, const uint16_t* __restrict__ Bm,
    const uint16_t* __restrict__ Am, const uint16_t* __restrict__ bias,
    uint16_t* __restrict__ Y, int64_t L, int R, int C, int r, float s, int tiles_m,
    int tiles_n) {
    using Lay = Layout<RK>;
    static_assert(Lay::TOTAL <= 160 * 1024, "LDS budget");
    static_assert(4 * BM * 128 <= 2 * Lay::STAGE, "output staging fits the stage buffers");
    __shared__ __attribute__((aligned(1024))) uint8_t smem[Lay::TOTAL];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31;
    const int h = lane >> 5;

    int tm, tn;
    tile_coords(blockIdx.x, tiles_m, tiles_n, GROUP_M, tm, tn);
    const int64_t m0 = (int64_t)tm * BM;
    const int n0 = tn * BN;
    const int nk = (C + BK - 1) / BK;
    const int wpr = (C + 31) >> 5;
    const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
    const uint8_t* zsrc = (const uint8_t*)g_zero_page + 16 * (lane & 7);

    // ---- selector LUT (visible after the first stage barrier) and the
    // resident B operand of the merge (column n = 64 wave + 32 nb + l32)
    *(u32x2*)(smem + Lay::PLUT + 8 * tid) = u32x2{group_selector(tid & 15u), group_selector((uint32_t)tid >> 4)};
    const bool b_vec = (r & 7) == 0;
    bf16x8 bfr[2][RK];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
        const int gn = n0 + 64 * wave + 32 * nb + l32;
#pragma unroll
        for (int c = 0; c < RK; ++c) {
            u32x4 v = zero_u32x4();
            const int j0 = 16 * c + 8 * h;
            if (gn < R) {
                const uint16_t* src = Bm + (int64_t)gn * r + j0;
                if (b_vec) {
                    if (j0 < r) v = *(const u32x4*)src;
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        v[e >> 1] |= (j0 + e < r ? (uint32_t)src[e] : 0u) << ((e & 1) * 16);
                }
            }
            bfr[nb][c] = as_bf16x8(v);
        }
    }

    // ---- slab copies (as in the dense forward)
    uint32_t offXW[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int row = 8 * (8 * wave + q) + (lane >> 3);
        const int lc = (lane & 7) ^ ((row >> 1) & 7);
        offXW[q] = (uint32_t)((row * C + 8 * lc) * 2);
    }
    const uint16_t* aptr[Lay::NAW];
#pragma unroll
    for (int q = 0; q < Lay::NAW; ++q) {
        const int row = 8 * (4 * q + wave) + (lane >> 3);
        const int lc = (lane & 7) ^ ((row >> 1) & 7);
        aptr[q] = Am + (int64_t)row * C + 8 * lc;
    }
    uint32_t offM[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int e = 64 * (2 * wave + q) + lane;
        offM[q] = (uint32_t)(((e >> 1) * wpr + (e & 1)) * 4);
    }
    const uint16_t* Xt = uniform_ptr(X + m0 * C);
    const uint16_t* Wt = uniform_ptr(W + (int64_t)n0 * C);
    const uint32_t* Mt = uniform_ptr(Mp + (int64_t)n0 * wpr);

    auto copy_j = [&](int j, int k0, uint32_t sb) {
        if (j < 16) {
            const int q = j & 7;
            const bool isx = j < 8;
            const uint32_t dst = sb + (isx ? Lay::X : Lay::W) + 1024 * (8 * wave + q);
            if constexpr (!RAGGED) {
                copy16s_to_lds(uniform_ptr((isx ? Xt : Wt) + k0), offXW[q], dst);
            } else {
                const int row = 8 * (8 * wave + q) + (lane >> 3);
                const int lc = (lane & 7) ^ ((row >> 1) & 7);
                const bool ok = (isx ? m0 + row < L : n0 + row < R) && k0 + 8 * lc < C;
                const uint16_t* src = (isx ? Xt : Wt) + (int64_t)row * C + k0 + 8 * lc;
                copy16_to_lds(ok ? (const void*)src : (const void*)zsrc, dst);
            }
        } else if (j < 16 + Lay::NAW) {
            const int q = j - 16, blk = 4 * q + wave;
            const bool has = blk < 2 * RK;
            const int row = 8 * blk + (lane >> 3);
            const int lc = (lane & 7) ^ ((row >> 1) & 7);
            const bool ok = has && row < r && (!RAGGED || k0 + 8 * lc < C);
            copy16_to_lds(ok ? (const void*)(aptr[q] + k0) : (const void*)zsrc,
                          has ? sb + Lay::A + 1024 * blk : lds0 + Lay::SINK);
        } else {
            const int q = j - 16 - Lay::NAW;
            const uint32_t dst = sb + Lay::M + 256 * (2 * wave + q);
            if constexpr (!RAGGED) {
                copy4s_to_lds(uniform_ptr(Mt + (k0 >> 5)), offM[q], dst);
            } else {
                const int e = 64 * (2 * wave + q) + lane;
                const bool ok = n0 + (e >> 1) < R && (k0 >> 5) + (e & 1) < wpr;
                const uint32_t* src = Mt + (int64_t)(e >> 1) * wpr + (k0 >> 5) + (e & 1);
                copy4_to_lds(ok ? (const void*)src : (const void*)zsrc, dst);
            }
        }
    };

    // ---- per-lane LDS offsets
    int offAt[2][2];  // A^T operand of the merge (rows permuted), as in the dense forward
    {
        const int g = lane >> 4, jj = lane & 15;
        const int sig = ((jj & 3) == 1) ? 2 : ((jj & 3) == 2) ? 1 : (jj & 3);
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const int row = 8 * (g >> 1) + 4 * t + (jj >> 2);
                const int col = 32 * kb + 16 * (g & 1) + 4 * sig;
                offAt[kb][t] = Lay::A + slab64_elem_off(row, col);
            }
    }
    const int nrow0 = 64 * wave + l32;
    // X (B operand) of token block mb, half kb: chunks 4kb + 2h + e
    auto xoff = [&](int mb, int kb, int e) { return Lay::X + slab64_off(32 * mb + l32, 4 * kb + 2 * h + e); };
    // raw W of feature block nb, half kb, chunk c: chunk 4kb + 2c + h
    auto woff = [&](int nb, int kb, int c) { return Lay::W + slab64_off(nrow0 + 32 * nb, 4 * kb + 2 * c + h); };

    f32x16 acc[2][8];  // [feature block][token block]
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    bf16x16 xr[4];         // X operands of half 0: ring of token blocks mb % 4, read two blocks ahead
    bf16x16 xh[8];         // X operands of half 1, all read during half 0 (before the barrier)
    u32x4 wa[2], wb[2];    // compressed W' operands of alternate half-steps
    uint32_t ia[2], ib[2]; // their index operands
    // the first MFMA holds the last operands of a previous half-step as well
    xh[7] = bf16x16{};
    wb[1] = zero_u32x4();
    ib[1] = 0u;
    f32x16 T;              // rank-r block of the feature block being prepared
    uint32_t mw[2][2];     // mask words [nb][kb] of the stage being prepared
    u32x4 raw[2];          // raw W [c] of that feature block
    u32x2 psel[2];         // permute selectors [c]
    bf16x8 afr[RK];

    // kx, kw, ki: the operands of the previous structured-sparse MFMA.  The
    // matrix core reads its sources over several passes after issue, so they
    // are held here, as inputs of the next one, and no instruction in
    // between may reuse their registers.
    auto smf = [&](int i, const bf16x16& xf, const u32x4 (&wf)[2], const uint32_t (&ix)[2], const bf16x16& kx,
                   const u32x4& kw, uint32_t ki) {
        const int mb = i >> 1, nb = i & 1;
        asm volatile("v_smfmac_f32_32x32x32_bf16 %0, %1, %2, %3\n\ts_nop 7"
                     : "+a"(acc[nb][mb])
                     : "v"(wf[nb]), "v"(xf), "v"(ix[nb]), "v"(kx), "v"(kw), "v"(ki));
    };
    auto read_afr = [&](const uint8_t* sb, int kb) {
#pragma unroll
        for (int c = 0; c < RK; ++c)
            afr[c] = frag_from_tr(lds_tr_read(sb + offAt[kb][0] + 16 * kRow64 * c),
                                  lds_tr_read(sb + offAt[kb][1] + 16 * kRow64 * c));
    };
    auto read_mw = [&](const uint8_t* sb) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
            const u32x2 v = *(const u32x2*)(sb + Lay::M + 8 * (nrow0 + 32 * nb));
            mw[nb][0] = v[0];
            mw[nb][1] = v[1];
        }
    };
    // raw W, selectors and index operand of feature block nb for half kb
    auto read_blk = [&](const uint8_t* sb, int kb, int nb, uint32_t (&ix)[2]) {
#pragma unroll
        for (int c = 0; c < 2; ++c) raw[c] = *(const u32x4*)(sb + woff(nb, kb, c));
        const uint32_t w = mw[nb][kb];
        const uint32_t b0 = (w >> (8 * h)) & 0xFFu, b1 = (w >> (16 + 8 * h)) & 0xFFu;
        psel[0] = *(const u32x2*)(smem + Lay::PLUT + 8 * b0);
        psel[1] = *(const u32x2*)(smem + Lay::PLUT + 8 * b1);
        ix[nb] = b0 | (b1 << 8);
    };
    auto read_x = [&](bf16x16& xf, const uint8_t* sb, int kb, int mb) {
        const bf16x8 lo = *(const bf16x8*)(sb + xoff(mb, kb, 0));
        const bf16x8 hi = *(const bf16x8*)(sb + xoff(mb, kb, 1));
        xf = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
    };
    // piece p (0..3) of the compression of feature block nb: chunk c, group g
    auto piece = [&](u32x4 (&wf)[2], int nb, int p) {
        const int c = p >> 1, g = p & 1;
        const uint32_t lo = merge_pair_all(raw[c][2 * g], T[8 * c + 4 * g], T[8 * c + 4 * g + 1], s);
        const uint32_t hi = merge_pair_all(raw[c][2 * g + 1], T[8 * c + 4 * g + 2], T[8 * c + 4 * g + 3], s);
        wf[nb][2 * c + g] = __builtin_amdgcn_perm(hi, lo, psel[c][g]);
    };
    // Half-step 0 of a K-step: MFMAs of half 0 (X from the ring, block mb + 2
    // read at slot 2 mb) while reading all X operands of half 1 and preparing
    // its W' operand, one feature block at a time.  Every read of the stage
    // happens here, before the barrier.  cp(t) issues this slot's late
    // copies of the next stage.
    auto half0 = [&](const uint8_t* sb, auto cp) {
        smf(0, xr[0], wa, ia, xh[7], wb[1], ib[1]); read_x(xr[2], sb, 0, 2); read_afr(sb, 1); cp(0); SLOT_END();
        smf(1, xr[0], wa, ia, xr[0], wa[0], ia[0]); read_blk(sb, 1, 0, ib); read_x(xh[0], sb, 1, 0); cp(1); SLOT_END();
        smf(2, xr[1], wa, ia, xr[0], wa[1], ia[1]); read_x(xr[3], sb, 0, 3); rank_mfma1<RK>(T, afr, bfr[0]); cp(2); SLOT_END();
        smf(3, xr[1], wa, ia, xr[1], wa[0], ia[0]); read_x(xh[1], sb, 1, 1); piece(wb, 0, 0); cp(3); SLOT_END();
        smf(4, xr[2], wa, ia, xr[1], wa[1], ia[1]); read_x(xr[0], sb, 0, 4); piece(wb, 0, 1); cp(4); SLOT_END();
        smf(5, xr[2], wa, ia, xr[2], wa[0], ia[0]); read_x(xh[2], sb, 1, 2); piece(wb, 0, 2); cp(5); SLOT_END();
        smf(6, xr[3], wa, ia, xr[2], wa[1], ia[1]); read_x(xr[1], sb, 0, 5); piece(wb, 0, 3); cp(6); SLOT_END();
        smf(7, xr[3], wa, ia, xr[3], wa[0], ia[0]); read_blk(sb, 1, 1, ib); read_x(xh[3], sb, 1, 3); cp(7); SLOT_END();
        smf(8, xr[0], wa, ia, xr[3], wa[1], ia[1]); read_x(xr[2], sb, 0, 6); rank_mfma1<RK>(T, afr, bfr[1]); cp(8); SLOT_END();
        smf(9, xr[0], wa, ia, xr[0], wa[0], ia[0]); read_x(xh[4], sb, 1, 4); piece(wb, 1, 0); cp(9); SLOT_END();
        smf(10, xr[1], wa, ia, xr[0], wa[1], ia[1]); read_x(xr[3], sb, 0, 7); piece(wb, 1, 1); cp(10); SLOT_END();
        smf(11, xr[1], wa, ia, xr[1], wa[0], ia[0]); read_x(xh[5], sb, 1, 5); piece(wb, 1, 2); cp(11); SLOT_END();
        smf(12, xr[2], wa, ia, xr[1], wa[1], ia[1]); read_x(xh[6], sb, 1, 6); piece(wb, 1, 3); cp(12); SLOT_END();
        smf(13, xr[2], wa, ia, xr[2], wa[0], ia[0]); read_x(xh[7], sb, 1, 7); cp(13); SLOT_END();
        smf(14, xr[3], wa, ia, xr[2], wa[1], ia[1]); cp(14); SLOT_END();
        smf(15, xr[3], wa, ia, xr[3], wa[0], ia[0]); cp(15); SLOT_END();
    };
    // Half-step 1: MFMAs of half 1 (X from xh) while preparing half 0 of the
    // next stage at sn (ring blocks 0, 1 and its W' operand); cp(t) issues
    // this slot's copies of stage kt+2.
    auto half1 = [&](const uint8_t* sn, auto cp) {
        smf(0, xh[0], wb, ib, xr[3], wa[1], ia[1]); read_mw(sn); read_afr(sn, 0); cp(0); SLOT_END();
        smf(1, xh[0], wb, ib, xh[0], wb[0], ib[0]); read_blk(sn, 0, 0, ia); cp(1); SLOT_END();
        smf(2, xh[1], wb, ib, xh[0], wb[1], ib[1]); rank_mfma1<RK>(T, afr, bfr[0]); cp(2); SLOT_END();
        smf(3, xh[1], wb, ib, xh[1], wb[0], ib[0]); piece(wa, 0, 0); cp(3); SLOT_END();
        smf(4, xh[2], wb, ib, xh[1], wb[1], ib[1]); piece(wa, 0, 1); cp(4); SLOT_END();
        smf(5, xh[2], wb, ib, xh[2], wb[0], ib[0]); piece(wa, 0, 2); cp(5); SLOT_END();
        smf(6, xh[3], wb, ib, xh[2], wb[1], ib[1]); piece(wa, 0, 3); cp(6); SLOT_END();
        smf(7, xh[3], wb, ib, xh[3], wb[0], ib[0]); read_blk(sn, 0, 1, ia); cp(7); SLOT_END();
        smf(8, xh[4], wb, ib, xh[3], wb[1], ib[1]); rank_mfma1<RK>(T, afr, bfr[1]); cp(8); SLOT_END();
        smf(9, xh[4], wb, ib, xh[4], wb[0], ib[0]); piece(wa, 1, 0); cp(9); SLOT_END();
        smf(10, xh[5], wb, ib, xh[4], wb[1], ib[1]); piece(wa, 1, 1); cp(10); SLOT_END();
        smf(11, xh[5], wb, ib, xh[5], wb[0], ib[0]); piece(wa, 1, 2); cp(11); SLOT_END();
        smf(12, xh[6], wb, ib, xh[5], wb[1], ib[1]); piece(wa, 1, 3); read_x(xr[0], sn, 0, 0); cp(12); SLOT_END();
        smf(13, xh[6], wb, ib, xh[6], wb[0], ib[0]); read_x(xr[1], sn, 0, 1); cp(13); SLOT_END();
        smf(14, xh[7], wb, ib, xh[6], wb[1], ib[1]); cp(14); SLOT_END();
        smf(15, xh[7], wb, ib, xh[7], wb[0], ib[0]); cp(15); SLOT_END();
    };
    // prepare half 0 of the stage at sb without MFMAs (prologue)
    auto prepare = [&](const uint8_t* sb) {
        read_afr(sb, 0);
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
            read_blk(sb, 0, nb, ia);
            rank_mfma1<RK>(T, afr, bfr[nb]);
#pragma unroll
            for (int p = 0; p < 4; ++p) piece(wa, nb, p);
        }
        read_x(xr[0], sb, 0, 0);
        read_x(xr[1], sb, 0, 1);
    };

    // ---- prologue: stages 0 and 1 in flight, half 0 of stage 0 prepared
#pragma unroll
    for (int j = 0; j < Lay::COPIES; ++j) copy_j(j, 0, lds0);
#pragma unroll
    for (int j = 0; j < Lay::COPIES; ++j) copy_j(j, nk > 1 ? BK : 0, lds0 + Lay::STAGE);
    stage_barrier<0>();
    read_mw(smem);
    prepare(smem);

    // ---- main loop (branch-free: at the tail the copies repeat the last
    // K-slab into the buffer just consumed, and the preparation of the
    // "next" stage after the last K-step is never used)
    for (int kt = 0; kt < nk; ++kt) {
        const int st = kt & 1;
        const uint8_t* sb = smem + st * Lay::STAGE;
        const uint8_t* sn = smem + (st ^ 1) * Lay::STAGE;
        // copies 16.. of stage kt+1 (buffer st^1, free since the last barrier;
        // the barrier below waits for them); at kt = 0 the prologue issued
        // all of stage 1
        const int k1 = (kt + 1 < nk ? kt + 1 : nk - 1) * BK;
        const uint32_t sq1 = lds0 + (st ^ 1) * Lay::STAGE;
        half0(sb, [&](int t) {
            if (kt > 0 && (t & 1) == 0 && 16 + t / 2 < Lay::COPIES) copy_j(16 + t / 2, k1, sq1);
        });
        // stage kt+1 landed everywhere; every read of stage kt is done
        stage_barrier<0>();
        const int k2 = (kt + 2 < nk ? kt + 2 : nk - 1) * BK;
        const uint32_t sq = lds0 + st * Lay::STAGE;
        // one copy per MFMA slot: a second copy behind the same MFMA would
        // stall the wave past it
        half1(sn, [&](int t) { copy_j(t, k2, sq); });
    }
    // ---- epilogue: (+bias), round to bf16, stage the wave's 256 tokens x 64
    // features block in LDS (rows of 64 outputs), then 16-byte row stores
    wait_vmcnt<0>();
    lds_barrier();
    uint16_t* ol = (uint16_t*)(smem + wave * (BM * 128));
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
#pragma unroll
        for (int v = 0; v < 16; v += 2) {
            const int f = 32 * nb + 8 * (v >> 2) + 4 * h + (v & 3);  // feature within the wave's 64
            const int gn = n0 + 64 * wave + f;
            const float b0 = (bias != nullptr && gn < R) ? bf16_bits_to_f32(bias[gn]) : 0.f;
            const float b1 = (bias != nullptr && gn + 1 < R) ? bf16_bits_to_f32(bias[gn + 1]) : 0.f;
#pragma unroll
            for (int mb = 0; mb < 8; ++mb)
                *(uint32_t*)(ol + (32 * mb + l32) * 64 + f) = pack_bf16x2(acc[nb][mb][v] + b0, acc[nb][mb][v + 1] + b1);
        }
    }
    __syncthreads();
#pragma unroll 4
    for (int it = 0; it < BM / 8; ++it) {
        const int row = 8 * it + (lane >> 3), ch = lane & 7;
        const u32x4 v = *(const u32x4*)(ol + row * 64 + 8 * ch);
        const int64_t gm = m0 + row;
        const int gn = n0 + 64 * wave + 8 * ch;
        if (gm < L && gn < R) *(u32x4*)(Y + gm * R + gn) = v;
    }
}

template <int RK>
hipError_t launch_rk(const LayerArgs& a, hipStream_t st) {
    const int tiles_m = (int)((a.L + BM - 1) / BM);
    const int tiles_n = (int)((a.R + BN - 1) / BN);
    dim3 grid(tiles_m * tiles_n), block(NT);
    auto* X = (const uint16_t*)a.X;
    auto* W = (const uint16_t*)a.W;
    auto* B = (const uint16_t*)a.B;
    auto* A = (const uint16_t*)a.A;
    auto* bias = (const uint16_t*)a.bias;
    auto* Y = (uint16_t*)a.Y;
    const bool ragged = a.L % BM != 0 || a.R % BN != 0 || a.C % BK != 0 || (int64_t)BM * a.C * 2 >= (1ll << 31);
    if (ragged)
        hipLaunchKernelGGL((fwd24_kernel<RK, true>), grid, block, 0, st, X, W, a.M, B, A, bias, Y, a.L, (int)a.R,
                           (int)a.C, (int)a.r, a.scale, tiles_m, tiles_n);
    else
        hipLaunchKernelGGL((fwd24_kernel<RK, false>), grid, block, 0, st, X, W, a.M, B, A, bias, Y, a.L, (int)a.R,
                           (int)a.C, (int)a.r, a.scale, tiles_m, tiles_n);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_fwd24_bf16(const LayerArgs& a, hipStream_t st) {
    if (a.L == 0) return hipSuccess;
    switch ((a.r + 15) / 16) {
        case 1: return launch_rk<1>(a, st);
        case 2: return launch_rk<2>(a, st);
        case 3: return launch_rk<3>(a, st);
        case 4: return launch_rk<4>(a, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace lors
