// Backward adapter gradients, bf16 on gfx950.
//
//   G  = select(M, dY^T . X, 0)      (R x C, never written to HBM)
//   dB += s . G . A^T   (R x r, fp32)     dA += s . B^T . G   (r x C, fp32)
//
// (I_w^4, I_w^5 and the two adapter gradients of the SP-LoRA backward list in
// Section 2.2, with the scale of the listing.)  The weight-gradient GEMM runs
// over K = L with both operands token-major: each K-step copies a 64-token
// slab of dY and of X straight from HBM into LDS in natural layout, and the
// MFMA operands are read back with the LDS transpose load, so no lane ever
// shuffles data.  Four waves each own a 128 x 128 block of the 256 x 256 G
// tile (fp32 accumulators in AGPRs); LDS is double-buffered.
//
// Epilogue: the accumulators are masked in registers (keep bits from the
// transposed bitmap M^T, one word per lane and 32 rows) and rounded to bf16.
// dA uses them directly as the MFMA B operand (contraction over the rows of G
// in the accumulator's own row order); dB reads G^T back from LDS.  Per-tile
// partial sums are added into dB and dA with fp32 atomics, so dB and dA must
// be zero on entry.
#include "gemm_common.hpp"
#include "kernels.hpp"

namespace lors {
namespace {

constexpr int NT = 256;
constexpr int BM = 256;  // rows of G (output features, R) per tile
constexpr int BN = 256;  // columns of G (input features, C) per tile
constexpr int BK = 64;   // tokens per K-step
constexpr int TILEB = BK * kRowBytes;  // 32 KiB: one operand slab
constexpr int STAGEB = 2 * TILEB;      // dY slab + X slab
constexpr int SMEM = 2 * STAGEB;       // two stages
constexpr int GROUP_M = 4;
constexpr int LOADS = TILEB / 1024 / (NT / kWave);  // 1 KiB copies per wave per slab (8)
// copy pairs of a stage issued right after the barrier; the rest go out a
// sub-step later (a wave stalls on a burst of asynchronous copies)
constexpr int kEarlyPairs = 4;

// Epilogue LDS carve-up (reuses the stage buffers; EP_A lies past them).
constexpr int GT_PITCH = 512;                      // G^T tile: [j][i], 256 i per row
constexpr int GT_BYTES = BN * GT_PITCH;            // 128 KiB
constexpr int EP_MT = 0;                           // M^T words [j][8]: 8 KiB
constexpr int EP_LUT = 8192;                       // select LUT: 4 KiB
constexpr int EP_B = 12288;                        // B block [i][32*JB] bf16: 16 KiB per 32 ranks
                                                   // (then the dA exchange, see the kernel)
constexpr int EP_A = SMEM;                         // A block [32 j'][256 j]: 16 KiB
constexpr int SMEM_ALL = SMEM + 32 * kRowBytes;

// RAGGED: some tile reaches past R, C or the token count L (copies check
// every lane and read the zero page outside the tensors); otherwise copies
// use uniform bases plus fixed per-lane offsets.
template <int RK, bool RAGGED>
__global__ __launch_bounds__(NT, 1) void g_kernel(
    const uint16_t* __restrict__ dY, const uint16_t* __restrict__ X,
    const uint32_t* __restrict__ Mt, const uint16_t* __restrict__ Bm,
    const uint16_t* __restrict__ Am, float* __restrict__ dB, float* __restrict__ dA,
    int64_t L, int R, int C, int r, float s, int tiles_m, int tiles_n, int n_full, int split) {
    constexpr int JB = (RK + 1) / 2;  // 32-wide blocks of the rank
    // dA exchange: JBC rank blocks per round, one 4 KiB slot [v/4][lane][4]
    // per (wj, column block b, rank block of the round), right after the B block
    constexpr int JBC = JB <= 2 ? JB : 1;
    constexpr int EP_X = EP_B + BM * 32 * JB * 2;
    static_assert(GT_BYTES <= SMEM, "G^T tile fits");
    static_assert(EP_X + 2 * 4 * JBC * 16 * kWave * 4 <= SMEM, "B block and dA exchange fit");
    __shared__ __attribute__((aligned(1024))) uint8_t smem[SMEM_ALL];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31;
    const int h = lane >> 5;
    const int wi = wave >> 1, wj = wave & 1;

    // tile and token range: a piece of a split tile covers K-steps
    // [kbeg, kbeg + nk); its G is a partial sum over those tokens, and since
    // the mask select and both rank-r products are linear in G, the pieces'
    // contributions add up in dB and dA like those of different tiles
    int tm, tn;
    int kbeg, nk32;
    work_coords(blockIdx.x, tiles_m, tiles_n, GROUP_M, n_full, split, (int)((L + BK - 1) / BK), tm, tn, kbeg, nk32);
    const int64_t nk = nk32;
    const int i0 = tm * BM;
    const int j0 = tn * BN;
    const int64_t kofs = (int64_t)kbeg * BK;
    const int wprT = (R + 31) >> 5;  // words per row of M^T

    // ---- asynchronous slab copies: copy pair q of this wave fills tile row
    // 2*(8*wave + q) + h of the dY slab and of the X slab; lane l covers
    // physical chunk l % 32 of its row.  Rows past L and columns past R / C
    // read the zero page.
    const int pchunk = lane & 31;
    const uint8_t* zsrc = (const uint8_t*)g_zero_page + 16 * lane;
    const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
    uint32_t offD[LOADS], offX[LOADS];
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
        const int row = 2 * (LOADS * wave + q) + h;
        const int lc = swz_chunk(row, pchunk);
        offD[q] = (uint32_t)((row * R + lc * 8) * 2);
        offX[q] = (uint32_t)((row * C + lc * 8) * 2);
    }
    const uint16_t* dYt = uniform_ptr(dY + i0);
    const uint16_t* Xt = uniform_ptr(X + j0);
    auto copy_pair = [&](int q, int64_t k0, uint32_t sb) {
        k0 += kofs;
        const uint32_t da = sb + (LOADS * wave + q) * 1024, xa = da + TILEB;
        if constexpr (!RAGGED) {
            copy16s_to_lds(uniform_ptr(dYt + k0 * R), offD[q], da);
            copy16s_to_lds(uniform_ptr(Xt + k0 * C), offX[q], xa);
        } else {
            const int row = 2 * (LOADS * wave + q) + h;
            const int lc = swz_chunk(row, pchunk);
            const int64_t gl = k0 + row;
            const int gi = i0 + lc * 8, gj = j0 + lc * 8;
            const void* a = (gl < L && gi < R) ? (const void*)(dY + gl * R + gi) : (const void*)zsrc;
            const void* b = (gl < L && gj < C) ? (const void*)(X + gl * C + gj) : (const void*)zsrc;
            copy16_to_lds(a, da);
            copy16_to_lds(b, xa);
        }
    };

    // Per-lane fragment offsets inside a stage (sub-step rows added later).
    int offA[4][2], offB[4][2];
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            offA[b][t] = tr_frag_off(lane, 0, wi * 128 + 32 * b, t);
            offB[b][t] = TILEB + tr_frag_off(lane, 0, wj * 128 + 32 * b, t);
        }
    auto load_frags = [&](bf16x8 (&fa)[4], bf16x8 (&fb)[4], const uint8_t* base, int c) {
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            fa[b] = frag_from_tr(lds_tr_read(base + 16 * c * kRowBytes + offA[b][0]),
                                 lds_tr_read(base + 16 * c * kRowBytes + offA[b][1]));
            fb[b] = frag_from_tr(lds_tr_read(base + 16 * c * kRowBytes + offB[b][0]),
                                 lds_tr_read(base + 16 * c * kRowBytes + offB[b][1]));
        }
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;

    // ---- main loop.  Software pipeline: the operand fragments of sub-step
    // c+1 are read from LDS while the 16 MFMAs of sub-step c run.  One
    // barrier per K-step, before its last sub-step: after it every wave has
    // finished reading the current stage and the next stage has landed, so
    // the last sub-step interleaves its MFMAs with the first kEarlyPairs copy
    // pairs of stage kt+2 (into the buffer just consumed) and the first
    // fragment reads of stage kt+1; the remaining pairs of stage kt+2 go out
    // during sub-step 0 of the next K-step.  The body has no data-dependent
    // branches besides the first K-step's: at the tail the copies repeat the
    // last K-slab into a buffer that is never read again.
    static_assert(BK / 16 == 4 && LOADS == 8, "sub-step schedule below assumes 4 sub-steps, 8 copy pairs");
#pragma unroll
    for (int st = 0; st < 2; ++st) {
        const int64_t k0 = (int64_t)(st < nk ? st : nk - 1) * BK;
#pragma unroll
        for (int q = 0; q < LOADS; ++q) copy_pair(q, k0, lds0 + st * STAGEB);
    }
    stage_barrier<2 * LOADS>();  // stage 0 landed everywhere; stage 1 may still fly

    bf16x8 fa0[4], fb0[4], fa1[4], fb1[4];
    load_frags(fa0, fb0, smem, 0);
    auto mfma16 = [&](const bf16x8 (&fa)[4], const bf16x8 (&fb)[4]) {
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < 4; ++b) acc[a][b] = mfma_32x32x16(fa[a], fb[b], acc[a][b]);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
        }
    };
    for (int64_t kt = 0; kt < nk; ++kt) {
        const int st = (int)(kt & 1);
        const uint8_t* sb = smem + st * STAGEB;
        const uint8_t* sn = smem + (st ^ 1) * STAGEB;
        {
            // sub-step 0, with the transpose reads of sub-step 1 and copy
            // pairs kEarlyPairs.. of stage kt+1 interleaved (that stage's
            // buffer, st^1, is free since the last barrier, and the barrier
            // below waits for the copies; at kt = 0 the prologue issued all
            // of stage 1)
            const int64_t k1 = (kt + 1 < nk ? kt + 1 : nk - 1) * BK;
            const uint32_t sq1 = lds0 + (st ^ 1) * STAGEB;
            const uint8_t* s1 = sb + 16 * kRowBytes;
            u32x2 lo = {0u, 0u};
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int f = i >> 2, part = i & 3;
                acc[f][part] = mfma_32x32x16(fa0[f], fb0[part], acc[f][part]);
                if (part == 0) lo = lds_tr_read(s1 + offA[f][0]);
                if (part == 1) fa1[f] = frag_from_tr(lo, lds_tr_read(s1 + offA[f][1]));
                if (part == 2) lo = lds_tr_read(s1 + offB[f][0]);
                if (part == 3) fb1[f] = frag_from_tr(lo, lds_tr_read(s1 + offB[f][1]));
                if (kt > 0 && part == 1 && kEarlyPairs + f < LOADS) copy_pair(kEarlyPairs + f, k1, sq1);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        load_frags(fa0, fb0, sb, 2);
        mfma16(fa1, fb1);
        load_frags(fa1, fb1, sb, 3);
        mfma16(fa0, fb0);
        stage_barrier<0>();
        const int64_t k0 = (kt + 2 < nk ? kt + 2 : nk - 1) * BK;
        const uint32_t sbq = lds0 + st * STAGEB;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int a = i >> 2, b = i & 3;
            acc[a][b] = mfma_32x32x16(fa1[a], fb1[b], acc[a][b]);
            if ((i & 1) == 0 && (i >> 1) < kEarlyPairs) copy_pair(i >> 1, k0, sbq);
            if (i < 8) {
                // fragment i/2 of A (even i) or B (odd i) of sub-step 0, stage kt+1
                if ((i & 1) == 0)
                    fa0[i >> 1] = frag_from_tr(lds_tr_read(sn + offA[i >> 1][0]), lds_tr_read(sn + offA[i >> 1][1]));
                else
                    fb0[i >> 1] = frag_from_tr(lds_tr_read(sn + offB[i >> 1][0]), lds_tr_read(sn + offB[i >> 1][1]));
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    stage_barrier<0>();

    // ---- epilogue 1: side data, all requests in flight together:
    //   M^T words of the tile [j][8 words] and the A block of rank block 0
    //   (copies into LDS), the select LUT, and B[i0 .. i0+255][0 .. 32*JB)
    //   as [i][32*JB] with ranks >= r zero: thread t loads row i0 + t with
    //   16-byte loads (all issued before the first use).
    uint32_t* mtl = (uint32_t*)(smem + EP_MT);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int blk = 8 * wave + q;          // 32 copies of 64 words
        const int e = 64 * blk + lane;
        const int j = e >> 3, iw = e & 7;
        const int gj = j0 + j, giw = (i0 >> 5) + iw;
        copy4_to_lds((gj < C && giw < wprT) ? (const void*)(Mt + mt_index(gj, giw, C, wprT)) : (const void*)zsrc,
                     lds0 + EP_MT + 256 * blk);
    }
    auto copy_a_block = [&](int jb) {  // A[32jb .. +31][j0 .. j0+255] -> EP_A
#pragma unroll
        for (int q = 0; q < 4; ++q) {          // 32 rows x 512 B = 16 copies, 4 per wave
            const int blk = 4 * wave + q;
            const int row = 2 * blk + h;
            const int lc = swz_chunk(row, lane & 31);
            const int jr = 32 * jb + row, gj = j0 + 8 * lc;
            copy16_to_lds((jr < r && gj < C) ? (const void*)(Am + (int64_t)jr * C + gj) : (const void*)zsrc,
                          lds0 + EP_A + 1024 * blk);
        }
    };
    copy_a_block(0);
    *(u32x4*)(smem + EP_LUT + 16 * tid) = select_lut_entry<false>((uint32_t)tid);
    {
        const int gi = i0 + tid;
        const bool b_vec = (r & 7) == 0;
        u32x4 bv[4 * JB];
#pragma unroll
        for (int c = 0; c < 4 * JB; ++c) {
            bv[c] = zero_u32x4();
            const int jr0 = 8 * c;
            if (gi < R && jr0 < r) {
                const uint16_t* src = Bm + (int64_t)gi * r + jr0;
                if (b_vec) {
                    bv[c] = *(const u32x4*)src;
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        bv[c][e >> 1] |= (jr0 + e < r ? (uint32_t)src[e] : 0u) << ((e & 1) * 16);
                }
            }
        }
#pragma unroll
        for (int c = 0; c < 4 * JB; ++c) *(u32x4*)(smem + EP_B + 2 * (tid * 32 * JB + 8 * c)) = bv[c];
    }
    stage_barrier<0>();

    // ---- epilogue 2: select by the mask, round to bf16.  gb[a][b][c] holds
    // accumulator elements 8c .. 8c+7 of block (a, b): rows 16c + 4h + {0..3}
    // and 16c + 8 + 4h + {0..3} of column j = l32.
    u32x4 gb[4][4][2];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int jl = wj * 128 + 32 * b + l32;
            const uint32_t word = mtl[jl * 8 + wi * 4 + a];
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const uint32_t byte = ((word >> (16 * c + 4 * h)) & 0xFu) | (((word >> (16 * c + 8 + 4 * h)) & 0xFu) << 4);
                const u32x4 sel = *(const u32x4*)(smem + EP_LUT + 16 * byte);
#pragma unroll
                for (int p = 0; p < 4; ++p)
                    gb[a][b][c][p] = pack_bf16x2(acc[a][b][8 * c + 2 * p], acc[a][b][8 * c + 2 * p + 1]) & sel[p];
            }
        }

    // ---- epilogue 3: dA[j'][j] += s * sum_i B[i][j'] G[i][j], with the masked
    // bf16 accumulators as the MFMA B operand (K = rows i in accumulator
    // order); the A operand B^T comes from the B block by transpose loads, one
    // fragment per (row block, rank block) shared by the four column blocks b.
    // The two waves with the same wj hold partial sums over the two halves of
    // the tile's rows: for column blocks b = 0, 1 wave wi = 1 hands its partials
    // to wave wi = 0 through LDS, for b = 2, 3 the other way round, so each dA
    // element receives one atomic add per tile.  All partials of a round are
    // formed first, then exchanged behind one barrier.
    {
        const int g = lane >> 4, jj = lane & 15;
        auto slot = [&](int b, int jl) {
            return (u32x4*)(smem + EP_X) + ((wj * 4 + b) * JBC + jl) * 4 * kWave;
        };
#pragma unroll
        for (int jb0 = 0; jb0 < JB; jb0 += JBC) {
            f32x16 part[4][JBC];
#pragma unroll
            for (int b = 0; b < 4; ++b)
#pragma unroll
                for (int jl = 0; jl < JBC; ++jl)
#pragma unroll
                    for (int v = 0; v < 16; ++v) part[b][jl][v] = 0.f;
#pragma unroll
            for (int jl = 0; jl < JBC; ++jl) {
                const int col = 32 * (jb0 + jl) + 16 * (g & 1) + 4 * (jj & 3);
#pragma unroll
                for (int a = 0; a < 4; ++a)
#pragma unroll
                    for (int c = 0; c < 2; ++c) {
                        const int row = wi * 128 + 32 * a + 16 * c + 4 * (g >> 1) + (jj >> 2);
                        const bf16x8 bt = frag_from_tr(lds_tr_read(smem + EP_B + 2 * (row * 32 * JB + col)),
                                                       lds_tr_read(smem + EP_B + 2 * ((row + 8) * 32 * JB + col)));
#pragma unroll
                        for (int b = 0; b < 4; ++b) part[b][jl] = mfma_32x32x16(bt, as_bf16x8(gb[a][b][c]), part[b][jl]);
                    }
            }
#pragma unroll
            for (int b = 0; b < 4; ++b)
                if ((b < 2) == (wi == 1)) {  // giver
#pragma unroll
                    for (int jl = 0; jl < JBC; ++jl)
#pragma unroll
                        for (int v4 = 0; v4 < 4; ++v4)
                            slot(b, jl)[v4 * kWave + lane] = u32x4{__float_as_uint(part[b][jl][4 * v4]),
                                                                   __float_as_uint(part[b][jl][4 * v4 + 1]),
                                                                   __float_as_uint(part[b][jl][4 * v4 + 2]),
                                                                   __float_as_uint(part[b][jl][4 * v4 + 3])};
                }
            lds_barrier();
#pragma unroll
            for (int b = 0; b < 4; ++b)
                if ((b < 2) == (wi == 0)) {  // receiver
                    const int gj = j0 + wj * 128 + 32 * b + l32;
#pragma unroll
                    for (int jl = 0; jl < JBC; ++jl) {
#pragma unroll
                        for (int v4 = 0; v4 < 4; ++v4) {
                            const u32x4 o = slot(b, jl)[v4 * kWave + lane];
#pragma unroll
                            for (int e = 0; e < 4; ++e) part[b][jl][4 * v4 + e] += __uint_as_float(o[e]);
                        }
                        if (gj < C) {
#pragma unroll
                            for (int v = 0; v < 16; ++v) {
                                const int jr = 32 * (jb0 + jl) + 8 * (v >> 2) + 4 * h + (v & 3);
                                if (jr < r) atomicAdd(dA + (int64_t)jr * C + gj, s * part[b][jl][v]);
                            }
                        }
                    }
                }
            lds_barrier();  // exchange slots free again (and, after the last round, for G^T)
        }
    }

    // ---- epilogue 4: G^T -> LDS as [j][i] (pitch 512 B; the quad of 16-byte
    // chunks is XORed with j % 8 so that transpose reads of 4 consecutive j
    // hit different banks).  Lane (j, h) stores rows 8*v4 + 4h + {0..3}.
    auto gt_off = [](int j, int i) {
        return j * GT_PITCH + (((i >> 3) ^ ((j & 7) << 2)) << 4) + ((i & 7) << 1);
    };
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int jl = wj * 128 + 32 * b + l32;
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
                const int il = wi * 128 + 32 * a + 8 * v4 + 4 * h;
                const u32x4& gv = gb[a][b][v4 >> 1];
                u32x2 o;
                o[0] = gv[2 * (v4 & 1)];
                o[1] = gv[2 * (v4 & 1) + 1];
                *(u32x2*)(smem + gt_off(jl, il)) = o;
            }
        }

    // ---- epilogue 5: dB[i][j'] += s * sum_j G[i][j] A[j'][j], one 32-wide
    // rank block at a time: A[32jb .. +31][j0 .. j0+255] is copied to LDS and
    // wave w accumulates rows i = 64w .. 64w+63 of the tile, both 32-row blocks
    // together (each A fragment read once for the two).
    for (int jb = 0; jb < JB; ++jb) {
        if (jb > 0) copy_a_block(jb);  // block 0 was requested with the side data
        stage_barrier<0>();  // A block landed; G^T complete
        const int g = lane >> 4, jj = lane & 15;
        f32x16 db[2];
#pragma unroll
        for (int ib = 0; ib < 2; ++ib)
#pragma unroll
            for (int v = 0; v < 16; ++v) db[ib][v] = 0.f;
#pragma unroll 4
        for (int kc = 0; kc < BN / 16; ++kc) {
            const int jr0 = 16 * kc + 8 * (g >> 1) + (jj >> 2);
            const bf16x8 av = *(const bf16x8*)(smem + EP_A + tile_off(l32, 16 * kc + 8 * h));
#pragma unroll
            for (int ib = 0; ib < 2; ++ib) {
                const int ic = 64 * wave + 32 * ib + 16 * (g & 1) + 4 * (jj & 3);
                const bf16x8 ga = frag_from_tr(lds_tr_read(smem + gt_off(jr0, ic)), lds_tr_read(smem + gt_off(jr0 + 4, ic)));
                db[ib] = mfma_32x32x16(ga, av, db[ib]);
            }
        }
        const int jr = 32 * jb + l32;
        if (jr < r) {
#pragma unroll
            for (int ib = 0; ib < 2; ++ib)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int gi = i0 + 64 * wave + 32 * ib + 8 * (v >> 2) + 4 * h + (v & 3);
                    if (gi < R) atomicAdd(dB + (int64_t)gi * r + jr, s * db[ib][v]);
                }
        }
        lds_barrier();  // A block free for the next rank block
    }
}

template <int RK>
hipError_t launch_rk(const LayerArgs& a, hipStream_t st) {
    const int tiles_m = (int)((a.R + BM - 1) / BM);
    const int tiles_n = (int)((a.C + BN - 1) / BN);
    const TailSplit sp = tail_split((int64_t)tiles_m * tiles_n, (a.L + BK - 1) / BK, kNoPartials);
    dim3 grid(sp.grid), block(NT);
    auto* dY = (const uint16_t*)a.dY;
    auto* X = (const uint16_t*)a.X;
    auto* B = (const uint16_t*)a.B;
    auto* A = (const uint16_t*)a.A;
    // fixed-offset copies: whole tiles and K-steps, per-lane byte offsets
    // (64 token rows of R or C) inside 32 bits
    const bool ragged = a.R % BM != 0 || a.C % BN != 0 || a.L % BK != 0 ||
                        (int64_t)BK * a.R * 2 >= (1ll << 31) || (int64_t)BK * a.C * 2 >= (1ll << 31);
    if (ragged)
        hipLaunchKernelGGL((g_kernel<RK, true>), grid, block, 0, st, dY, X, a.Mt, B, A, a.dB, a.dA, a.L,
                           (int)a.R, (int)a.C, (int)a.r, a.scale, tiles_m, tiles_n, sp.n_full, sp.split);
    else
        hipLaunchKernelGGL((g_kernel<RK, false>), grid, block, 0, st, dY, X, a.Mt, B, A, a.dB, a.dA, a.L,
                           (int)a.R, (int)a.C, (int)a.r, a.scale, tiles_m, tiles_n, sp.n_full, sp.split);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_g_bf16(const LayerArgs& a, hipStream_t st) {
    if (a.L == 0) return hipSuccess;  // dB, dA stay zero
    switch ((a.r + 15) / 16) {
        case 1: return launch_rk<1>(a, st);
        case 2: return launch_rk<2>(a, st);
        case 3: return launch_rk<3>(a, st);
        case 4: return launch_rk<4>(a, st);
        case 5: return launch_rk<5>(a, st);
        case 6: return launch_rk<6>(a, st);
        case 7: return launch_rk<7>(a, st);
        case 8: return launch_rk<8>(a, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace lors
