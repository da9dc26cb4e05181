// Fused forward of the sparsity-preserved LoRA linear, bf16 on gfx950.
//
//   Y[L x R] = X[L x C] . W'^T,   W' = select(M, W + s.B.A, 0)
//
// (Eq. 3 of Section 2.2 and Algorithm 1, with the listing's scale factor.)
// W' never reaches HBM, and never even reaches LDS: each of the 4 waves owns
// 64 output features (n) of the 256 x 256 tile and rebuilds exactly those 64
// rows of W' per K-step in registers, in the operand layout of the main MFMA.
//
// Merge: the rank-r product T = B.A for a 32(k) x 32(n) block is one
// 32x32x16 MFMA per 16 ranks whose A operand is A^T with its 32 rows taken in
// the order pi(8i + 4h + q) = 16(i/2) + 8h + 4(i%2) + q.  With that order the
// 16 accumulator values a lane holds are, in register order, the k values
// 16c + 8h + {0..7} for c = 0, 1 -- exactly two 32x32x16 B-operand fragments.
// Each lane then adds its W values (one 16-byte LDS read per fragment), picks
// the select masks for its eight k from a 256-entry LUT indexed by the mask
// byte, rounds once to bf16, and feeds the MFMA directly.
//
// Data movement: X, W and A slabs for a 64-wide K-step are copied from HBM
// into LDS with global_load_lds (no registers), double-buffered; the mask
// words come the same way.  Accumulators (256 x 64 per wave) live in AGPRs.
#include "gemm_common.hpp"
#include "kernels.hpp"

namespace lors {
namespace {

constexpr int NT = 256;
constexpr int BM = 256;   // tokens per tile
constexpr int BN = 256;   // output features per tile (64 per wave)
constexpr int BK = 64;    // input features per K-step
constexpr int GROUP_M = 4;
constexpr int MAXRK = 4;  // ranks up to 64 (wider ranks use the LDS-merge kernel)

constexpr int XB = BM * kRow64;  // 32 KiB
constexpr int WB = BN * kRow64;  // 32 KiB
constexpr int MB = BN * 2 * 4;   // 2 mask words per row of W: 2 KiB

template <int RK>
struct Layout {
    static constexpr int AB = 16 * RK * kRow64;   // A slab: 16*RK rows of 64 k
    static constexpr int X = 0, W = XB, A = XB + WB, M = XB + WB + AB;
    static constexpr int STAGE = XB + WB + AB + MB;
    static constexpr int LUT = 2 * STAGE;         // 256 x 16 B
    static constexpr int DUMMY = LUT + 4096;      // 1 KiB sink for padding copies
    static constexpr int TOTAL = DUMMY + 1024;
    static constexpr int NA = (2 * RK + 3) / 4;   // A-slab copies per wave
    static constexpr int LOADS = 8 + 8 + NA + 2;  // copies per wave per stage
};

template <int RK, bool TWO_FOUR>
__global__ __launch_bounds__(NT, 1) void fwd_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
    const uint32_t* __restrict__ Mp, const uint16_t* __restrict__ Bm,
    const uint16_t* __restrict__ Am, const uint16_t* __restrict__ bias,
    uint16_t* __restrict__ Y, int64_t L, int R, int C, int r, float s, int tiles_m,
    int tiles_n) {
    using Lay = Layout<RK>;
    static_assert(Lay::TOTAL <= 160 * 1024, "LDS budget");
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
    const uint8_t* zsrc = (const uint8_t*)g_zero_page + 16 * lane;

    // ---- select LUT (visible to all waves after the first stage barrier)
    // and the resident B operand of the merge
    *(u32x4*)(smem + Lay::LUT + 16 * tid) = select_lut_entry<TWO_FOUR>((uint32_t)tid);

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

    // ---- asynchronous slab copies for K-step kt into stage st
    auto issue = [&](int kt, int st) {
        const int k0 = kt * BK;
        const uint32_t sb = lds0 + st * Lay::STAGE;
#pragma unroll
        for (int q = 0; q < 8; ++q) {      // X and W: 8 rows x 8 chunks per copy
            const int blk = 8 * wave + q;
            const int row = 8 * blk + (lane >> 3);
            const int lc = (lane & 7) ^ ((row >> 1) & 7);
            const int gk = k0 + 8 * lc;
            const int64_t gm = m0 + row;
            const int gn = n0 + row;
            copy16_to_lds((gm < L && gk < C) ? (const void*)(X + gm * C + gk) : (const void*)zsrc,
                          sb + Lay::X + 1024 * blk);
            copy16_to_lds((gn < R && gk < C) ? (const void*)(W + (int64_t)gn * C + gk) : (const void*)zsrc,
                          sb + Lay::W + 1024 * blk);
        }
#pragma unroll
        for (int q = 0; q < Lay::NA; ++q) {  // A: 16*RK rows; copies beyond go to the sink
            const int blk = 4 * q + wave;
            const int row = 8 * blk + (lane >> 3);
            const int lc = (lane & 7) ^ ((row >> 1) & 7);
            const int gk = k0 + 8 * lc;
            const bool real = blk < 2 * RK;
            const bool ok = real && row < r && gk < C;
            copy16_to_lds(ok ? (const void*)(Am + (int64_t)row * C + gk) : (const void*)zsrc,
                          real ? sb + Lay::A + 1024 * blk : lds0 + Lay::DUMMY);
        }
#pragma unroll
        for (int q = 0; q < 2; ++q) {      // mask words: [row n][kb]
            const int e = 64 * (2 * wave + q) + lane;
            const int row = e >> 1, kb = e & 1;
            const int gw = (k0 >> 5) + kb;
            const int gn = n0 + row;
            copy4_to_lds((gn < R && gw < wpr) ? (const void*)(Mp + (int64_t)gn * wpr + gw) : (const void*)zsrc,
                         sb + Lay::M + 256 * (2 * wave + q));
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
                offAt[kb][t] = Lay::A + slab64_elem_off(row, col);
            }
    }
    const int nrow[2] = {64 * wave + l32, 64 * wave + 32 + l32};

    f32x16 acc[8][2];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    issue(0, 0);
    if (nk > 1) issue(1, 1);

    for (int kt = 0; kt < nk; ++kt) {
        const int st = kt & 1;
        if (kt + 1 < nk)
            stage_barrier<Lay::LOADS>();
        else
            stage_barrier<0>();
        const uint8_t* sb = smem + st * Lay::STAGE;

#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            // A^T fragments for this 32-wide half of the K-step
            bf16x8 afr[RK];
#pragma unroll
            for (int c = 0; c < RK; ++c)
                afr[c] = frag_from_tr(lds_tr_read(sb + offAt[kb][0] + 16 * kRow64 * c),
                                      lds_tr_read(sb + offAt[kb][1] + 16 * kRow64 * c));
            bf16x8 wf[2][2];  // [nb][c'] merged W' fragments for chunks 2kb + c'
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) {
                f32x16 T;
#pragma unroll
                for (int v = 0; v < 16; ++v) T[v] = 0.f;
#pragma unroll
                for (int c = 0; c < RK; ++c) T = mfma_32x32x16(afr[c], bfr[nb][c], T);
                const uint32_t word = *(const uint32_t*)(sb + Lay::M + 8 * nrow[nb] + 4 * kb);
#pragma unroll
                for (int cp = 0; cp < 2; ++cp) {
                    const u32x4 raw = *(const u32x4*)(sb + Lay::W + slab64_off(nrow[nb], 4 * kb + 2 * cp + h));
                    const uint32_t byte = (word >> (8 * (2 * cp + h))) & 0xFFu;
                    const u32x4 sel = *(const u32x4*)(smem + Lay::LUT + 16 * byte);
                    float t8[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) t8[e] = T[8 * cp + e];
                    wf[nb][cp] = as_bf16x8(merge8(raw, t8, s, sel));
                }
            }
#pragma unroll
            for (int cp = 0; cp < 2; ++cp) {
                const int c4 = 2 * kb + cp;
                bf16x8 xf[8];
#pragma unroll
                for (int mb = 0; mb < 8; ++mb)
                    xf[mb] = *(const bf16x8*)(sb + Lay::X + slab64_off(32 * mb + l32, 2 * c4 + h));
#pragma unroll
                for (int mb = 0; mb < 8; ++mb)
#pragma unroll
                    for (int nb = 0; nb < 2; ++nb) acc[mb][nb] = mfma_32x32x16(xf[mb], wf[nb][cp], acc[mb][nb]);
            }
        }
        lds_barrier();
        if (kt + 2 < nk) issue(kt + 2, st);
    }

    // ---- epilogue: (+bias), round to bf16, store
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
        const int gn = n0 + nrow[nb];
        if (gn >= R) continue;
        const float bv = bias ? bf16_bits_to_f32(bias[gn]) : 0.f;
#pragma unroll
        for (int mb = 0; mb < 8; ++mb) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t gm = m0 + 32 * mb + 8 * (v >> 2) + 4 * h + (v & 3);
                if (gm < L) Y[gm * R + gn] = bf16_bits(acc[mb][nb][v] + bv);
            }
        }
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
    if (a.two_four)
        hipLaunchKernelGGL((fwd_kernel<RK, true>), grid, block, 0, st, X, W, a.M, B, A, bias, Y, a.L,
                           (int)a.R, (int)a.C, (int)a.r, a.scale, tiles_m, tiles_n);
    else
        hipLaunchKernelGGL((fwd_kernel<RK, false>), grid, block, 0, st, X, W, a.M, B, A, bias, Y, a.L,
                           (int)a.R, (int)a.C, (int)a.r, a.scale, tiles_m, tiles_n);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_fwd_bf16(const LayerArgs& a, hipStream_t st) {
    if (a.L == 0) return hipSuccess;
    switch ((a.r + 15) / 16) {
        case 1: return launch_rk<1>(a, st);
        case 2: return launch_rk<2>(a, st);
        case 3: return launch_rk<3>(a, st);
        case 4: return launch_rk<4>(a, st);
        default: return launch_fwd_bf16_wide(a, st);
    }
}

}  // namespace lors
