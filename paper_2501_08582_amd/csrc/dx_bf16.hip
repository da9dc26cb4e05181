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
//     consecutive k of one column n -- come from two LDS transpose loads;
//   * the k-rows of the rank-r product are B[k][:], read from a B slab copied
//     contiguously into LDS each K-step; A[:, n] is resident in registers;
//   * the mask bits a lane needs run along k for a fixed n, so they are read
//     from the transposed bitmap M^T (built once per backward call).
// Requires r % 8 == 0 and r <= 64 (other ranks use the LDS-merge kernel).
#include "gemm_common.hpp"
#include "kernels.hpp"

namespace lors {
namespace {

constexpr int NT = 256;
constexpr int BM = 256;  // tokens per tile
constexpr int BN = 256;  // input features per tile (64 per wave)
constexpr int BK = 64;   // output features (rows of W) per K-step
constexpr int GROUP_M = 4;

constexpr int DB = BM * kRow64;      // dY slab: 32 KiB
constexpr int WB = BK * kRowBytes;   // W slab [k][n]: 32 KiB
constexpr int MB = BN * 2 * 4;       // M^T words [n][kb]: 2 KiB

template <int RK>
struct Layout {
    static constexpr int BB = BK * 32 * RK;        // B slab [k][r], pitch 2r <= 32*RK bytes
    static constexpr int D = 0, W = DB, B = DB + WB, M = DB + WB + BB;
    static constexpr int STAGE = DB + WB + BB + MB;
    static constexpr int LUT = 2 * STAGE;
    static constexpr int DUMMY = LUT + 4096;
    static constexpr int TOTAL = DUMMY + 1024;
    static constexpr int NB = (2 * RK + 3) / 4;    // B-slab copies per wave (r/8 copies in all)
    static constexpr int LOADS = 8 + 8 + NB + 2;
};

template <int RK, bool TWO_FOUR_UNUSED>
__global__ __launch_bounds__(NT, 1) void dx_kernel(
    const uint16_t* __restrict__ dY, const uint16_t* __restrict__ W,
    const uint32_t* __restrict__ Mt, const uint16_t* __restrict__ Bm,
    const uint16_t* __restrict__ Am, uint16_t* __restrict__ dX, int64_t L, int R, int C, int r,
    float s, int tiles_m, int tiles_n) {
    using Lay = Layout<RK>;
    static_assert(Lay::TOTAL <= 160 * 1024, "LDS budget");
    static_assert(16 * RK * kRowBytes <= Lay::STAGE, "A block fits one stage");
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
    const int nk = (R + BK - 1) / BK;
    const int wprT = (R + 31) >> 5;  // words per row of M^T
    const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
    const uint8_t* zsrc = (const uint8_t*)g_zero_page + 16 * lane;
    const int slab_b = 2 * r;        // bytes per B row
    const int nbcopies = r >> 3;     // 1 KiB copies per B slab (64 rows x 2r bytes)

    // M^T is a plain bitmap whatever the caller's layout.
    *(u32x4*)(smem + Lay::LUT + 16 * tid) = select_lut_entry<false>((uint32_t)tid);

    // ---- prologue: A[:, n0 .. n0+255] (16*RK rows) -> stage 1, then the
    // merge's B operand A[16c + 8h + e][n] into registers via transpose loads.
#pragma unroll
    for (int q = 0; q < 2 * RK; ++q) {
        const int blk = 4 * q + wave;
        const int row = 2 * blk + h;
        const int lc = swz_chunk(row, lane & 31);
        const int gn = n0 + 8 * lc;
        copy16_to_lds((row < r && gn < C) ? (const void*)(Am + (int64_t)row * C + gn) : (const void*)zsrc,
                      lds0 + Lay::STAGE + 1024 * blk);
    }
    stage_barrier<0>();
    bf16x8 afr[2][RK];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int c = 0; c < RK; ++c)
            afr[nb][c] = frag_from_tr(lds_tr_read(smem + Lay::STAGE + tr_frag_off(lane, 16 * c, 64 * wave + 32 * nb, 0)),
                                      lds_tr_read(smem + Lay::STAGE + tr_frag_off(lane, 16 * c, 64 * wave + 32 * nb, 1)));
    lds_barrier();

    auto issue = [&](int kt, int st) {
        const int k0 = kt * BK;
        const uint32_t sb = lds0 + st * Lay::STAGE;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int blk = 8 * wave + q;
            {   // dY slab: rows m, 64 k per row
                const int row = 8 * blk + (lane >> 3);
                const int lc = (lane & 7) ^ ((row >> 1) & 7);
                const int gk = k0 + 8 * lc;
                const int64_t gm = m0 + row;
                copy16_to_lds((gm < L && gk < R) ? (const void*)(dY + gm * R + gk) : (const void*)zsrc,
                              sb + Lay::D + 1024 * blk);
            }
            {   // W slab: rows k, 256 n per row
                const int row = 2 * blk + h;
                const int lc = swz_chunk(row, lane & 31);
                const int gk = k0 + row, gn = n0 + 8 * lc;
                copy16_to_lds((gk < R && gn < C) ? (const void*)(W + (int64_t)gk * C + gn) : (const void*)zsrc,
                              sb + Lay::W + 1024 * blk);
            }
        }
#pragma unroll
        for (int q = 0; q < Lay::NB; ++q) {  // B rows k0 .. k0+63: one contiguous block
            const int blk = 4 * q + wave;
            const bool real = blk < nbcopies;
            const int off = 1024 * blk + 16 * lane;   // byte offset inside the slab
            const bool ok = real && k0 + off / slab_b < R;
            copy16_to_lds(ok ? (const void*)((const uint8_t*)Bm + (int64_t)k0 * slab_b + off) : (const void*)zsrc,
                          real ? sb + Lay::B + 1024 * blk : lds0 + Lay::DUMMY);
        }
#pragma unroll
        for (int q = 0; q < 2; ++q) {      // M^T words: [n][kb]
            const int e = 64 * (2 * wave + q) + lane;
            const int n = e >> 1, kb = e & 1;
            const int gw = (k0 >> 5) + kb;
            const int gn = n0 + n;
            copy4_to_lds((gn < C && gw < wprT) ? (const void*)(Mt + (int64_t)gn * wprT + gw) : (const void*)zsrc,
                         sb + Lay::M + 256 * (2 * wave + q));
        }
    };

    // Rows of the merge A operand: lane (rho = l32, h) reads B row pi(rho).
    const int rho = l32;
    const int pik = 16 * (rho >> 4) + 8 * ((rho >> 2) & 1) + 4 * ((rho >> 3) & 1) + (rho & 3);
    const int ncol[2] = {64 * wave + l32, 64 * wave + 32 + l32};

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
            bf16x8 bfr[RK];  // B[32kb + pi(rho)][16c + 8h .. +7]
#pragma unroll
            for (int c = 0; c < RK; ++c) {
                const int j0 = 16 * c + 8 * h;
                u32x4 v = zero_u32x4();
                if (j0 < r) v = *(const u32x4*)(sb + Lay::B + (32 * kb + pik) * slab_b + 2 * j0);
                bfr[c] = as_bf16x8(v);
            }
            bf16x8 wf[2][2];
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) {
                f32x16 T;
#pragma unroll
                for (int v = 0; v < 16; ++v) T[v] = 0.f;
#pragma unroll
                for (int c = 0; c < RK; ++c) T = mfma_32x32x16(bfr[c], afr[nb][c], T);
                const uint32_t word = *(const uint32_t*)(sb + Lay::M + 8 * ncol[nb] + 4 * kb);
#pragma unroll
                for (int cp = 0; cp < 2; ++cp) {
                    const int row0 = 32 * kb + 16 * cp;
                    const u32x2 lo = lds_tr_read(sb + Lay::W + tr_frag_off(lane, row0, 64 * wave + 32 * nb, 0));
                    const u32x2 hi = lds_tr_read(sb + Lay::W + tr_frag_off(lane, row0, 64 * wave + 32 * nb, 1));
                    u32x4 raw;
                    raw[0] = lo[0]; raw[1] = lo[1]; raw[2] = hi[0]; raw[3] = hi[1];
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
                bf16x8 df[8];
#pragma unroll
                for (int mb = 0; mb < 8; ++mb)
                    df[mb] = *(const bf16x8*)(sb + Lay::D + slab64_off(32 * mb + l32, 2 * c4 + h));
#pragma unroll
                for (int mb = 0; mb < 8; ++mb)
#pragma unroll
                    for (int nb = 0; nb < 2; ++nb) acc[mb][nb] = mfma_32x32x16(df[mb], wf[nb][cp], acc[mb][nb]);
            }
        }
        lds_barrier();
        if (kt + 2 < nk) issue(kt + 2, st);
    }

#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
        const int gn = n0 + ncol[nb];
        if (gn >= C) continue;
#pragma unroll
        for (int mb = 0; mb < 8; ++mb) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t gm = m0 + 32 * mb + 8 * (v >> 2) + 4 * h + (v & 3);
                if (gm < L) dX[gm * C + gn] = bf16_bits(acc[mb][nb][v]);
            }
        }
    }
}

template <int RK>
hipError_t launch_rk(const LayerArgs& a, hipStream_t st) {
    const int tiles_m = (int)((a.L + BM - 1) / BM);
    const int tiles_n = (int)((a.C + BN - 1) / BN);
    dim3 grid(tiles_m * tiles_n), block(NT);
    hipLaunchKernelGGL((dx_kernel<RK, false>), grid, block, 0, st, (const uint16_t*)a.dY, (const uint16_t*)a.W,
                       a.Mt, (const uint16_t*)a.B, (const uint16_t*)a.A, (uint16_t*)a.dX, a.L, (int)a.R,
                       (int)a.C, (int)a.r, a.scale, tiles_m, tiles_n);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_dx_bf16(const LayerArgs& a, hipStream_t st) {
    if (a.L == 0 || a.dX == nullptr) return hipSuccess;
    if (a.r % 8 != 0 || a.Mt == nullptr) return launch_dx_bf16_wide(a, st);
    switch ((a.r + 15) / 16) {
        case 1: return launch_rk<1>(a, st);
        case 2: return launch_rk<2>(a, st);
        case 3: return launch_rk<3>(a, st);
        case 4: return launch_rk<4>(a, st);
        default: return launch_dx_bf16_wide(a, st);
    }
}

}  // namespace lors
