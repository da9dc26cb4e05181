// Backward data gradient for adapter ranks above 64 or not a multiple of 8
// (8 waves, W' rebuilt in LDS).
//
//   dX[L x C] = dY[L x R] . W',   W' = select(M, W + s.B.A, 0)
//
// (dX step of the SP-LoRA backward list in Section 2.2; the merged weight is
// recomputed instead of stored, Algorithm 2 / Section 2.3.)  The GEMM runs
// over K = R.  Each K-step stages the dY tile and the raw W tile (64 rows of
// R, natural layout), rebuilds W' for that tile with a rank-r MFMA, and writes
// W' transposed into LDS so that both MFMA operands are read K-contiguous.
#include "device_common.hpp"
#include "kernels.hpp"

namespace lors {
namespace wide {
namespace {  // file-local: both wide kernels have launchers of the same shape

constexpr int BM = 256;  // tokens per tile (GEMM M)
constexpr int BN = 256;  // input features per tile (GEMM N)
constexpr int BK = 64;   // rows of W (output features) per K-step
constexpr int NT = 512;
constexpr int WM = 2, WN = 4;
constexpr int FM = BM / WM / 32;
constexpr int FN = BN / WN / 32;
constexpr int LDT = BK + 8;   // pitch of the dY tile and of the transposed W' tile
constexpr int LDW = BN + 8;   // pitch of the raw W tile (rows of R)
constexpr int GROUP_M = 4;

static_assert(BN / 32 == NT / kWave, "one merge n-block per wave");

constexpr int kDsBytes = BM * LDT * 2;
constexpr int kWnBytes = BK * LDW * 2;
constexpr int kWtBytes = BN * LDT * 2;
constexpr int kSmemBytes = kDsBytes + kWnBytes + kWtBytes;

template <int RK, bool TWO_FOUR>
__global__ __launch_bounds__(NT, 1) void dx_kernel_wide(
    const uint16_t* __restrict__ dY, const uint16_t* __restrict__ W,
    const uint32_t* __restrict__ Mp, const uint16_t* __restrict__ Bm,
    const uint16_t* __restrict__ Am, uint16_t* __restrict__ dX, int64_t L, int R, int C,
    int r, float s, int tiles_m, int tiles_n) {
    constexpr int LDA = RK * 16 + 8;  // pitch of the transposed A block (rows = n)
    static_assert(BN * LDA * 2 <= kWnBytes + kWtBytes, "A block fits the W regions");
    __shared__ __attribute__((aligned(16))) uint8_t smem[kSmemBytes];
    uint16_t* Ds = (uint16_t*)smem;                            // [m][k]
    uint16_t* Wn = (uint16_t*)(smem + kDsBytes);               // [k][n] raw W
    uint16_t* Wt = (uint16_t*)(smem + kDsBytes + kWnBytes);    // [n][k] W'
    uint16_t* Ast = (uint16_t*)(smem + kDsBytes);              // [n][j], prologue only

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int l32 = lane & 31;
    const int h = lane >> 5;

    int tm, tn;
    tile_coords(blockIdx.x, tiles_m, tiles_n, GROUP_M, tm, tn);
    const int64_t m0 = (int64_t)tm * BM;
    const int n0 = tn * BN;
    const int nk = (R + BK - 1) / BK;
    const int wpr = (C + 31) >> 5;
    const bool b_vec = (r & 7) == 0;

    // Prologue: A[:, n0 .. n0+255] transposed into LDS, then each wave keeps
    // the merge operand A^T[32*wave + l32][16c + 8h .. +7] in registers.
    for (int c = tid; c < RK * 16 * (BN / 8); c += NT) {
        const int j = c / (BN / 8), nc = c % (BN / 8);
        const int gn = n0 + nc * 8;
        const u32x4 v = (j < r && gn < C) ? *(const u32x4*)(Am + (int64_t)j * C + gn) : zero_u32x4();
#pragma unroll
        for (int e = 0; e < 8; ++e) Ast[(nc * 8 + e) * LDA + j] = (uint16_t)u16_at(v, e);
    }
    __syncthreads();
    bf16x8 afr[RK];
#pragma unroll
    for (int c = 0; c < RK; ++c)
        afr[c] = *(const bf16x8*)(Ast + (wave * 32 + l32) * LDA + 16 * c + 8 * h);
    __syncthreads();

    const int nw = (n0 >> 5) + wave;  // mask word column of this wave's merge rows
    u32x4 dr[4], wr[4];
    bf16x8 bfr[2][RK];
    uint32_t mw[2];

    auto load_tiles = [&](int kt) {
        const int k0 = kt * BK;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int c = tid + q * NT;
            {   // dY tile: 256 rows (tokens) x 64 columns (R)
                const int row = c >> 3, kc = c & 7;
                const int gk = k0 + kc * 8;
                const int64_t gm = m0 + row;
                dr[q] = (gm < L && gk < R) ? *(const u32x4*)(dY + gm * R + gk) : zero_u32x4();
            }
            {   // raw W tile: 64 rows (R) x 256 columns (C)
                const int row = c >> 5, nc = c & 31;
                const int gk = k0 + row, gn = n0 + nc * 8;
                wr[q] = (gk < R && gn < C) ? *(const u32x4*)(W + (int64_t)gk * C + gn) : zero_u32x4();
            }
        }
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const int gk = k0 + 32 * kb + l32;
#pragma unroll
            for (int c = 0; c < RK; ++c) {
                u32x4 v = zero_u32x4();
                if (gk < R) {
                    const uint16_t* src = Bm + (int64_t)gk * r + 16 * c + 8 * h;
                    if (b_vec) {
                        if (16 * c + 8 * h < r) v = *(const u32x4*)src;
                    } else {
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const uint32_t x = (16 * c + 8 * h + e < r) ? (uint32_t)src[e] : 0u;
                            v[e >> 1] |= x << ((e & 1) * 16);
                        }
                    }
                }
                bfr[kb][c] = as_bf16x8(v);
            }
            mw[kb] = (gk < R && nw < wpr) ? Mp[(int64_t)gk * wpr + nw] : 0u;
        }
    };

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const int wm = wave / WN, wn = wave % WN;

    load_tiles(0);
    for (int kt = 0; kt < nk; ++kt) {
        __syncthreads();
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int c = tid + q * NT;
            *(u32x4*)(Ds + (c >> 3) * LDT + (c & 7) * 8) = dr[q];
            *(u32x4*)(Wn + (c >> 5) * LDW + (c & 31) * 8) = wr[q];
        }
        __syncthreads();

        // Merge: C[n][k] = sum_j A[j][n] B[k][j] for this wave's 32 columns n
        // and the 64 rows k of the step; lane (l32, h) owns row k = 32kb + l32
        // and columns n = 32*wave + 8i + 4h + q.
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            f32x16 T;
#pragma unroll
            for (int v = 0; v < 16; ++v) T[v] = 0.f;
#pragma unroll
            for (int c = 0; c < RK; ++c) T = mfma_32x32x16(afr[c], bfr[kb][c], T);
            const int kl = 32 * kb + l32;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int nl = wave * 32 + 8 * i + 4 * h;
                const u32x2 wv = *(const u32x2*)(Wn + kl * LDW + nl);
                const uint32_t keep = keep4<TWO_FOUR>(mw[kb], 8 * i + 4 * h);
                float w0 = fmaf(s, T[4 * i + 0], bf16_bits_to_f32(wv[0] & 0xFFFFu));
                float w1 = fmaf(s, T[4 * i + 1], bf16_bits_to_f32(wv[0] >> 16));
                float w2 = fmaf(s, T[4 * i + 2], bf16_bits_to_f32(wv[1] & 0xFFFFu));
                float w3 = fmaf(s, T[4 * i + 3], bf16_bits_to_f32(wv[1] >> 16));
                Wt[(nl + 0) * LDT + kl] = (keep & 1u) ? bf16_bits(w0) : (uint16_t)0;
                Wt[(nl + 1) * LDT + kl] = (keep & 2u) ? bf16_bits(w1) : (uint16_t)0;
                Wt[(nl + 2) * LDT + kl] = (keep & 4u) ? bf16_bits(w2) : (uint16_t)0;
                Wt[(nl + 3) * LDT + kl] = (keep & 8u) ? bf16_bits(w3) : (uint16_t)0;
            }
        }
        __syncthreads();

        if (kt + 1 < nk) load_tiles(kt + 1);

#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            bf16x8 a[FM], b[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i)
                a[i] = *(const bf16x8*)(Ds + (wm * (BM / WM) + 32 * i + l32) * LDT + 16 * ks + 8 * h);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                b[j] = *(const bf16x8*)(Wt + (wn * (BN / WN) + 32 * j + l32) * LDT + 16 * ks + 8 * h);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = mfma_32x32x16(a[i], b[j], acc[i][j]);
        }
    }

#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int gn = n0 + wn * (BN / WN) + 32 * j + l32;
        if (gn >= C) continue;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t gm = m0 + wm * (BM / WM) + 32 * i + 8 * (v >> 2) + 4 * h + (v & 3);
                if (gm < L) dX[gm * C + gn] = bf16_bits(acc[i][j][v]);
            }
        }
    }
}

template <int RK>
hipError_t launch_wide(const LayerArgs& a, hipStream_t st) {
    const int tiles_m = (int)((a.L + BM - 1) / BM);
    const int tiles_n = (int)((a.C + BN - 1) / BN);
    dim3 grid(tiles_m * tiles_n), block(NT);
    auto* dY = (const uint16_t*)a.dY;
    auto* W = (const uint16_t*)a.W;
    auto* B = (const uint16_t*)a.B;
    auto* A = (const uint16_t*)a.A;
    auto* dX = (uint16_t*)a.dX;
    if (a.two_four)
        hipLaunchKernelGGL((dx_kernel_wide<RK, true>), grid, block, 0, st, dY, W, a.M, B, A, dX, a.L,
                           (int)a.R, (int)a.C, (int)a.r, a.scale, tiles_m, tiles_n);
    else
        hipLaunchKernelGGL((dx_kernel_wide<RK, false>), grid, block, 0, st, dY, W, a.M, B, A, dX, a.L,
                           (int)a.R, (int)a.C, (int)a.r, a.scale, tiles_m, tiles_n);
    return hipGetLastError();
}

}  // namespace
}  // namespace wide

hipError_t launch_dx_bf16_wide(const LayerArgs& a, hipStream_t st) {
    if (a.L == 0 || a.dX == nullptr) return hipSuccess;
    switch ((a.r + 15) / 16) {
        case 1: return wide::launch_wide<1>(a, st);
        case 2: return wide::launch_wide<2>(a, st);
        case 3: return wide::launch_wide<3>(a, st);
        case 4: return wide::launch_wide<4>(a, st);
        case 5: return wide::launch_wide<5>(a, st);
        case 6: return wide::launch_wide<6>(a, st);
        case 7: return wide::launch_wide<7>(a, st);
        case 8: return wide::launch_wide<8>(a, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace lors
