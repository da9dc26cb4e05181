// Forward for adapter ranks above 64 (8 waves, W' merged in place in LDS).
//
//   Y[L x R] = X[L x C] . W'^T,   W' = select(M, W + s.B.A, 0)
//
// (Eq. 3 of Section 2.2 and Algorithm 1, with the listing's scale factor.)
// For each K-step a workgroup stages its X tile and its raw W tile, runs the
// rank-r product B_blk . A_blk on the matrix cores, adds it to W in fp32,
// applies the mask as a select, rounds once to bf16 and overwrites the raw W
// tile with W' in place; the main MFMA loop then reads X and W' from LDS.
#include "device_common.hpp"
#include "kernels.hpp"

namespace lors {
namespace wide {
namespace {  // file-local: both wide kernels have launchers of the same shape

constexpr int BM = 256;  // tokens per tile (GEMM M)
constexpr int BN = 256;  // output features per tile (GEMM N)
constexpr int BK = 64;   // input features per K-step
constexpr int NT = 512;  // 8 waves
constexpr int WM = 2, WN = 4;
constexpr int FM = BM / WM / 32;  // 32x32 blocks per wave along M
constexpr int FN = BN / WN / 32;  // ... along N
constexpr int LDT = BK + 8;       // LDS row pitch (elements) of the X and W tiles
constexpr int GROUP_M = 4;

static_assert(BN / 32 == NT / kWave, "one merge n-block per wave");

template <int RK, bool TWO_FOUR>
__global__ __launch_bounds__(NT, 1) void fwd_kernel_wide(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
    const uint32_t* __restrict__ Mp, const uint16_t* __restrict__ Bm,
    const uint16_t* __restrict__ Am, const uint16_t* __restrict__ bias,
    uint16_t* __restrict__ Y, int64_t L, int R, int C, int r, float s, int tiles_m,
    int tiles_n) {
    constexpr int LDA = RK * 16 + 8;           // pitch of the transposed A block
    constexpr int ACH = (RK * 16 * 8 + NT - 1) / NT;  // 16B chunks of A per thread
    __shared__ __attribute__((aligned(16))) uint16_t Xs[BM * LDT];
    __shared__ __attribute__((aligned(16))) uint16_t Ws[BN * LDT];
    __shared__ __attribute__((aligned(16))) uint16_t At[BK * LDA];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int l32 = lane & 31;
    const int h = lane >> 5;

    int tm, tn;
    tile_coords(blockIdx.x, tiles_m, tiles_n, GROUP_M, tm, tn);
    const int64_t m0 = (int64_t)tm * BM;
    const int n0 = tn * BN;
    const int nk = (C + BK - 1) / BK;
    const int wpr = (C + 31) >> 5;

    // Rank-r operand of the merge held for the whole tile: lane (l32, h) keeps
    // B[n0 + 32*wave + l32][16c + 8h .. +7] for every 16-wide rank chunk c.
    const int nl_merge = wave * 32 + l32;
    const int gn_merge = n0 + nl_merge;
    bf16x8 bfr[RK];
#pragma unroll
    for (int c = 0; c < RK; ++c) {
        u32x4 v = zero_u32x4();
        if (gn_merge < R) {
            const uint16_t* src = Bm + (int64_t)gn_merge * r;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int j = 16 * c + 8 * h + e;
                const uint32_t x = (j < r) ? (uint32_t)src[j] : 0u;
                v[e >> 1] |= x << ((e & 1) * 16);
            }
        }
        bfr[c] = as_bf16x8(v);
    }

    u32x4 xr[4], wr[4], ar[ACH];
    uint32_t mw[2];

    auto load_tiles = [&](int kt) {
        const int k0 = kt * BK;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int c = tid + q * NT;
            const int row = c >> 3, kc = c & 7;
            const int gk = k0 + kc * 8;
            const int64_t gm = m0 + row;
            const int gn = n0 + row;
            xr[q] = (gm < L && gk < C) ? *(const u32x4*)(X + gm * C + gk) : zero_u32x4();
            wr[q] = (gn < R && gk < C) ? *(const u32x4*)(W + (int64_t)gn * C + gk) : zero_u32x4();
        }
#pragma unroll
        for (int q = 0; q < ACH; ++q) {
            const int c = tid + q * NT;
            const int j = c >> 3, kc = c & 7;
            const int gk = k0 + kc * 8;
            ar[q] = (c < RK * 128 && j < r && gk < C) ? *(const u32x4*)(Am + (int64_t)j * C + gk)
                                                       : zero_u32x4();
        }
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const int gk = k0 + 32 * kb;
            mw[kb] = (gn_merge < R && gk < C) ? Mp[(int64_t)gn_merge * wpr + (gk >> 5)] : 0u;
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
        __syncthreads();  // the previous step's MFMAs are done with Xs / Ws / At
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int c = tid + q * NT;
            const int row = c >> 3, kc = c & 7;
            *(u32x4*)(Xs + row * LDT + kc * 8) = xr[q];
            *(u32x4*)(Ws + row * LDT + kc * 8) = wr[q];
        }
#pragma unroll
        for (int q = 0; q < ACH; ++q) {
            const int c = tid + q * NT;
            if (c < RK * 128) {
                const int j = c >> 3, kc = c & 7;
#pragma unroll
                for (int e = 0; e < 8; ++e) At[(kc * 8 + e) * LDA + j] = (uint16_t)u16_at(ar[q], e);
            }
        }
        const uint32_t mcur0 = mw[0], mcur1 = mw[1];
        __syncthreads();

        // Merge: W'[n][k] for this wave's 32 rows n and the 64 columns k of
        // the step, computed as C[k][n] = sum_j A[j][k] B[n][j] so that each
        // lane ends up owning four consecutive k of one row n.
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            f32x16 T;
#pragma unroll
            for (int v = 0; v < 16; ++v) T[v] = 0.f;
#pragma unroll
            for (int c = 0; c < RK; ++c) {
                const bf16x8 afr = *(const bf16x8*)(At + (32 * kb + l32) * LDA + 16 * c + 8 * h);
                T = mfma_32x32x16(afr, bfr[c], T);
            }
            const uint32_t word = kb ? mcur1 : mcur0;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int kl = 32 * kb + 8 * i + 4 * h;
                u32x2* p = (u32x2*)(Ws + nl_merge * LDT + kl);
                u32x2 wv = *p;
                const uint32_t keep = keep4<TWO_FOUR>(word, 8 * i + 4 * h);
                float w0 = fmaf(s, T[4 * i + 0], bf16_bits_to_f32(wv[0] & 0xFFFFu));
                float w1 = fmaf(s, T[4 * i + 1], bf16_bits_to_f32(wv[0] >> 16));
                float w2 = fmaf(s, T[4 * i + 2], bf16_bits_to_f32(wv[1] & 0xFFFFu));
                float w3 = fmaf(s, T[4 * i + 3], bf16_bits_to_f32(wv[1] >> 16));
                w0 = (keep & 1u) ? w0 : 0.f;
                w1 = (keep & 2u) ? w1 : 0.f;
                w2 = (keep & 4u) ? w2 : 0.f;
                w3 = (keep & 8u) ? w3 : 0.f;
                wv[0] = pack_bf16x2(w0, w1);
                wv[1] = pack_bf16x2(w2, w3);
                *p = wv;
            }
        }
        __syncthreads();

        if (kt + 1 < nk) load_tiles(kt + 1);

#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            bf16x8 a[FM], b[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i)
                a[i] = *(const bf16x8*)(Xs + (wm * (BM / WM) + 32 * i + l32) * LDT + 16 * ks + 8 * h);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                b[j] = *(const bf16x8*)(Ws + (wn * (BN / WN) + 32 * j + l32) * LDT + 16 * ks + 8 * h);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = mfma_32x32x16(a[i], b[j], acc[i][j]);
        }
    }

    // Epilogue: (+bias), round to bf16, store.
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int gn = n0 + wn * (BN / WN) + 32 * j + l32;
        if (gn >= R) continue;
        const float bv = bias ? bf16_bits_to_f32(bias[gn]) : 0.f;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t gm = m0 + wm * (BM / WM) + 32 * i + 8 * (v >> 2) + 4 * h + (v & 3);
                if (gm < L) Y[gm * R + gn] = bf16_bits(acc[i][j][v] + bv);
            }
        }
    }
}

template <int RK>
hipError_t launch_wide(const LayerArgs& a, hipStream_t st) {
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
        hipLaunchKernelGGL((fwd_kernel_wide<RK, true>), grid, block, 0, st, X, W, a.M, B, A, bias, Y,
                           a.L, (int)a.R, (int)a.C, (int)a.r, a.scale, tiles_m, tiles_n);
    else
        hipLaunchKernelGGL((fwd_kernel_wide<RK, false>), grid, block, 0, st, X, W, a.M, B, A, bias, Y,
                           a.L, (int)a.R, (int)a.C, (int)a.r, a.scale, tiles_m, tiles_n);
    return hipGetLastError();
}

}  // namespace
}  // namespace wide

hipError_t launch_fwd_bf16_wide(const LayerArgs& a, hipStream_t st) {
    if (a.L == 0) return hipSuccess;
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
