// Backward adapter gradients, bf16 on gfx950.
//
//   G  = select(M, dY^T . X, 0)      (R x C, never written to HBM)
//   dB += s . G . A^T   (R x r, fp32)     dA += s . B^T . G   (r x C, fp32)
//
// (I_w^4, I_w^5 and the two adapter gradients of the SP-LoRA backward list in
// Section 2.2, with the scale of the listing.)  The weight-gradient GEMM runs
// over K = L with both operands token-major, so each K-step transposes its dY
// and X tiles into LDS.  After the K loop the fp32 accumulators are masked in
// registers, rounded to bf16, and fed to two rank-r MFMA products whose
// per-tile partial sums are added into dB and dA with fp32 atomics (dB and dA
// must be zero on entry).
#include "device_common.hpp"
#include "kernels.hpp"

namespace lors {
namespace {

constexpr int BM = 256;  // rows of G (output features, R) per tile
constexpr int BN = 256;  // columns of G (input features, C) per tile
constexpr int BK = 64;   // tokens per K-step
constexpr int NT = 512;
constexpr int WM = 2, WN = 4;
constexpr int FM = BM / WM / 32;
constexpr int FN = BN / WN / 32;
constexpr int LDT = BK + 8;   // pitch of the transposed tiles [i][l] and [j][l]
constexpr int LDG = BN + 8;   // pitch of the bf16 G tile [i][j]
constexpr int GROUP_M = 4;

constexpr int kMainBytes = (BM + BN) * LDT * 2;
constexpr int kGBytes = BM * LDG * 2;
constexpr int kSmemBytes = kMainBytes > kGBytes ? kMainBytes : kGBytes;

static_assert(BM / 32 == NT / kWave, "one dB row block per wave");

template <int RK, bool TWO_FOUR>
__global__ __launch_bounds__(NT, 1) void g_kernel(
    const uint16_t* __restrict__ dY, const uint16_t* __restrict__ X,
    const uint32_t* __restrict__ Mp, const uint16_t* __restrict__ Bm,
    const uint16_t* __restrict__ Am, float* __restrict__ dB, float* __restrict__ dA,
    int64_t L, int R, int C, int r, float s, int tiles_m, int tiles_n) {
    constexpr int JB = (RK + 1) / 2;         // 32-wide blocks of the rank
    constexpr int LDB = BM + 8;              // pitch of B^T [j][i]
    static_assert(JB * 32 * LDB * 2 <= kSmemBytes, "B^T fits");
    __shared__ __attribute__((aligned(16))) uint8_t smem[kSmemBytes];
    uint16_t* Dt = (uint16_t*)smem;                    // [i][l]
    uint16_t* Xt = (uint16_t*)(smem + BM * LDT * 2);   // [j][l]
    uint16_t* Gs = (uint16_t*)smem;                    // [i][j], epilogue
    uint16_t* Bt = (uint16_t*)smem;                    // [j'][i], epilogue

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int l32 = lane & 31;
    const int h = lane >> 5;

    int tm, tn;
    tile_coords(blockIdx.x, tiles_m, tiles_n, GROUP_M, tm, tn);
    const int i0 = tm * BM;
    const int j0 = tn * BN;
    const int64_t nk = (L + BK - 1) / BK;
    const int wpr = (C + 31) >> 5;

    // K-step staging: thread t loads rows 4*(t/32) .. +3 of the token block and
    // 8 consecutive columns starting at 8*(t%32), for dY (columns = R) and X
    // (columns = C), then writes them transposed, four tokens per 8-byte store.
    const int cq = tid & 31;
    const int rg = tid >> 5;
    u32x4 dr[4], xr[4];

    auto load_tiles = [&](int64_t kt) {
        const int64_t l0 = kt * BK + 4 * rg;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t gl = l0 + q;
            const int gi = i0 + cq * 8, gj = j0 + cq * 8;
            dr[q] = (gl < L && gi < R) ? *(const u32x4*)(dY + gl * R + gi) : zero_u32x4();
            xr[q] = (gl < L && gj < C) ? *(const u32x4*)(X + gl * C + gj) : zero_u32x4();
        }
    };

    auto store_transposed = [&](uint16_t* dst, const u32x4* v) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int sh = (e & 1) * 16;
            const int w = e >> 1;
            u32x2 o;
            o[0] = ((v[0][w] >> sh) & 0xFFFFu) | (((v[1][w] >> sh) & 0xFFFFu) << 16);
            o[1] = ((v[2][w] >> sh) & 0xFFFFu) | (((v[3][w] >> sh) & 0xFFFFu) << 16);
            *(u32x2*)(dst + (cq * 8 + e) * LDT + 4 * rg) = o;
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

    if (nk > 0) load_tiles(0);
    for (int64_t kt = 0; kt < nk; ++kt) {
        __syncthreads();
        store_transposed(Dt, dr);
        store_transposed(Xt, xr);
        __syncthreads();
        if (kt + 1 < nk) load_tiles(kt + 1);
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            bf16x8 a[FM], b[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i)
                a[i] = *(const bf16x8*)(Dt + (wm * (BM / WM) + 32 * i + l32) * LDT + 16 * ks + 8 * h);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                b[j] = *(const bf16x8*)(Xt + (wn * (BN / WN) + 32 * j + l32) * LDT + 16 * ks + 8 * h);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = mfma_32x32x16(a[i], b[j], acc[i][j]);
        }
    }

    // ---- epilogue 1: mask in registers, round to bf16, keep in acc, and
    // write the bf16 G tile to LDS as [i][j].
    __syncthreads();
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int jl = wn * (BN / WN) + 32 * j + l32;
        const int gj = j0 + jl;
        const int wcol = gj >> 5;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int il = wm * (BM / WM) + 32 * i + 8 * (v >> 2) + 4 * h + (v & 3);
                const int gi = i0 + il;
                const uint32_t word = (gi < R && gj < C) ? Mp[(int64_t)gi * wpr + wcol] : 0u;
                const float g = keep1<TWO_FOUR>(word, (uint32_t)(gj & 31)) ? acc[i][j][v] : 0.f;
                const uint16_t gb = bf16_bits(g);
                acc[i][j][v] = bf16_bits_to_f32(gb);
                Gs[il * LDG + jl] = gb;
            }
        }
    }
    __syncthreads();

    // ---- epilogue 2: dB[i][j'] += s * sum_j G[i][j] A[j'][j]; wave w owns
    // rows i = 32w .. 32w+31 of the tile, all 32-wide rank blocks.
    {
        f32x16 db[JB];
#pragma unroll
        for (int b = 0; b < JB; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) db[b][v] = 0.f;
        const bool a_ok = true;
        (void)a_ok;
#pragma unroll 4
        for (int ks = 0; ks < BN / 16; ++ks) {
            const bf16x8 ga = *(const bf16x8*)(Gs + (wave * 32 + l32) * LDG + 16 * ks + 8 * h);
            const int gj = j0 + 16 * ks + 8 * h;
#pragma unroll
            for (int b = 0; b < JB; ++b) {
                const int jr = 32 * b + l32;  // rank index j'
                const u32x4 av = (jr < r && gj < C) ? *(const u32x4*)(Am + (int64_t)jr * C + gj)
                                                   : zero_u32x4();
                db[b] = mfma_32x32x16(ga, as_bf16x8(av), db[b]);
            }
        }
#pragma unroll
        for (int b = 0; b < JB; ++b) {
            const int jr = 32 * b + l32;
            if (jr >= r) continue;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int gi = i0 + wave * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
                if (gi < R) atomicAdd(dB + (int64_t)gi * r + jr, s * db[b][v]);
            }
        }
    }
    __syncthreads();

    // ---- epilogue 3: B^T of the tile's rows into LDS as [j'][i].
    for (int c = tid; c < BM * JB * 32; c += NT) {
        const int il = c / (JB * 32), jr = c % (JB * 32);
        const int gi = i0 + il;
        Bt[jr * LDB + il] = (gi < R && jr < r) ? Bm[(int64_t)gi * r + jr] : (uint16_t)0;
    }
    __syncthreads();

    // ---- epilogue 4: dA[j'][j] += s * sum_i B[i][j'] G[i][j], straight from
    // the masked accumulators.  For a 32-row block, MFMA K-chunk c uses
    // accumulator elements 8c .. 8c+7, i.e. rows 16c + 4h + {0..3} and
    // 16c + 8 + 4h + {0..3}; the B^T operand is read with the same row order.
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int gj = j0 + wn * (BN / WN) + 32 * j + l32;
#pragma unroll
        for (int b = 0; b < JB; ++b) {
            f32x16 da;
#pragma unroll
            for (int v = 0; v < 16; ++v) da[v] = 0.f;
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int ib = wm * (BM / WM) + 32 * i;
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    bf16x8 gb;
#pragma unroll
                    for (int e = 0; e < 8; ++e) gb[e] = (__bf16)acc[i][j][8 * c + e];
                    const uint16_t* bt = Bt + (32 * b + l32) * LDB + ib + 16 * c + 4 * h;
                    u32x4 bv;
                    const u32x2 lo = *(const u32x2*)(bt);
                    const u32x2 hi = *(const u32x2*)(bt + 8);
                    bv[0] = lo[0]; bv[1] = lo[1]; bv[2] = hi[0]; bv[3] = hi[1];
                    da = mfma_32x32x16(as_bf16x8(bv), gb, da);
                }
            }
            if (gj < C) {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int jr = 32 * b + 8 * (v >> 2) + 4 * h + (v & 3);
                    if (jr < r) atomicAdd(dA + (int64_t)jr * C + gj, s * da[v]);
                }
            }
        }
    }
}

template <int RK>
hipError_t launch_rk(const LayerArgs& a, hipStream_t st) {
    const int tiles_m = (int)((a.R + BM - 1) / BM);
    const int tiles_n = (int)((a.C + BN - 1) / BN);
    dim3 grid(tiles_m * tiles_n), block(NT);
    auto* dY = (const uint16_t*)a.dY;
    auto* X = (const uint16_t*)a.X;
    auto* B = (const uint16_t*)a.B;
    auto* A = (const uint16_t*)a.A;
    if (a.two_four)
        hipLaunchKernelGGL((g_kernel<RK, true>), grid, block, 0, st, dY, X, a.M, B, A, a.dB, a.dA,
                           a.L, (int)a.R, (int)a.C, (int)a.r, a.scale, tiles_m, tiles_n);
    else
        hipLaunchKernelGGL((g_kernel<RK, false>), grid, block, 0, st, dY, X, a.M, B, A, a.dB, a.dA,
                           a.L, (int)a.R, (int)a.C, (int)a.r, a.scale, tiles_m, tiles_n);
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
