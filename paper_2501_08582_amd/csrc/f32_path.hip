// fp32 kernels of the sparsity-preserved LoRA linear (debug/reference dtype).
//
// Same fused structure as the bf16 path -- W' is rebuilt tile by tile in LDS
// and G never leaves the workgroup -- but every product runs on the fp32 VALU
// with fp32 accumulation, no reduced-precision matrix mode.  Tiles are 64x64
// with 256 threads, each thread owning a 4x4 block of outputs.
#include "device_common.hpp"
#include "kernels.hpp"

namespace lors {
namespace {

constexpr int T = 64;   // tile edge
constexpr int KS = 16;  // K-step
constexpr int NT = 256;
constexpr int RMAX = 128;

// keep-bit of element (row, col) of the packed mask
template <bool TWO_FOUR>
__device__ __forceinline__ bool kept(const uint32_t* Mp, int wpr, int row, int col) {
    const uint32_t w = Mp[(int64_t)row * wpr + (col >> 5)];
    return keep1<TWO_FOUR>(w, (uint32_t)(col & 31)) != 0u;
}

// Y[L x R] = X . W'^T (+bias); GEMM M = L, N = R, K = C.
template <bool TWO_FOUR>
__global__ __launch_bounds__(NT) void fwd_f32(const float* __restrict__ X, const float* __restrict__ W,
                                              const uint32_t* __restrict__ Mp,
                                              const float* __restrict__ Bm,
                                              const float* __restrict__ Am,
                                              const float* __restrict__ bias, float* __restrict__ Y,
                                              int64_t L, int R, int C, int r, float s) {
    __shared__ float Xs[KS][T + 1];   // [k][m]
    __shared__ float Ws[KS][T + 1];   // [k][n] merged
    __shared__ float Bs[T][RMAX + 1]; // B rows of the tile
    const int tid = threadIdx.x;
    const int64_t m0 = (int64_t)blockIdx.y * T;
    const int n0 = blockIdx.x * T;
    const int wpr = (C + 31) >> 5;
    for (int c = tid; c < T * r; c += NT) {
        const int n = c / r, j = c % r;
        Bs[n][j] = (n0 + n < R) ? Bm[(int64_t)(n0 + n) * r + j] : 0.f;
    }
    float acc[4][4] = {};
    const int tx = tid % 16, ty = tid / 16;
    for (int k0 = 0; k0 < C; k0 += KS) {
        __syncthreads();
        for (int c = tid; c < T * KS; c += NT) {
            const int row = c / KS, k = c % KS;
            const int64_t gm = m0 + row;
            const int gk = k0 + k;
            Xs[k][row] = (gm < L && gk < C) ? X[gm * C + gk] : 0.f;
            const int gn = n0 + row;
            float w = 0.f;
            if (gn < R && gk < C && kept<TWO_FOUR>(Mp, wpr, gn, gk)) {
                float t = 0.f;
                for (int j = 0; j < r; ++j) t = fmaf(Bs[row][j], Am[(int64_t)j * C + gk], t);
                w = fmaf(s, t, W[(int64_t)gn * C + gk]);
            }
            Ws[k][row] = w;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < KS; ++k) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = Xs[k][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Ws[k][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t gm = m0 + ty * 4 + i;
        if (gm >= L) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int gn = n0 + tx * 4 + j;
            if (gn < R) Y[gm * R + gn] = acc[i][j] + (bias ? bias[gn] : 0.f);
        }
    }
}

// dX[L x C] = dY . W'; GEMM M = L, N = C, K = R.
template <bool TWO_FOUR>
__global__ __launch_bounds__(NT) void dx_f32(const float* __restrict__ dY, const float* __restrict__ W,
                                             const uint32_t* __restrict__ Mp,
                                             const float* __restrict__ Bm,
                                             const float* __restrict__ Am, float* __restrict__ dX,
                                             int64_t L, int R, int C, int r, float s) {
    __shared__ float Ds[KS][T + 1];    // [k][m]
    __shared__ float Ws[KS][T + 1];    // [k][n] merged
    __shared__ float As[RMAX][T + 1];  // A columns of the tile
    const int tid = threadIdx.x;
    const int64_t m0 = (int64_t)blockIdx.y * T;
    const int n0 = blockIdx.x * T;
    const int wpr = (C + 31) >> 5;
    for (int c = tid; c < T * r; c += NT) {
        const int j = c / T, n = c % T;
        As[j][n] = (n0 + n < C) ? Am[(int64_t)j * C + n0 + n] : 0.f;
    }
    float acc[4][4] = {};
    const int tx = tid % 16, ty = tid / 16;
    for (int k0 = 0; k0 < R; k0 += KS) {
        __syncthreads();
        for (int c = tid; c < T * KS; c += NT) {
            {
                const int row = c / KS, k = c % KS;
                const int64_t gm = m0 + row;
                const int gk = k0 + k;
                Ds[k][row] = (gm < L && gk < R) ? dY[gm * R + gk] : 0.f;
            }
            {
                const int k = c / T, n = c % T;
                const int gk = k0 + k, gn = n0 + n;
                float w = 0.f;
                if (gk < R && gn < C && kept<TWO_FOUR>(Mp, wpr, gk, gn)) {
                    float t = 0.f;
                    for (int j = 0; j < r; ++j) t = fmaf(Bm[(int64_t)gk * r + j], As[j][n], t);
                    w = fmaf(s, t, W[(int64_t)gk * C + gn]);
                }
                Ws[k][n] = w;
            }
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < KS; ++k) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = Ds[k][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Ws[k][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t gm = m0 + ty * 4 + i;
        if (gm >= L) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int gn = n0 + tx * 4 + j;
            if (gn < C) dX[gm * C + gn] = acc[i][j];
        }
    }
}

// G tile = select(M, dY^T X, 0) over K = L, then fp32 atomics of the tile's
// contributions to dB = s G A^T and dA = s B^T G.
template <bool TWO_FOUR>
__global__ __launch_bounds__(NT) void g_f32(const float* __restrict__ dY, const float* __restrict__ X,
                                            const uint32_t* __restrict__ Mp,
                                            const float* __restrict__ Bm,
                                            const float* __restrict__ Am, float* __restrict__ dB,
                                            float* __restrict__ dA, int64_t L, int R, int C, int r,
                                            float s) {
    __shared__ float Ds[KS][T + 1];  // [l][i]
    __shared__ float Xs[KS][T + 1];  // [l][j]
    __shared__ float Gs[T][T + 1];   // [i][j]
    const int tid = threadIdx.x;
    const int i0 = blockIdx.y * T;
    const int j0 = blockIdx.x * T;
    const int wpr = (C + 31) >> 5;
    float acc[4][4] = {};
    const int tx = tid % 16, ty = tid / 16;
    for (int64_t l0 = 0; l0 < L; l0 += KS) {
        __syncthreads();
        for (int c = tid; c < T * KS; c += NT) {
            const int k = c / T, col = c % T;
            const int64_t gl = l0 + k;
            Ds[k][col] = (gl < L && i0 + col < R) ? dY[gl * R + i0 + col] : 0.f;
            Xs[k][col] = (gl < L && j0 + col < C) ? X[gl * C + j0 + col] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < KS; ++k) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = Ds[k][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Xs[k][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int gi = i0 + ty * 4 + i, gj = j0 + tx * 4 + j;
            const bool k = gi < R && gj < C && kept<TWO_FOUR>(Mp, wpr, gi, gj);
            Gs[ty * 4 + i][tx * 4 + j] = k ? acc[i][j] : 0.f;
        }
    __syncthreads();
    for (int c = tid; c < T * r; c += NT) {
        const int il = c / r, jr = c % r;
        if (i0 + il >= R) continue;
        float t = 0.f;
        for (int jl = 0; jl < T && j0 + jl < C; ++jl) t = fmaf(Gs[il][jl], Am[(int64_t)jr * C + j0 + jl], t);
        atomicAdd(dB + (int64_t)(i0 + il) * r + jr, s * t);
    }
    for (int c = tid; c < T * r; c += NT) {
        const int jr = c / T, jl = c % T;
        if (j0 + jl >= C) continue;
        float t = 0.f;
        for (int il = 0; il < T && i0 + il < R; ++il) t = fmaf(Bm[(int64_t)(i0 + il) * r + jr], Gs[il][jl], t);
        atomicAdd(dA + (int64_t)jr * C + j0 + jl, s * t);
    }
}

}  // namespace

hipError_t launch_fwd_f32(const LayerArgs& a, hipStream_t st) {
    if (a.L == 0) return hipSuccess;
    dim3 grid((unsigned)((a.R + T - 1) / T), (unsigned)((a.L + T - 1) / T)), block(NT);
    if (a.two_four)
        hipLaunchKernelGGL(fwd_f32<true>, grid, block, 0, st, (const float*)a.X, (const float*)a.W, a.M,
                           (const float*)a.B, (const float*)a.A, (const float*)a.bias, (float*)a.Y,
                           a.L, (int)a.R, (int)a.C, (int)a.r, a.scale);
    else
        hipLaunchKernelGGL(fwd_f32<false>, grid, block, 0, st, (const float*)a.X, (const float*)a.W, a.M,
                           (const float*)a.B, (const float*)a.A, (const float*)a.bias, (float*)a.Y,
                           a.L, (int)a.R, (int)a.C, (int)a.r, a.scale);
    return hipGetLastError();
}

hipError_t launch_dx_f32(const LayerArgs& a, hipStream_t st) {
    if (a.L == 0 || a.dX == nullptr) return hipSuccess;
    dim3 grid((unsigned)((a.C + T - 1) / T), (unsigned)((a.L + T - 1) / T)), block(NT);
    if (a.two_four)
        hipLaunchKernelGGL(dx_f32<true>, grid, block, 0, st, (const float*)a.dY, (const float*)a.W, a.M,
                           (const float*)a.B, (const float*)a.A, (float*)a.dX, a.L, (int)a.R,
                           (int)a.C, (int)a.r, a.scale);
    else
        hipLaunchKernelGGL(dx_f32<false>, grid, block, 0, st, (const float*)a.dY, (const float*)a.W, a.M,
                           (const float*)a.B, (const float*)a.A, (float*)a.dX, a.L, (int)a.R,
                           (int)a.C, (int)a.r, a.scale);
    return hipGetLastError();
}

hipError_t launch_g_f32(const LayerArgs& a, hipStream_t st) {
    if (a.L == 0) return hipSuccess;
    dim3 grid((unsigned)((a.C + T - 1) / T), (unsigned)((a.R + T - 1) / T)), block(NT);
    if (a.two_four)
        hipLaunchKernelGGL(g_f32<true>, grid, block, 0, st, (const float*)a.dY, (const float*)a.X, a.M,
                           (const float*)a.B, (const float*)a.A, a.dB, a.dA, a.L, (int)a.R,
                           (int)a.C, (int)a.r, a.scale);
    else
        hipLaunchKernelGGL(g_f32<false>, grid, block, 0, st, (const float*)a.dY, (const float*)a.X, a.M,
                           (const float*)a.B, (const float*)a.A, a.dB, a.dA, a.L, (int)a.R,
                           (int)a.C, (int)a.r, a.scale);
    return hipGetLastError();
}

}  // namespace lors
