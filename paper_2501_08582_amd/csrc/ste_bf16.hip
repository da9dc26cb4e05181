// Straight-through, re-associated adapter gradients, bf16 on gfx950.
//
//   P  = X . A^T      (L x r)        Q  = dY . B      (L x r)
//   dB = s . dY^T . P (R x r)        dA = s . Q^T . X (r x C)
//
// (Section 2.3 and Algorithm 2: the mask on the weight gradient is dropped,
// so the adapter gradients re-associate into products with the token
// dimension and the R x C weight gradient is never formed.)  Every product
// has one dimension of size r <= 128, so all four are bound by streaming X
// and dY from HBM, not by the matrix cores: X and dY are each read twice.
//
//   * rows_kernel: P and Q in one launch (grid y selects which).  A
//     workgroup owns 32 tokens; its four waves split the contraction over K
//     (C for P, R for Q) four ways and add their partial tiles through LDS.
//     Operand fragments come straight from global memory (both operands are
//     K-contiguous: X rows and A rows; dY rows and the rows of B^T, which
//     bt_kernel writes first).  P and Q are rounded to bf16.
//   * contract_kernel: out[i][j] += s . sum over tokens of U[l][i] V[l][j]
//     for dB (U = dY, V = P) and dA (U = X, V = Q, stored transposed).  A
//     workgroup owns 256 rows i and a slice of the tokens; both operands are
//     token-major and are staged through LDS and read back with transpose
//     loads.  Slices are combined with fp32 atomics, so outputs start at 0.
#include "gemm_common.hpp"
#include "kernels.hpp"

namespace lors {
namespace {

constexpr int NT = 256;

// bytes of P or Q in the workspace, rounded up to keep the next buffer aligned
inline int64_t ste_pq_bytes(int64_t L, int64_t r) { return (2 * L * r + 255) / 256 * 256; }

// B (R x r) -> B^T (r x R)
__global__ __launch_bounds__(NT) void bt_kernel(const uint16_t* __restrict__ B, uint16_t* __restrict__ BT,
                                                int64_t R, int r) {
    const int64_t t = (int64_t)blockIdx.x * NT + threadIdx.x;
    if (t < R * r) {
        const int64_t i = t / r, j = t % r;
        BT[j * R + i] = B[t];
    }
}

// out[L x r] (bf16) = U[L x K] . V[r x K]^T; grid.y = 0: (X, A) -> P, 1: (dY, B^T) -> Q
template <int RK32>
__global__ __launch_bounds__(NT) void rows_kernel(const uint16_t* __restrict__ X, const uint16_t* __restrict__ A,
                                                  const uint16_t* __restrict__ dY, const uint16_t* __restrict__ BT,
                                                  uint16_t* __restrict__ P, uint16_t* __restrict__ Q, int64_t L,
                                                  int R, int C, int r) {
    __shared__ __attribute__((aligned(16))) float red[4][RK32][16][64];
    const bool isq = blockIdx.y == 1;
    const uint16_t* U = isq ? dY : X;
    const uint16_t* V = isq ? BT : A;
    uint16_t* out = isq ? Q : P;
    const int K = isq ? R : C;
    const int lane = threadIdx.x & 63, l32 = lane & 31, h = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t row = (int64_t)blockIdx.x * 32 + l32;
    const bool rok = row < L;
    const uint16_t* urow = U + (rok ? row : 0) * (int64_t)K;
    f32x16 acc[RK32];
#pragma unroll
    for (int jb = 0; jb < RK32; ++jb)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[jb][v] = 0.f;
    const int nks = (K + 15) / 16;  // k-steps of 16; wave w takes steps w, w+4, ...
#pragma unroll 4
    for (int ks = wave; ks < nks; ks += 4) {
        const int k = 16 * ks + 8 * h;  // K % 8 == 0: a chunk is wholly in or out
        const bool kok = k < K;
        const u32x4 a = (rok && kok) ? *(const u32x4*)(urow + k) : zero_u32x4();
#pragma unroll
        for (int jb = 0; jb < RK32; ++jb) {
            const int j = 32 * jb + l32;
            const u32x4 b = (j < r && kok) ? *(const u32x4*)(V + (int64_t)j * K + k) : zero_u32x4();
            acc[jb] = mfma_32x32x16(as_bf16x8(a), as_bf16x8(b), acc[jb]);
        }
    }
#pragma unroll
    for (int jb = 0; jb < RK32; ++jb)
#pragma unroll
        for (int v = 0; v < 16; ++v) red[wave][jb][v][lane] = acc[jb][v];
    __syncthreads();
    if (wave == 0) {
#pragma unroll
        for (int jb = 0; jb < RK32; ++jb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const float sum = red[0][jb][v][lane] + red[1][jb][v][lane] + red[2][jb][v][lane] + red[3][jb][v][lane];
                // accumulator element v: token row 8(v/4) + 4h + v%4, rank column l32
                const int64_t tr = (int64_t)blockIdx.x * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
                const int j = 32 * jb + l32;
                if (tr < L && j < r) out[tr * r + j] = bf16_bits(sum);
            }
    }
}

// out (fp32, atomics) += s . U^T V over tokens [t0, t1):
//   U: L x BIG token-major, V: L x r token-major (bf16)
//   TRANS_OUT = false: out[i * r + j] (dB, R x r); true: out[j * BIG + i] (dA, r x C)
constexpr int CK = 32;                    // tokens per stage
constexpr int UB = CK * kRowBytes;        // U slab [32 tokens][256 i]: 16 KiB

template <int RK32, bool TRANS_OUT>
__global__ __launch_bounds__(NT) void contract_kernel(const uint16_t* __restrict__ U, const uint16_t* __restrict__ V,
                                                      float* __restrict__ out, int64_t L, int BIG, int r, float s,
                                                      int64_t tok_per_split) {
    constexpr int RP = 32 * RK32;         // padded rank
    constexpr int VB = CK * RP * 2;       // V slab [32 tokens][RP]
    __shared__ __attribute__((aligned(1024))) uint8_t smem[UB + VB];
    const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, h = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int i0 = blockIdx.x * 256;
    const int64_t t0 = (int64_t)blockIdx.y * tok_per_split;
    const int64_t t1 = (t0 + tok_per_split < L) ? t0 + tok_per_split : L;
    const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
    const uint8_t* zsrc = (const uint8_t*)g_zero_page + 16 * lane;
    f32x16 acc[2][RK32];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int jb = 0; jb < RK32; ++jb)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[a][jb][v] = 0.f;
    // transpose-read offsets: U slab rows = tokens (512 B rows, swizzled), V slab rows of RP bf16
    int offU[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int t = 0; t < 2; ++t) offU[a][t] = tr_frag_off(lane, 0, 64 * wave + 32 * a, t);
    int offV[RK32][2];
    {
        const int g = lane >> 4, jj = lane & 15;
#pragma unroll
        for (int jb = 0; jb < RK32; ++jb)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const int row = 8 * (g >> 1) + 4 * t + (jj >> 2);
                const int col = 32 * jb + 16 * (g & 1) + 4 * (jj & 3);
                offV[jb][t] = UB + (row * RP + col) * 2;
            }
    }
    for (int64_t tc = t0; tc < t1; tc += CK) {
        // U slab: 32 token rows x 256 i (copy q of this wave fills rows 2(4 wave + q) + h)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int blk = 4 * wave + q, row = 2 * blk + h;
            const int lc = swz_chunk(row, lane & 31);
            const int64_t gl = tc + row;
            const int gi = i0 + 8 * lc;
            copy16_to_lds((gl < t1 && gi < BIG) ? (const void*)(U + gl * BIG + gi) : (const void*)zsrc,
                          lds0 + 1024 * blk);
        }
        // V slab: 32 token rows x RP ranks, ranks >= r zero (16-byte chunks via registers)
        for (int e = tid; e < CK * RP / 8; e += NT) {
            const int row = e / (RP / 8), ch = e % (RP / 8);
            const int64_t gl = tc + row;
            u32x4 v = zero_u32x4();
            if (gl < t1 && 8 * ch < r) {
                const uint16_t* src = V + gl * r + 8 * ch;
                if ((r & 7) == 0) {
                    v = *(const u32x4*)src;
                } else {
#pragma unroll
                    for (int q = 0; q < 8; ++q)
                        v[q >> 1] |= (8 * ch + q < r ? (uint32_t)src[q] : 0u) << ((q & 1) * 16);
                }
            }
            *(u32x4*)(smem + UB + (row * RP + 8 * ch) * 2) = v;
        }
        stage_barrier<0>();
#pragma unroll
        for (int kc = 0; kc < CK / 16; ++kc) {
            const int ro = 16 * kc;
            bf16x8 fu[2], fv[RK32];
#pragma unroll
            for (int a = 0; a < 2; ++a)
                fu[a] = frag_from_tr(lds_tr_read(smem + ro * kRowBytes + offU[a][0]),
                                     lds_tr_read(smem + ro * kRowBytes + offU[a][1]));
#pragma unroll
            for (int jb = 0; jb < RK32; ++jb)
                fv[jb] = frag_from_tr(lds_tr_read(smem + offV[jb][0] + ro * RP * 2),
                                      lds_tr_read(smem + offV[jb][1] + ro * RP * 2));
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int jb = 0; jb < RK32; ++jb) acc[a][jb] = mfma_32x32x16(fu[a], fv[jb], acc[a][jb]);
        }
        lds_barrier();
    }
    // accumulator element v of block (a, jb): row i = 64 wave + 32 a + 8(v/4) + 4h + v%4, column j = 32 jb + l32
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int jb = 0; jb < RK32; ++jb) {
            const int j = 32 * jb + l32;
            if (j >= r) continue;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int i = i0 + 64 * wave + 32 * a + 8 * (v >> 2) + 4 * h + (v & 3);
                if (i < BIG) atomicAdd(out + (TRANS_OUT ? (int64_t)j * BIG + i : (int64_t)i * r + j), s * acc[a][jb][v]);
            }
        }
}

template <int RK32>
hipError_t launch_rk(const LayerArgs& a, hipStream_t st) {
    auto* X = (const uint16_t*)a.X;
    auto* dY = (const uint16_t*)a.dY;
    auto* B = (const uint16_t*)a.B;
    auto* A = (const uint16_t*)a.A;
    const int64_t pq = ste_pq_bytes(a.L, a.r);
    uint16_t* P = (uint16_t*)a.ste_ws;
    uint16_t* Q = (uint16_t*)((uint8_t*)a.ste_ws + pq);
    uint16_t* BT = (uint16_t*)((uint8_t*)a.ste_ws + 2 * pq);
    const int64_t nb = a.R * a.r;
    hipLaunchKernelGGL(bt_kernel, dim3((unsigned)((nb + NT - 1) / NT)), dim3(NT), 0, st, B, BT, a.R, (int)a.r);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((rows_kernel<RK32>), dim3((unsigned)((a.L + 31) / 32), 2), dim3(NT), 0, st, X, A, dY, BT, P, Q,
                       a.L, (int)a.R, (int)a.C, (int)a.r);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // token slices: enough workgroups for the whole chip (about 512 over both
    // products), at least 64 tokens each
    const int64_t rb = (a.R + 255) / 256, cb = (a.C + 255) / 256;
    int64_t splits = (512 + rb + cb - 1) / (rb + cb);
    const int64_t max_splits = (a.L + 63) / 64;
    if (splits > max_splits) splits = max_splits;
    if (splits > 65535) splits = 65535;
    const int64_t per = ((a.L + splits - 1) / splits + CK - 1) / CK * CK;
    splits = (a.L + per - 1) / per;
    hipLaunchKernelGGL((contract_kernel<RK32, false>), dim3((unsigned)rb, (unsigned)splits), dim3(NT), 0, st, dY, P,
                       a.dB, a.L, (int)a.R, (int)a.r, a.scale, per);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((contract_kernel<RK32, true>), dim3((unsigned)cb, (unsigned)splits), dim3(NT), 0, st, X, Q,
                       a.dA, a.L, (int)a.C, (int)a.r, a.scale, per);
    return hipGetLastError();
}

}  // namespace

size_t ste_workspace_bytes(int64_t R, int64_t L, int64_t r) {
    // P, Q (L x r) and B^T (r x R), bf16, each 256-byte aligned
    return static_cast<size_t>(2 * ste_pq_bytes(L, r) + (2 * r * R + 255) / 256 * 256);
}

hipError_t launch_ste_bf16(const LayerArgs& a, hipStream_t st) {
    if (a.L == 0) return hipSuccess;  // dB, dA stay zero
    switch ((a.r + 31) / 32) {
        case 1: return launch_rk<1>(a, st);
        case 2: return launch_rk<2>(a, st);
        case 3: return launch_rk<3>(a, st);
        case 4: return launch_rk<4>(a, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace lors
