// Straight-through, re-associated adapter gradients, bf16 on gfx950.
//
//   P  = X . A^T      (L x r)        Q  = dY . B      (L x r)
//   dB = s . dY^T . P (R x r)        dA = s . Q^T . X (r x C)
//
// (Section 2.3 and Algorithm 2: the mask on the weight gradient is dropped,
// so the adapter gradients re-associate into products with the token
// dimension and the R x C weight gradient is never formed.)  Every product
// has one dimension of size r <= 128, so all four are bound by streaming X
// and dY from HBM, not by the matrix cores: X and dY are each read twice,
// and the three launches below are built to keep HBM busy.
//
//   * prep_kernel: B^T (so that Q's second operand is K-contiguous like A)
//     and the zeroing of dB and dA, which the contraction accumulates into.
//   * rows_kernel / rows_staged_kernel: P and Q in one launch (grid y
//     selects which).  A workgroup owns 32 tokens and its four waves add
//     their partial tiles through LDS.  rows_kernel: the waves split the
//     contraction over K (C for P, R for Q) into four contiguous ranges, and
//     operands go from global memory into registers in double-buffered
//     batches, the token rows in whole cache lines re-laid through LDS into
//     the MFMA layout; its adapter-side loads touch 32 rows per instruction,
//     which is cheap for one 32-rank block and limits it beyond that.
//     rows_staged_kernel: both operands stream through a ring of LDS stages
//     (128 k of every row per stage, asynchronous copies of whole 256-byte
//     row segments, one barrier per stage) and the waves split each stage's
//     k range; it is taken for ranks above 32 when a row is at least 8192
//     long, where it measured 1.4x to 1.8x faster (at 4096-long rows the
//     register form still led).  P and Q are rounded to bf16 and stored
//     with the rank padded to a multiple of 32 (pad columns zero), which
//     makes every token row of them 64-byte aligned for the contraction's
//     LDS copies.
//   * contract_kernel: out[i][j] += s . sum over tokens of U[l][i] V[l][j],
//     dB tiles (U = dY, V = P) and dA tiles (U = X, V = Q) in one grid.  A
//     workgroup owns 256 rows i and a slice of the tokens; both operands are
//     token-major and go through an NS-deep ring of LDS stages (32 tokens
//     each, asynchronous global -> LDS copies, one barrier per stage) and
//     are read back with transpose loads.  For dA the MFMA operands are
//     swapped so that the 32 lanes of an accumulator row hold 32 consecutive
//     columns of the r x C output: every fp32 atomic instruction then covers
//     whole cache lines.  Token slices are combined with those atomics.
#include "gemm_common.hpp"
#include "kernels.hpp"

namespace lors {
namespace {

constexpr int NT = 256;

// rank padded to the MFMA column block
inline int64_t rank_pad(int64_t r) { return (r + 31) / 32 * 32; }

// bytes of P or Q (L x rank_pad(r) bf16) in the workspace, rounded up to
// keep the next buffer aligned
inline int64_t ste_pq_bytes(int64_t L, int64_t r) { return (2 * L * rank_pad(r) + 255) / 256 * 256; }

// ---------------------------------------------------------------------------
// B (R x r) -> B^T (r x R) through an LDS tile of 64 rows, then dB and dA
// set to zero (grid-stride over every workgroup).
// ---------------------------------------------------------------------------
constexpr int BT_ROWS = 64;
constexpr int BT_STRIDE = 129;  // odd: the column reads spread over the banks

__global__ __launch_bounds__(NT) void prep_kernel(const uint16_t* __restrict__ B, uint16_t* __restrict__ BT,
                                                  float* __restrict__ dB, float* __restrict__ dA, int64_t R, int r,
                                                  int64_t nB, int64_t nA) {
    __shared__ uint16_t t[BT_ROWS * BT_STRIDE];
    const int tid = threadIdx.x;
    const int64_t i0 = (int64_t)blockIdx.x * BT_ROWS;
    if (i0 < R) {  // uniform over the workgroup
        const int rows = (int)(R - i0 < BT_ROWS ? R - i0 : BT_ROWS);
        const uint16_t* src = B + i0 * r;
        for (int e = tid; e < rows * r; e += NT) t[(e / r) * BT_STRIDE + e % r] = src[e];
        __syncthreads();
        for (int e = tid; e < r * BT_ROWS; e += NT) {
            const int j = e / BT_ROWS, i = e % BT_ROWS;
            if (i < rows) BT[(int64_t)j * R + i0 + i] = t[i * BT_STRIDE + j];
        }
    }
    const int64_t g0 = (int64_t)blockIdx.x * NT + tid, gs = (int64_t)gridDim.x * NT;
    for (int64_t e = g0; e < nB; e += gs) dB[e] = 0.f;
    for (int64_t e = g0; e < nA; e += gs) dA[e] = 0.f;
}

// ---------------------------------------------------------------------------
// out[L x RP] (bf16) = U[L x K] . V[r x K]^T;
// grid.y = 0: (X, A) -> P with K = C; 1: (dY, B^T) -> Q with K = R.
//
// Each wave walks its K range in blocks of 64 k.  The U block (32 token rows
// x 128 bytes) is read in whole 128-byte lines (8 lanes per row, 8 rows per
// load) and re-laid through a wave-private LDS buffer into the MFMA operand
// layout (row l32, k 8h .. 8h+7 of each 16-k step), so that every HBM
// request covers a full line; the V rows are L2-resident and are read in the
// operand layout directly.
// ---------------------------------------------------------------------------
template <int RK32>
struct RowsCfg {
    static constexpr int NB = RK32 == 1 ? 2 : 1;  // 64-k blocks per register batch
};

template <int RK32>
__global__ __launch_bounds__(NT) void rows_kernel(const uint16_t* __restrict__ X, const uint16_t* __restrict__ A,
                                                  const uint16_t* __restrict__ dY, const uint16_t* __restrict__ BT,
                                                  uint16_t* __restrict__ P, uint16_t* __restrict__ Q, int64_t L,
                                                  int R, int C, int r) {
    constexpr int RP = 32 * RK32;
    constexpr int NB = RowsCfg<RK32>::NB;
    __shared__ __attribute__((aligned(16))) float red[4][RK32][16][64];
    __shared__ __attribute__((aligned(1024))) uint8_t stg[4][NB][32 * kRow64];
    const bool isq = blockIdx.y == 1;
    const uint16_t* U = isq ? dY : X;
    const uint16_t* V = isq ? BT : A;
    uint16_t* out = isq ? Q : P;
    const int K = isq ? R : C;
    const int lane = threadIdx.x & 63, l32 = lane & 31, h = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // Rows past L and ranks past r read valid rows (their results are not
    // kept); chunks past this wave's range or past K read the zero page.
    // Line load i (0..3) of a block covers rows 8i + lane/8, chunk lane%8.
    const int crow = lane >> 3, cch = lane & 7;
    const uint16_t* ubase[4];
    int woff[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t row = (int64_t)blockIdx.x * 32 + 8 * i + crow;
        ubase[i] = U + (row < L ? row : L - 1) * (int64_t)K + 8 * cch;
        woff[i] = slab64_off(8 * i + crow, cch);
    }
    int roff[4];  // operand of 16-k step q: row l32, chunk 2q + h
#pragma unroll
    for (int q = 0; q < 4; ++q) roff[q] = slab64_off(l32, 2 * q + h);
    const uint16_t* vrow[RK32];
#pragma unroll
    for (int jb = 0; jb < RK32; ++jb) {
        const int j = 32 * jb + l32;
        vrow[jb] = V + (int64_t)(j < r ? j : r - 1) * K + 8 * h;
    }
    const uint16_t* zp = (const uint16_t*)g_zero_page + 8 * lane;
    const int nkb = (K + 63) / 64;  // wave w takes a contiguous quarter of the blocks
    const int per = (nkb + 3) / 4;
    const int b0 = wave * per;
    const int b1 = b0 + per < nkb ? b0 + per : nkb;
    f32x16 acc[RK32];
#pragma unroll
    for (int jb = 0; jb < RK32; ++jb)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[jb][v] = 0.f;

    u32x4 ua[NB][4], ub[NB][4], va[NB][4][RK32], vb[NB][4][RK32];
    auto load = [&](u32x4(&u)[NB][4], u32x4(&v)[NB][4][RK32], int b) {
#pragma unroll
        for (int n = 0; n < NB; ++n) {
            const int k0 = 64 * (b + n);
            const bool blk = b + n < b1;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const bool ok = blk && k0 + 8 * cch < K;  // K % 8 == 0: a chunk is wholly in or out
                u[n][i] = *(const u32x4*)(ok ? ubase[i] + k0 : zp);
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int k = k0 + 16 * q;
                const bool ok = blk && k + 8 * h < K;
#pragma unroll
                for (int jb = 0; jb < RK32; ++jb) v[n][q][jb] = *(const u32x4*)(ok ? vrow[jb] + k : zp);
            }
        }
    };
    auto mul = [&](const u32x4(&u)[NB][4], const u32x4(&v)[NB][4][RK32]) {
#pragma unroll
        for (int n = 0; n < NB; ++n) {
            uint8_t* sb = &stg[wave][n][0];
#pragma unroll
            for (int i = 0; i < 4; ++i) *(u32x4*)(sb + woff[i]) = u[n][i];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const u32x4 a = *(const u32x4*)(sb + roff[q]);
#pragma unroll
                for (int jb = 0; jb < RK32; ++jb)
                    acc[jb] = mfma_32x32x16(as_bf16x8(a), as_bf16x8(v[n][q][jb]), acc[jb]);
            }
        }
    };
    load(ua, va, b0);
    for (int b = b0; b < b1; b += 2 * NB) {
        load(ub, vb, b + NB);
        mul(ua, va);
        load(ua, va, b + 2 * NB);
        mul(ub, vb);
    }
#pragma unroll
    for (int jb = 0; jb < RK32; ++jb)
#pragma unroll
        for (int v = 0; v < 16; ++v) red[wave][jb][v][lane] = acc[jb][v];
    __syncthreads();
    // Wave w adds up accumulator elements 4w .. 4w+3: token row
    // 8(v/4) + 4h + v%4 = 8w + 4h + q, rank column 32 jb + l32.
    const int64_t tr0 = (int64_t)blockIdx.x * 32 + 8 * wave + 4 * h;
#pragma unroll
    for (int jb = 0; jb < RK32; ++jb) {
        const int j = 32 * jb + l32;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int v = 4 * wave + q;
            const float sum = red[0][jb][v][lane] + red[1][jb][v][lane] + red[2][jb][v][lane] + red[3][jb][v][lane];
            if (tr0 + q < L) out[(tr0 + q) * RP + j] = j < r ? bf16_bits(sum) : (uint16_t)0;
        }
    }
}

// ---------------------------------------------------------------------------
// P and Q through a ring of LDS stages.  Stage: U [32 tokens][KS] and
// V [RP][KS] (KS = 128 k, 256-byte row segments); the 16-byte chunk c of
// segment row q is stored at chunk c ^ (q & 15), so the MFMA-layout reads
// (32 rows, one chunk each) fall on distinct banks.  Each 1 KiB copy fills
// four segment rows; the waves take equal shares of the copies and a
// quarter of each stage's k range.
// ---------------------------------------------------------------------------
constexpr int SK = 128;                  // k per stage
constexpr int SROW = 2 * SK;             // bytes per staged row
constexpr int SCH = SROW / 16;           // chunks per staged row
constexpr int SRPC = 1024 / SROW;        // staged rows per copy
constexpr int SUB = 32 * SROW;           // U stage bytes

template <int RK32>
struct StagedCfg {
    static constexpr int RP = 32 * RK32;
    static constexpr int VB = RP * SROW;                 // V stage bytes
    static constexpr int SB = SUB + VB;                  // one stage
    static constexpr int NS = 131072 / SB < 6 ? 131072 / SB : 6;  // ring depth within 128 KiB
    static constexpr int UC = SUB / 4096, VC = VB / 4096;  // copies per wave per stage
    static constexpr int CPS = UC + VC;
    static_assert(SUB % 4096 == 0 && VB % 4096 == 0, "copies split evenly over the four waves");
    static_assert(NS >= 3 && RK32 * 16384 <= NS * SB, "ring depth; the reduction reuses the ring");
};

template <int RK32>
__global__ __launch_bounds__(NT) void rows_staged_kernel(const uint16_t* __restrict__ X,
                                                         const uint16_t* __restrict__ A,
                                                         const uint16_t* __restrict__ dY,
                                                         const uint16_t* __restrict__ BT, uint16_t* __restrict__ P,
                                                         uint16_t* __restrict__ Q, int64_t L, int R, int C, int r) {
    using Cfg = StagedCfg<RK32>;
    constexpr int RP = Cfg::RP, NS = Cfg::NS, SB = Cfg::SB, UC = Cfg::UC, VC = Cfg::VC;
    __shared__ __attribute__((aligned(1024))) uint8_t smem[NS * SB];
    const bool isq = blockIdx.y == 1;
    const uint16_t* U = isq ? dY : X;
    const uint16_t* V = isq ? BT : A;
    uint16_t* out = isq ? Q : P;
    const int K = isq ? R : C;
    const int lane = threadIdx.x & 63, l32 = lane & 31, h = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t t0 = (int64_t)blockIdx.x * 32;
    const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
    const void* zsrc = (const uint8_t*)g_zero_page + 16 * lane;
    const int nst = (K + SK - 1) / SK;
    // Lane of a copy: staged row lane / SCH of the copy's SRPC rows, stored
    // chunk lane % SCH, which holds logical chunk (lane % SCH) ^ (row & 15).
    // Rows past L or r and chunks past K (K % 8 == 0) read the zero page.
    const int crow = lane / SCH, pch = lane % SCH;
    auto issue = [&](int st) {
        const int k0 = (st < nst ? st : nst - 1) * SK;  // past the end: repeat the last stage (never read)
        const uint32_t base = lds0 + (uint32_t)((st % NS) * SB);
#pragma unroll
        for (int q = 0; q < UC; ++q) {
            const int blk = UC * wave + q, row = SRPC * blk + crow;
            const int k = k0 + 8 * (pch ^ (row & 15));
            const bool ok = t0 + row < L && k < K;
            copy16_to_lds(ok ? (const void*)(U + (t0 + row) * K + k) : zsrc, base + 1024 * blk);
        }
#pragma unroll
        for (int q = 0; q < VC; ++q) {
            const int blk = VC * wave + q, row = SRPC * blk + crow;
            const int k = k0 + 8 * (pch ^ (row & 15));
            const bool ok = row < r && k < K;
            copy16_to_lds(ok ? (const void*)(V + (int64_t)row * K + k) : zsrc, base + SUB + 1024 * blk);
        }
    };
    f32x16 acc[RK32];
#pragma unroll
    for (int jb = 0; jb < RK32; ++jb)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[jb][v] = 0.f;
#pragma unroll
    for (int st = 0; st < NS - 1; ++st) issue(st);
    for (int st = 0; st < nst; ++st) {
        stage_barrier<(NS - 2) * Cfg::CPS>();  // stage st landed; stage st - 1 is no longer read
        issue(st + NS - 1);
        const uint8_t* sb = smem + (st % NS) * SB;
#pragma unroll
        for (int ks = 0; ks < SK / 64; ++ks) {  // this wave's quarter: 16-k steps of 32 k
            const int c = (SK / 4 * wave + 16 * ks) / 8 + h;  // logical chunk of this lane
            const bf16x8 a = *(const bf16x8*)(sb + l32 * SROW + ((c ^ (l32 & 15)) << 4));
#pragma unroll
            for (int jb = 0; jb < RK32; ++jb) {
                const int j = 32 * jb + l32;
                const bf16x8 b = *(const bf16x8*)(sb + SUB + j * SROW + ((c ^ (j & 15)) << 4));
                acc[jb] = mfma_32x32x16(a, b, acc[jb]);
            }
        }
    }
    wait_vmcnt<0>();  // the repeated tail stages still land in the ring
    lds_barrier();
    float* red = (float*)smem;  // [4 waves][RK32][16][64]
#pragma unroll
    for (int jb = 0; jb < RK32; ++jb)
#pragma unroll
        for (int v = 0; v < 16; ++v) red[((wave * RK32 + jb) * 16 + v) * 64 + lane] = acc[jb][v];
    __syncthreads();
    // as in rows_kernel: wave w adds up accumulator elements 4w .. 4w+3
    const int64_t tr0 = t0 + 8 * wave + 4 * h;
#pragma unroll
    for (int jb = 0; jb < RK32; ++jb) {
        const int j = 32 * jb + l32;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int v = 4 * wave + q;
            float sum = 0.f;
#pragma unroll
            for (int w = 0; w < 4; ++w) sum += red[((w * RK32 + jb) * 16 + v) * 64 + lane];
            if (tr0 + q < L) out[(tr0 + q) * RP + j] = j < r ? bf16_bits(sum) : (uint16_t)0;
        }
    }
}

// Row length from which the staged form is taken for ranks above 32.
constexpr int64_t kStagedMinK = 8192;

// ---------------------------------------------------------------------------
// out (fp32, atomics) += s . U^T V over the tokens [t0, t1) of grid.y's slice.
//   U: L x BIG token-major bf16, V: L x RP token-major bf16
//   TRANS_OUT = false: out[i * r + j] (dB, R x r); true: out[j * BIG + i] (dA, r x C)
// ---------------------------------------------------------------------------
constexpr int CK = 32;              // tokens per stage
constexpr int UB = CK * kRowBytes;  // U stage [32 tokens][256 i]: 16 KiB
constexpr int SINK = 1024;          // destination of the padding copies

template <int RK32>
struct ContractCfg {
    static constexpr int RP = 32 * RK32;
    static constexpr int VB = CK * RP * 2;        // V stage [32 tokens][RP]
    static constexpr int SB = UB + VB;            // one stage
    static constexpr int NS = RK32 == 1 ? 4 : 3;  // ring depth: two workgroups per CU fit in LDS
    static constexpr int VCOPIES = VB / 1024;     // 16-byte-per-lane copies of one V stage
    static constexpr int VC = (VCOPIES + 3) / 4;  // per wave (padding copies go to the sink)
    static constexpr int CPS = 4 + VC;            // copies per wave per stage
    static constexpr int LDS = NS * SB + SINK;
};

template <int RK32, bool TRANS_OUT>
__device__ __forceinline__ void contract_tile(uint8_t* smem, const uint16_t* __restrict__ U,
                                              const uint16_t* __restrict__ V, float* __restrict__ out, int64_t L,
                                              int BIG, int r, float s, int tile, int64_t per) {
    using Cfg = ContractCfg<RK32>;
    constexpr int RP = Cfg::RP, NS = Cfg::NS, SB = Cfg::SB;
    const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, h = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int i0 = tile * 256;
    const int64_t t0 = (int64_t)blockIdx.y * per;
    const int64_t t1 = t0 + per < L ? t0 + per : L;
    const int nst = (int)((t1 - t0 + CK - 1) / CK);
    const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
    const void* zsrc = (const uint8_t*)g_zero_page + 16 * lane;

    // U copy q of this wave fills tile rows 2(4 wave + q) + h of the stage
    // (lane l32 -> 16-byte chunk l32 in LDS, logical chunk swz_chunk(row, l32)).
    int64_t ugo[4];  // element offset of the lane's chunk from the stage's first token row
    int urow[4];
    bool ucol[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        urow[q] = 2 * (4 * wave + q) + h;
        const int gi = i0 + 8 * swz_chunk(urow[q], l32);
        ucol[q] = gi < BIG;  // BIG % 8 == 0: a chunk is wholly in or out
        ugo[q] = (int64_t)urow[q] * BIG + gi;
    }
    // V copy m of this wave is stage copy c = wave + 4m: bytes 1024c + 16 lane
    // of the contiguous [32][RP] slab, token row (1024c + 16 lane) / (2 RP).
    int vrow[Cfg::VC];
    bool vreal[Cfg::VC];
#pragma unroll
    for (int m = 0; m < Cfg::VC; ++m) {
        const int c = wave + 4 * m;
        vreal[m] = c < Cfg::VCOPIES;
        vrow[m] = (1024 * c + 16 * lane) / (2 * RP);
    }
    auto issue = [&](int st) {
        const int64_t tc = t0 + (int64_t)CK * st;
        const uint32_t base = lds0 + (uint32_t)((st % NS) * SB);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const bool ok = ucol[q] && tc + urow[q] < t1;
            copy16_to_lds(ok ? (const void*)(U + tc * BIG + ugo[q]) : zsrc, base + 1024 * (4 * wave + q));
        }
#pragma unroll
        for (int m = 0; m < Cfg::VC; ++m) {
            const int c = wave + 4 * m;
            const bool ok = vreal[m] && tc + vrow[m] < t1;
            const void* src = ok ? (const void*)((const uint8_t*)(V + tc * RP) + 1024 * c + 16 * lane) : zsrc;
            copy16_to_lds(src, vreal[m] ? base + UB + 1024 * c : lds0 + (uint32_t)(NS * SB));
        }
    };

    f32x16 acc[2][RK32];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int jb = 0; jb < RK32; ++jb)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[a][jb][v] = 0.f;
    // transpose-read offsets: U stage rows = tokens (512 B rows, swizzled),
    // V stage rows = tokens (RP bf16 each, plain)
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

#pragma unroll
    for (int st = 0; st < NS - 1; ++st) issue(st);
    for (int st = 0; st < nst; ++st) {
        // stage st has landed and every wave is done with stage st - 1,
        // whose buffer the copies of stage st + NS - 1 overwrite
        stage_barrier<(NS - 2) * Cfg::CPS>();
        issue(st + NS - 1);
        const uint8_t* sb = smem + (st % NS) * SB;
#pragma unroll
        for (int kc = 0; kc < CK / 16; ++kc) {
            const int ro = 16 * kc;
            bf16x8 fu[2], fv[RK32];
#pragma unroll
            for (int a = 0; a < 2; ++a)
                fu[a] = frag_from_tr(lds_tr_read(sb + ro * kRowBytes + offU[a][0]),
                                     lds_tr_read(sb + ro * kRowBytes + offU[a][1]));
#pragma unroll
            for (int jb = 0; jb < RK32; ++jb)
                fv[jb] = frag_from_tr(lds_tr_read(sb + offV[jb][0] + ro * RP * 2),
                                      lds_tr_read(sb + offV[jb][1] + ro * RP * 2));
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int jb = 0; jb < RK32; ++jb)
                    acc[a][jb] = TRANS_OUT ? mfma_32x32x16(fv[jb], fu[a], acc[a][jb])
                                           : mfma_32x32x16(fu[a], fv[jb], acc[a][jb]);
        }
    }
    // no LDS copy may still be in flight when the workgroup ends
    wait_vmcnt<0>();
    // accumulator element v of block (a, jb) sits at row 8(v/4) + 4h + v%4,
    // column l32 of the 32 x 32 block: (i, j) for dB, (j, i) for dA
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int jb = 0; jb < RK32; ++jb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int rr = 8 * (v >> 2) + 4 * h + (v & 3);
                if (TRANS_OUT) {
                    const int j = 32 * jb + rr, i = i0 + 64 * wave + 32 * a + l32;
                    if (j < r && i < BIG) atomicAdd(out + (int64_t)j * BIG + i, s * acc[a][jb][v]);
                } else {
                    const int i = i0 + 64 * wave + 32 * a + rr, j = 32 * jb + l32;
                    if (j < r && i < BIG) atomicAdd(out + (int64_t)i * r + j, s * acc[a][jb][v]);
                }
            }
}

// grid.x: the ceil(R/256) dB tiles, then the ceil(C/256) dA tiles; grid.y: token slices
template <int RK32>
__global__ __launch_bounds__(NT) void contract_kernel(const uint16_t* __restrict__ dY, const uint16_t* __restrict__ X,
                                                      const uint16_t* __restrict__ P, const uint16_t* __restrict__ Q,
                                                      float* __restrict__ dB, float* __restrict__ dA, int64_t L, int R,
                                                      int C, int r, float s, int rb, int64_t per) {
    __shared__ __attribute__((aligned(1024))) uint8_t smem[ContractCfg<RK32>::LDS];
    const int bx = blockIdx.x;
    if (bx < rb)
        contract_tile<RK32, false>(smem, dY, P, dB, L, R, r, s, bx, per);
    else
        contract_tile<RK32, true>(smem, X, Q, dA, L, C, r, s, bx - rb, per);
}

template <int RK32>
hipError_t launch_rk(const LayerArgs& a, hipStream_t st) {
    auto* X = (const uint16_t*)a.X;
    auto* dY = (const uint16_t*)a.dY;
    auto* A = (const uint16_t*)a.A;
    const int64_t pq = ste_pq_bytes(a.L, a.r);
    uint16_t* P = (uint16_t*)a.ste_ws;
    uint16_t* Q = (uint16_t*)((uint8_t*)a.ste_ws + pq);
    uint16_t* BT = (uint16_t*)((uint8_t*)a.ste_ws + 2 * pq);
    const dim3 rgrid((unsigned)((a.L + 31) / 32), 2);
    bool staged = false;
    if constexpr (RK32 > 1) {
        staged = a.R >= kStagedMinK || a.C >= kStagedMinK;
        if (staged)
            hipLaunchKernelGGL((rows_staged_kernel<RK32>), rgrid, dim3(NT), 0, st, X, A, dY, (const uint16_t*)BT, P,
                               Q, a.L, (int)a.R, (int)a.C, (int)a.r);
    }
    if (!staged)
        hipLaunchKernelGGL((rows_kernel<RK32>), rgrid, dim3(NT), 0, st, X, A, dY, (const uint16_t*)BT, P, Q, a.L,
                           (int)a.R, (int)a.C, (int)a.r);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // Token slices: about two workgroups per CU over both products, at
    // least 128 tokens each (fewer slices also mean fewer atomics).
    const int64_t rb = (a.R + 255) / 256, cb = (a.C + 255) / 256;
    int64_t splits = (512 + rb + cb - 1) / (rb + cb);
    const int64_t max_splits = (a.L + 127) / 128;
    if (splits > max_splits) splits = max_splits;
    if (splits > 65535) splits = 65535;
    if (splits < 1) splits = 1;
    const int64_t per = ((a.L + splits - 1) / splits + CK - 1) / CK * CK;
    splits = (a.L + per - 1) / per;
    hipLaunchKernelGGL((contract_kernel<RK32>), dim3((unsigned)(rb + cb), (unsigned)splits), dim3(NT), 0, st, dY, X,
                       (const uint16_t*)P, (const uint16_t*)Q, a.dB, a.dA, a.L, (int)a.R, (int)a.C, (int)a.r, a.scale,
                       (int)rb, per);
    return hipGetLastError();
}

}  // namespace

size_t ste_workspace_bytes(int64_t R, int64_t L, int64_t r) {
    // P, Q (L x rank_pad(r)) and B^T (r x R), bf16, each 256-byte aligned
    return static_cast<size_t>(2 * ste_pq_bytes(L, r) + (2 * r * R + 255) / 256 * 256);
}

hipError_t launch_ste_bf16(const LayerArgs& a, hipStream_t st) {
    const int64_t nB = a.R * a.r, nA = a.r * a.C;
    // B^T takes ceil(R / 64) workgroups; the zeroing about 16 floats per thread
    int64_t g = (a.R + BT_ROWS - 1) / BT_ROWS;
    const int64_t gz = (nB + nA + 16 * NT - 1) / (16 * NT);
    if (gz > g) g = gz < 2048 ? gz : 2048;
    uint16_t* BT = (uint16_t*)((uint8_t*)a.ste_ws + 2 * ste_pq_bytes(a.L, a.r));
    hipLaunchKernelGGL(prep_kernel, dim3((unsigned)g), dim3(NT), 0, st, (const uint16_t*)a.B, BT, a.dB, a.dA, a.R,
                       (int)a.r, nB, nA);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.L == 0) return e;  // no tokens: dB, dA stay zero
    switch ((a.r + 31) / 32) {
        case 1: return launch_rk<1>(a, st);
        case 2: return launch_rk<2>(a, st);
        case 3: return launch_rk<3>(a, st);
        case 4: return launch_rk<4>(a, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace lors
