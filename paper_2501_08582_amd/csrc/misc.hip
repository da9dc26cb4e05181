// Mask packing (dense 0/1 or weight != 0 -> 1 bit per element), unpacking,
// output clearing, the bias gradient, and the split of a short last wave of
// tiles over K (the rule and the reduction of the pieces' partial sums).
//
// Packed layouts (the paper keeps the mask as a dense boolean; the packing is
// this library's own):
//   bitmap: element (i, j) is bit j % 32 of word i*ceil(C/32) + j/32
//   2:4:    group g of row i keeps p0 < p1; nibble p0 | p1 << 2 at bits
//           4*(g % 8) of word i*ceil(C/32) + g/8
// One thread produces one packed word from 32 consecutive elements of a row.
#include <atomic>

#include "device_common.hpp"
#include "kernels.hpp"

namespace lors {
namespace {

constexpr int NT = 256;
constexpr unsigned long long kNoBad = ~0ull;

// Reads the 32 "kept" flags of word w of row i (columns 32w .. 32w+31, those
// at or past C read as not kept).  Source is either a dense uint8 mask or a
// weight matrix (kept = value != 0, with -0 counting as zero).
struct DenseSrc {
    const uint8_t* p;
    __device__ uint32_t flags(int64_t i, int C, int w) const {
        const uint8_t* row = p + i * C;
        const int c0 = w * 32;
        uint32_t bits = 0;
        if (c0 + 32 <= C && (((uintptr_t)(row + c0)) & 15) == 0) {
            const u32x4 a = *(const u32x4*)(row + c0);
            const u32x4 b = *(const u32x4*)(row + c0 + 16);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const uint32_t v = q < 4 ? a[q] : b[q - 4];
#pragma unroll
                for (int e = 0; e < 4; ++e) bits |= (((v >> (8 * e)) & 0xFFu) != 0u ? 1u : 0u) << (4 * q + e);
            }
        } else {
            for (int e = 0; e < 32 && c0 + e < C; ++e) bits |= (row[c0 + e] != 0 ? 1u : 0u) << e;
        }
        return bits;
    }
};

struct Bf16WeightSrc {
    const uint16_t* p;
    __device__ uint32_t flags(int64_t i, int C, int w) const {
        const uint16_t* row = p + i * C;
        const int c0 = w * 32;
        uint32_t bits = 0;
        for (int e = 0; e < 32 && c0 + e < C; ++e) bits |= ((row[c0 + e] & 0x7FFFu) != 0u ? 1u : 0u) << e;
        return bits;
    }
};

struct F32WeightSrc {
    const float* p;
    __device__ uint32_t flags(int64_t i, int C, int w) const {
        const float* row = p + i * C;
        const int c0 = w * 32;
        uint32_t bits = 0;
        for (int e = 0; e < 32 && c0 + e < C; ++e) bits |= (row[c0 + e] != 0.f ? 1u : 0u) << e;
        return bits;
    }
};

template <class Src>
__global__ __launch_bounds__(NT) void pack_bitmap_kernel(Src src, int64_t R, int C, int wpr,
                                                         uint32_t* __restrict__ out) {
    const int64_t t = (int64_t)blockIdx.x * NT + threadIdx.x;
    if (t >= R * wpr) return;
    const int64_t i = t / wpr;
    const int w = (int)(t - i * wpr);
    out[t] = src.flags(i, C, w);
}

template <class Src>
__global__ __launch_bounds__(NT) void pack_2_4_kernel(Src src, int64_t R, int C, int wpr,
                                                      uint32_t* __restrict__ out,
                                                      unsigned long long* __restrict__ first_bad) {
    const int64_t t = (int64_t)blockIdx.x * NT + threadIdx.x;
    if (t >= R * wpr) return;
    const int64_t i = t / wpr;
    const int w = (int)(t - i * wpr);
    const uint32_t f = src.flags(i, C, w);
    uint32_t word = 0;
    const int groups = C / 4;
    for (int n = 0; n < 8; ++n) {
        const int g = w * 8 + n;
        if (g >= groups) break;
        const uint32_t nib = (f >> (4 * n)) & 0xFu;
        if (__popc(nib) != 2) {
            atomicMin(first_bad, (unsigned long long)(i * groups + g));
            continue;
        }
        const uint32_t p0 = __ffs(nib) - 1;
        const uint32_t p1 = 31 - __clz(nib);
        word |= (p0 | (p1 << 2)) << (4 * n);
    }
    out[t] = word;
}

__global__ void set_u64_kernel(unsigned long long* p, unsigned long long v) { *p = v; }

__global__ void finish_first_bad_kernel(unsigned long long* p) {
    if (*p == kNoBad) *(long long*)p = -1;
}

template <bool TWO_FOUR>
__global__ __launch_bounds__(NT) void unpack_kernel(const uint32_t* __restrict__ in, int64_t R, int C,
                                                    int wpr, uint8_t* __restrict__ dense) {
    const int64_t t = (int64_t)blockIdx.x * NT + threadIdx.x;
    if (t >= R * wpr) return;
    const int64_t i = t / wpr;
    const int w = (int)(t - i * wpr);
    const uint32_t word = in[t];
    uint8_t* row = dense + i * C;
    const int c0 = w * 32;
    for (int e = 0; e < 32 && c0 + e < C; ++e) row[c0 + e] = (uint8_t)keep1<TWO_FOUR>(word, (uint32_t)e);
}

// Transposed bitmap (K-step-major, see mt_index): one wave handles a 32-row
// block of the mask and two 32-column words.  Lane l < 32 reads row
// 32*iw + l of word jw, lane l >= 32 the same row of word jw + 1 (2:4 codes
// are first expanded to keep bits); one ballot per bit position then yields,
// for every column, its 32 keep bits.
template <bool TWO_FOUR>
__global__ __launch_bounds__(NT) void transpose_kernel(const uint32_t* __restrict__ in, int64_t R, int C, int wpr,
                                                       int wprT, uint32_t* __restrict__ out) {
    const int lane = threadIdx.x & 63;
    const int64_t task = (int64_t)blockIdx.x * (NT / 64) + (threadIdx.x >> 6);
    const int jpairs = (wpr + 1) >> 1;
    const int64_t iw = task / jpairs;
    const int jw = (int)(task % jpairs) * 2 + (lane >> 5);
    if (iw >= wprT) return;  // whole wave leaves together
    const int64_t row = iw * 32 + (lane & 31);
    uint32_t w = (row < R && jw < wpr) ? in[row * wpr + jw] : 0u;
    if constexpr (TWO_FOUR) {
        uint32_t keep = 0;
#pragma unroll
        for (int n = 0; n < 8; ++n) {
            const uint32_t code = (w >> (4 * n)) & 0xFu;
            keep |= ((1u << (code & 3u)) | (1u << (code >> 2))) << (4 * n);
        }
        // groups past C/4 hold no codes: clear their expansion
        const int cols = C - 32 * jw;
        w = cols >= 32 ? keep : (cols > 0 ? keep & ((1u << cols) - 1u) : 0u);
    }
    uint32_t mine = 0;
#pragma unroll
    for (int b = 0; b < 32; ++b) {
        const uint64_t bal = __ballot((w >> b) & 1u);
        const uint32_t lo = (uint32_t)bal, hi = (uint32_t)(bal >> 32);
        mine = ((lane & 31) == b) ? (lane < 32 ? lo : hi) : mine;
    }
    const int64_t col = (int64_t)32 * jw + (lane & 31);
    if (jw < wpr && col < C) out[mt_index(col, (int)iw, C, wprT)] = mine;
}

__global__ __launch_bounds__(NT) void zero_kernel(float* __restrict__ p, int64_t n) {
    for (int64_t t = (int64_t)blockIdx.x * NT + threadIdx.x; t < n; t += (int64_t)gridDim.x * NT) p[t] = 0.f;
}

__global__ __launch_bounds__(NT) void zero2_kernel(float* __restrict__ a, int64_t na, float* __restrict__ b,
                                                   int64_t nb) {
    const int64_t stride = (int64_t)gridDim.x * NT;
    for (int64_t t = (int64_t)blockIdx.x * NT + threadIdx.x; t < na + nb; t += stride) {
        if (t < na) a[t] = 0.f;
        else b[t - na] = 0.f;
    }
}

// out[R x rp] = B[R x r] with columns r .. rp-1 zero (bf16 bit patterns).
__global__ __launch_bounds__(NT) void pad_cols_kernel(const uint16_t* __restrict__ B, int64_t R, int r, int rp,
                                                      uint16_t* __restrict__ out) {
    const int64_t n = R * rp, stride = (int64_t)gridDim.x * NT;
    for (int64_t t = (int64_t)blockIdx.x * NT + threadIdx.x; t < n; t += stride) {
        const int64_t i = t / rp;
        const int j = (int)(t - i * rp);
        out[t] = j < r ? B[i * r + j] : (uint16_t)0;
    }
}

// dbias[R] = column sums of dY[L x R]; thread owns one column and a slice of
// rows, partial sums are combined with fp32 atomics (dbias zeroed first).
template <bool BF16>
__global__ __launch_bounds__(NT) void dbias_kernel(const void* __restrict__ dY, int64_t L, int R,
                                                   int64_t rows_per_block, float* __restrict__ dbias) {
    const int col = blockIdx.x * NT + threadIdx.x;
    if (col >= R) return;
    const int64_t l0 = (int64_t)blockIdx.y * rows_per_block;
    const int64_t l1 = min(L, l0 + rows_per_block);
    float acc = 0.f;
    for (int64_t l = l0; l < l1; ++l) {
        if constexpr (BF16)
            acc += bf16_bits_to_f32(((const uint16_t*)dY)[l * R + col]);
        else
            acc += ((const float*)dY)[l * R + col];
    }
    atomicAdd(dbias + col, acc);
}

template <class Src>
hipError_t launch_pack(Src src, int64_t R, int64_t C, bool two_four, uint32_t* packed,
                       int64_t* first_bad, hipStream_t st) {
    const int wpr = (int)((C + 31) / 32);
    const int64_t n = R * wpr;
    const unsigned blocks = (unsigned)((n + NT - 1) / NT);
    if (two_four) {
        auto* fb = (unsigned long long*)first_bad;
        hipLaunchKernelGGL(set_u64_kernel, dim3(1), dim3(1), 0, st, fb, kNoBad);
        if (n > 0)
            hipLaunchKernelGGL(pack_2_4_kernel<Src>, dim3(blocks), dim3(NT), 0, st, src, R, (int)C, wpr,
                               packed, fb);
        hipLaunchKernelGGL(finish_first_bad_kernel, dim3(1), dim3(1), 0, st, fb);
    } else {
        if (first_bad)
            hipLaunchKernelGGL(set_u64_kernel, dim3(1), dim3(1), 0, st, (unsigned long long*)first_bad,
                               ~0ull);  // -1
        if (n > 0)
            hipLaunchKernelGGL(pack_bitmap_kernel<Src>, dim3(blocks), dim3(NT), 0, st, src, R, (int)C, wpr,
                               packed);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_mask_pack(const uint8_t* dense, int64_t R, int64_t C, bool two_four,
                            uint32_t* packed, int64_t* first_bad, hipStream_t st) {
    return launch_pack(DenseSrc{dense}, R, C, two_four, packed, first_bad, st);
}

hipError_t launch_mask_from_weight(const void* W, bool w_is_bf16, int64_t R, int64_t C, bool two_four,
                                   uint32_t* packed, int64_t* first_bad, hipStream_t st) {
    if (w_is_bf16) return launch_pack(Bf16WeightSrc{(const uint16_t*)W}, R, C, two_four, packed, first_bad, st);
    return launch_pack(F32WeightSrc{(const float*)W}, R, C, two_four, packed, first_bad, st);
}

hipError_t launch_mask_unpack(const uint32_t* packed, int64_t R, int64_t C, bool two_four, uint8_t* dense,
                              hipStream_t st) {
    const int wpr = (int)((C + 31) / 32);
    const int64_t n = R * wpr;
    if (n == 0) return hipSuccess;
    const unsigned blocks = (unsigned)((n + NT - 1) / NT);
    if (two_four)
        hipLaunchKernelGGL(unpack_kernel<true>, dim3(blocks), dim3(NT), 0, st, packed, R, (int)C, wpr, dense);
    else
        hipLaunchKernelGGL(unpack_kernel<false>, dim3(blocks), dim3(NT), 0, st, packed, R, (int)C, wpr, dense);
    return hipGetLastError();
}

hipError_t launch_mask_transpose(const uint32_t* packed, int64_t R, int64_t C, bool two_four, uint32_t* mt,
                                 hipStream_t st) {
    const int wpr = (int)((C + 31) / 32);
    const int wprT = (int)((R + 31) / 32);
    const int64_t tasks = (int64_t)wprT * ((wpr + 1) / 2);
    if (tasks == 0) return hipSuccess;
    const unsigned blocks = (unsigned)((tasks + (NT / 64) - 1) / (NT / 64));
    if (two_four)
        hipLaunchKernelGGL(transpose_kernel<true>, dim3(blocks), dim3(NT), 0, st, packed, R, (int)C, wpr, wprT, mt);
    else
        hipLaunchKernelGGL(transpose_kernel<false>, dim3(blocks), dim3(NT), 0, st, packed, R, (int)C, wpr, wprT, mt);
    return hipGetLastError();
}

hipError_t launch_zero_f32(float* p, int64_t n, hipStream_t st) {
    if (n == 0) return hipSuccess;
    const int64_t want = (n + NT - 1) / NT;
    const unsigned blocks = (unsigned)(want < 4096 ? want : 4096);
    hipLaunchKernelGGL(zero_kernel, dim3(blocks), dim3(NT), 0, st, p, n);
    return hipGetLastError();
}

// Workgroup (q, rb): rows 4*rb .. 4*rb+3 of split tile q (logical tile
// n_full + q); thread t covers 4 columns of one of those rows.
__global__ __launch_bounds__(NT) void split_reduce_kernel(const float* __restrict__ part, int n_full, int split,
                                                          int tiles_m, int tiles_n, int group_m, int64_t rows,
                                                          int cols, const uint16_t* __restrict__ bias,
                                                          uint16_t* __restrict__ out) {
    const int q = blockIdx.x >> 6, rb = blockIdx.x & 63;
    int tm, tn;
    group_coords(n_full + q, tiles_m, tiles_n, group_m, tm, tn);
    const int tr = 4 * rb + (threadIdx.x >> 6), tc = 4 * (threadIdx.x & 63);
    const int64_t gm = (int64_t)tm * 256 + tr;
    const int gn = tn * 256 + tc;
    if (gm >= rows || gn >= cols) return;
    f32x4 sum = {0.f, 0.f, 0.f, 0.f};
    for (int p = 0; p < split; ++p)
        sum += *(const f32x4*)(part + ((int64_t)q * split + p) * 65536 + tr * 256 + tc);
    uint16_t* o = out + gm * cols + gn;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        if (gn + e < cols) {
            const float b = bias != nullptr ? bf16_bits_to_f32(bias[gn + e]) : 0.f;
            o[e] = bf16_bits(sum[e] + b);
        }
    }
}

hipError_t launch_split_reduce_bf16(const float* part, int n_full, int split, int tiles_m, int tiles_n,
                                    int group_m, int64_t rows, int cols, const void* bias, void* out,
                                    hipStream_t st) {
    const int tail = tiles_m * tiles_n - n_full;
    if (tail <= 0 || split < 2) return hipSuccess;
    hipLaunchKernelGGL(split_reduce_kernel, dim3(tail * 64), dim3(NT), 0, st, part, n_full, split, tiles_m, tiles_n,
                       group_m, rows, cols, (const uint16_t*)bias, (uint16_t*)out);
    return hipGetLastError();
}

// compute units of the current device, read once per device (calls from
// several host threads may both read it; they store the same value)
static int device_cus() {
    static std::atomic<int> cus_of[64];
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < 64) {
        int n = cus_of[dev].load(std::memory_order_relaxed);
        if (n == 0 && hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
            cus_of[dev].store(n, std::memory_order_relaxed);
        if (n > 0) cus = n;
    }
    return cus;
}

TailSplit tail_split(int64_t tiles, int64_t nk, int64_t max_part_bytes) {
    const int cus = device_cus();
    TailSplit t{(int)tiles, 1, (int)tiles};
    const int64_t tail = tiles % cus;
    if (tail == 0 || 2 * tail > cus) return t;
    int64_t s = cus / tail;
    if (s > 8) s = 8;
    if (s > nk / 4) s = nk / 4;
    if (max_part_bytes != kNoPartials) {
        const int64_t fit = max_part_bytes / (tail * kPieceBytes);
        if (s > fit) s = fit;
    }
    if (s < 2) return t;
    t.n_full = (int)(tiles - tail);
    t.split = (int)s;
    t.grid = (int)(t.n_full + tail * s);
    return t;
}

ThinPlan thin_plan(int64_t tiles) {
    const int cus = device_cus();
    ThinPlan t{(int)tiles, 0, 1};
    const int64_t tail = tiles % cus;
    if (tail == 0 || 2 * tail > cus) return t;
    int q = 2;
    while (q < 8 && 2 * q * tail <= cus) q *= 2;
    t.n_full = (int)(tiles - tail);
    t.tail = (int)tail;
    t.q = q;
    return t;
}

hipError_t launch_zero2_f32(float* a, int64_t na, float* b, int64_t nb, hipStream_t st) {
    const int64_t n = na + nb;
    if (n == 0) return hipSuccess;
    const int64_t want = (n + NT - 1) / NT;
    const unsigned blocks = (unsigned)(want < 2048 ? want : 2048);
    hipLaunchKernelGGL(zero2_kernel, dim3(blocks), dim3(NT), 0, st, a, na, b, nb);
    return hipGetLastError();
}

hipError_t launch_pad_cols_bf16(const void* B, int64_t R, int64_t r, int64_t rp, void* out, hipStream_t st) {
    const int64_t n = R * rp;
    if (n == 0) return hipSuccess;
    const int64_t want = (n + NT - 1) / NT;
    const unsigned blocks = (unsigned)(want < 2048 ? want : 2048);
    hipLaunchKernelGGL(pad_cols_kernel, dim3(blocks), dim3(NT), 0, st, (const uint16_t*)B, R, (int)r, (int)rp,
                       (uint16_t*)out);
    return hipGetLastError();
}

static hipError_t launch_dbias(const LayerArgs& a, hipStream_t st, bool bf16) {
    if (a.dbias == nullptr) return hipSuccess;
    hipError_t e = launch_zero_f32(a.dbias, a.R, st);
    if (e != hipSuccess || a.L == 0) return e;
    int64_t ychunks = (a.L + 255) / 256;
    if (ychunks > 4096) ychunks = 4096;
    const int64_t rows = (a.L + ychunks - 1) / ychunks;
    dim3 grid((unsigned)((a.R + NT - 1) / NT), (unsigned)ychunks), block(NT);
    if (bf16)
        hipLaunchKernelGGL(dbias_kernel<true>, grid, block, 0, st, a.dY, a.L, (int)a.R, rows, a.dbias);
    else
        hipLaunchKernelGGL(dbias_kernel<false>, grid, block, 0, st, a.dY, a.L, (int)a.R, rows, a.dbias);
    return hipGetLastError();
}

hipError_t launch_dbias_bf16(const LayerArgs& a, hipStream_t st) { return launch_dbias(a, st, true); }
hipError_t launch_dbias_f32(const LayerArgs& a, hipStream_t st) { return launch_dbias(a, st, false); }

}  // namespace lors
