// Device-side building blocks shared by the gfx950 kernels: vector types,
// the bf16 MFMA wrapper, bf16 conversions and the packed-mask decoders.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lors {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// D(32x32, fp32) += A(32x16, bf16) * B(16x32, bf16).
// Operand layout per lane l (h = l / 32):
//   A: row l % 32, k = 8h .. 8h+7     B: column l % 32, k = 8h .. 8h+7
//   D: element v (0..15) is row 8*(v/4) + 4h + (v%4), column l % 32.
__device__ __forceinline__ f32x16 mfma_32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h16) {
    return __uint_as_float(h16 << 16);
}

// Round-to-nearest-even fp32 -> bf16 (gfx950 converts in hardware).
__device__ __forceinline__ __bf16 to_bf16(float f) { return (__bf16)f; }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    bf16x2 v;
    v[0] = (__bf16)lo;
    v[1] = (__bf16)hi;
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint16_t bf16_bits(float f) {
    return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// Keep-bits of 4 consecutive columns starting at bit position `pos` (a
// multiple of 4, 0..28) of a packed mask word.  Bit q of the result says
// whether column pos+q is kept.
//   bitmap: the four bits themselves.
//   2:4:    the group's nibble p0 | p1 << 2 names the two kept positions.
template <bool kTwoFour>
__device__ __forceinline__ uint32_t keep4(uint32_t word, uint32_t pos) {
    uint32_t nib = (word >> pos) & 0xFu;
    if constexpr (kTwoFour) {
        return (1u << (nib & 3u)) | (1u << (nib >> 2));
    } else {
        return nib;
    }
}

// Keep-bit of column `col` (0..31 within the word).
template <bool kTwoFour>
__device__ __forceinline__ uint32_t keep1(uint32_t word, uint32_t col) {
    uint32_t q = col & 3u;
    return (keep4<kTwoFour>(word, col & ~3u) >> q) & 1u;
}

__device__ __forceinline__ uint32_t ceil_div_u32(uint32_t a, uint32_t b) {
    return (a + b - 1) / b;
}

// Map a workgroup id to an output tile (tm, tn).
// MI355X dispatches consecutive workgroup ids round-robin over its 8 XCDs,
// each with a private L2.  When the grid divides evenly, ids are first
// regrouped so that every XCD receives one contiguous range of logical tiles;
// the logical order then walks `group_m` tile rows at a time, so the tiles an
// XCD holds at once share few operand panels.
__device__ __forceinline__ void group_coords(int t, int tiles_m, int tiles_n, int group_m, int& tm, int& tn) {
    const int per_group = group_m * tiles_n;
    const int g = t / per_group;
    const int first_m = g * group_m;
    const int gsz = min(tiles_m - first_m, group_m);
    const int within = t - g * per_group;
    tm = first_m + within % gsz;
    tn = within / gsz;
}

__device__ __forceinline__ void tile_coords(int bid, int tiles_m, int tiles_n, int group_m,
                                            int& tm, int& tn) {
    const int total = tiles_m * tiles_n;
    int t = bid;
    if ((total & 7) == 0) t = (bid & 7) * (total >> 3) + (bid >> 3);
    group_coords(t, tiles_m, tiles_n, group_m, tm, tn);
}

// Tile and K-steps of a workgroup when the grid's last, partial wave of tiles
// is split over K (see tail_split in kernels.hpp).  Ids below n_full take
// whole tiles -- logical tiles 0 .. n_full-1, regrouped over the XCDs as in
// tile_coords -- with all nk_all K-steps.  Each remaining logical tile is cut
// into `split` pieces of consecutive K-steps, one piece per id:
// piece p covers K-steps [nk_all*p/split, nk_all*(p+1)/split).
// (K-step counts fit 32 bits: every extent is below 2^31 and a K-step spans
// 64 elements.)
__device__ __forceinline__ void work_coords(int bid, int tiles_m, int tiles_n, int group_m, int n_full,
                                            int split, int nk_all, int& tm, int& tn, int& kbeg, int& nk) {
    int t;
    if (bid < n_full) {
        t = bid;
        if ((n_full & 7) == 0) t = (bid & 7) * (n_full >> 3) + (bid >> 3);
        kbeg = 0;
        nk = nk_all;
    } else {
        const int j = bid - n_full;
        const int q = j / split, p = j - q * split;
        t = n_full + q;
        kbeg = nk_all * p / split;
        nk = nk_all * (p + 1) / split - kbeg;
    }
    group_coords(t, tiles_m, tiles_n, group_m, tm, tn);
}

// Tile and sub-tile of a workgroup of a thin-tile grid (see thin_plan in
// kernels.hpp): logical tiles first .. first+tail-1, in group_coords' order,
// each cut into q sub-tiles u = 0 .. q-1, one per id (the kernel maps u to a
// feature half and a token part).  When tail is a multiple of 8, the q
// sub-tiles of a tile get ids of one XCD (ids are dealt to the 8 XCDs
// round-robin), so they share its weight slabs in that XCD's L2.
__device__ __forceinline__ void thin_coords(int bid, int tiles_m, int tiles_n, int group_m, int first, int tail,
                                            int q, int& tm, int& tn, int& u) {
    int i;
    if ((tail & 7) == 0) {
        const int x = bid & 7, y = bid >> 3;
        u = y % q;
        i = 8 * (y / q) + x;
    } else {
        i = bid / q;
        u = bid - i * q;
    }
    group_coords(first + i, tiles_m, tiles_n, group_m, tm, tn);
}

// Index of word iw (rows 32 iw .. 32 iw + 31 of R) of column col in the
// transposed mask M^T (C columns, wprT words each).  M^T is stored K-step-major:
// the two words of each aligned pair (2p, 2p + 1) -- the 64 rows of R that
// one K-step of dX covers -- form one block, column after column, so the
// columns of a dX tile read one contiguous run per K-step; with an odd word
// count the last word forms a block of width 1.
__device__ __forceinline__ int64_t mt_index(int64_t col, int iw, int64_t C, int wprT) {
    const int p2 = iw & ~1;
    const int width = min(2, wprT - p2);
    return (int64_t)p2 * C + col * width + (iw - p2);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ u32x4 zero_u32x4() { return u32x4{0u, 0u, 0u, 0u}; }

// Eight bf16 sums a + b (pairs packed in 32-bit words), each rounded once to
// bf16 from the fp32 sum.
__device__ __forceinline__ u32x4 add_bf16x8(u32x4 a, u32x4 b) {
    u32x4 o;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const float lo = __uint_as_float(a[p] << 16) + __uint_as_float(b[p] << 16);
        const float hi = __uint_as_float(a[p] & 0xFFFF0000u) + __uint_as_float(b[p] & 0xFFFF0000u);
        o[p] = pack_bf16x2(lo, hi);
    }
    return o;
}

// 16-bit element e (0..7) of a 16-byte vector.
__device__ __forceinline__ uint32_t u16_at(u32x4 v, int e) {
    return (v[e >> 1] >> ((e & 1) * 16)) & 0xFFFFu;
}

}  // namespace lors
