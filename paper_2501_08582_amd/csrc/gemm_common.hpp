// Building blocks of the 4-wave gfx950 GEMM main loops: asynchronous
// global -> LDS copies, swizzled LDS tiles, and MFMA operand fragments read
// with the gfx950 LDS transpose load.
//
// Tiles are stored in LDS in their natural row-major order (one 512-byte row =
// 256 bf16) with the 16-byte chunks of row `row` permuted as
// chunk ^ (4 * (row % 4)), so that the 4-row x 16-column blocks fetched by
// ds_read_b64_tr_b16 hit 16 different bank groups per half wave.
#pragma once

#include "device_common.hpp"

namespace lors {

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

// 1 KiB of zeros (one copy per code object): the source of every lane whose
// tile element lies outside its tensor, so out-of-range parts of a tile read
// as 0.  Never written.
static __device__ __attribute__((aligned(1024))) uint32_t g_zero_page[256];

constexpr int kRowBytes = 512;  // one tile row: 256 bf16

__device__ __forceinline__ int swz_chunk(int row, int chunk) { return chunk ^ ((row & 3) << 2); }

// Byte offset of element (row, col) inside a swizzled 256-column tile.
__device__ __forceinline__ int tile_off(int row, int col) {
    return row * kRowBytes + (swz_chunk(row, col >> 3) << 4) + ((col & 7) << 1);
}

// LDS byte address of a pointer into __shared__ memory.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// One 16-byte global -> LDS copy per lane (global_load_lds_dwordx4): lane l's
// data lands at LDS byte address lds_wave_base + 16*l; lds_wave_base must be
// wave-uniform.  Issued as inline assembly so that the compiler does not
// serialise it against later LDS reads: completion is tracked explicitly with
// vmcnt (see stage_barrier).
// (M0 is written here and nowhere else in these kernels; one wait state
// separates the M0 write from the LDS DMA that reads it.)
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void copy16_to_lds(const void* src, uint32_t lds_wave_base) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(src), "s"(lds_wave_base)
                 : "memory", "m0");
}

// ---------------------------------------------------------------------------
// Slabs with 64 bf16 (128 bytes) per row, read one 16-byte chunk per lane
// (ds_read_b128).  Chunk c of row `row` is stored at c ^ ((row >> 1) & 7):
// the 16 lanes of one read pass (16 consecutive rows, same logical chunk)
// then cover all 64 banks.
// ---------------------------------------------------------------------------
constexpr int kRow64 = 128;

__device__ __forceinline__ int slab64_off(int row, int chunk) {
    return row * kRow64 + ((chunk ^ ((row >> 1) & 7)) << 4);
}

// Element (row, col) of a 64-column slab.
__device__ __forceinline__ int slab64_elem_off(int row, int col) {
    return slab64_off(row, col >> 3) + ((col & 7) << 1);
}

// Slabs with 64 bf16 per row that are read as transposed 4-row fragments
// (ds_read_b64_tr_b16): a 32-lane pass reads 4 consecutive rows x 4 chunks,
// and rows j and j + 2 are 256 bytes apart, on the same banks.  Chunk c of
// row j is therefore stored at c ^ tr64_swz(j), which gives every other row
// pair the other 64-byte half and makes the pass conflict-free.
__device__ __forceinline__ int tr64_swz(int row) { return ((row >> 1) & 1) << 2; }
__device__ __forceinline__ int tr64_elem_off(int row, int col) {
    return row * kRow64 + (((col >> 3) ^ tr64_swz(row)) << 4) + ((col & 7) << 1);
}

// Byte-to-select LUT: entry b holds four 32-bit AND masks, one per packed
// bf16 pair (2p, 2p+1), keeping element q iff bit q of the 8 keep bits is set.
// For the 2:4 layout the byte is two group codes and the keep bits are
// decoded from them.
template <bool TWO_FOUR>
__device__ __forceinline__ u32x4 select_lut_entry(uint32_t b) {
    uint32_t keep = b;
    if constexpr (TWO_FOUR) {
        const uint32_t lo = b & 0xFu, hi = b >> 4;
        keep = ((1u << (lo & 3u)) | (1u << (lo >> 2))) | (((1u << (hi & 3u)) | (1u << (hi >> 2))) << 4);
    }
    u32x4 e;
#pragma unroll
    for (int p = 0; p < 4; ++p)
        e[p] = (((keep >> (2 * p)) & 1u) ? 0x0000FFFFu : 0u) | (((keep >> (2 * p + 1)) & 1u) ? 0xFFFF0000u : 0u);
    return e;
}

// Half of a select entry: the two words for four consecutive elements whose
// keep bits are the nibble n (for the 2:4 layout: whose group code is n).
// The sixteen half entries make a 128-byte table; it spans distinct LDS
// banks, so lanes reading it with arbitrary nibbles never conflict (a lane
// group reading the 256-entry table of whole entries does, about 3.6-way on
// random masks).
template <bool TWO_FOUR>
__device__ __forceinline__ u32x2 select_lut16_entry(uint32_t n) {
    uint32_t keep = n;
    if constexpr (TWO_FOUR) keep = (1u << (n & 3u)) | (1u << (n >> 2));
    u32x2 e;
#pragma unroll
    for (int p = 0; p < 2; ++p)
        e[p] = (((keep >> (2 * p)) & 1u) ? 0x0000FFFFu : 0u) | (((keep >> (2 * p + 1)) & 1u) ? 0xFFFF0000u : 0u);
    return e;
}

// Select masks of the eight elements whose mask byte starts at bit `shift`
// of word w, from the 16-entry table at lut (two 8-byte reads).
__device__ __forceinline__ u32x4 read_sel16(const uint8_t* lut, uint32_t w, uint32_t shift) {
    // bit-field extracts, so that each address is one more shift-and-add
    const uint32_t nlo = __builtin_amdgcn_ubfe(w, shift, 4u);
    const uint32_t nhi = __builtin_amdgcn_ubfe(w, shift + 4u, 4u);
    const u32x2 lo = *(const u32x2*)(lut + (nlo << 3));
    const u32x2 hi = *(const u32x2*)(lut + (nhi << 3));
    return u32x4{lo[0], lo[1], hi[0], hi[1]};
}

// W' = select(M, W + s.T, 0) for eight consecutive elements: raw holds the
// eight bf16 of W (pairs), t the eight fp32 rank-r sums, sel the LUT masks.
__device__ __forceinline__ u32x4 merge8(u32x4 raw, const float* t, float s, u32x4 sel) {
    u32x4 out;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const float lo = __uint_as_float(raw[p] << 16);
        const float hi = __uint_as_float(raw[p] & 0xFFFF0000u);
        out[p] = pack_bf16x2(fmaf(s, t[2 * p], lo), fmaf(s, t[2 * p + 1], hi)) & sel[p];
    }
    return out;
}

// One 4-byte global -> LDS copy per lane (global_load_lds_dword): lane l's
// word lands at lds_wave_base + 4*l.
__device__ __forceinline__ void copy4_to_lds(const void* src, uint32_t lds_wave_base) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
                 :
                 : "v"(src), "s"(lds_wave_base)
                 : "memory", "m0");
}

// A wave-uniform pointer moved into scalar registers (the copies below take
// their base address from an SGPR pair).
template <typename T>
__device__ __forceinline__ const T* uniform_ptr(const T* p) {
    const uint64_t v = (uint64_t)(uintptr_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return (const T*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}

// The same copies addressed as a wave-uniform base (SGPR pair) plus a 32-bit
// per-lane byte offset: no per-lane 64-bit address arithmetic.
__device__ __forceinline__ void copy16s_to_lds(const void* sbase, uint32_t voff, uint32_t lds_wave_base) {
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(voff), "s"(sbase), "s"(lds_wave_base)
                 : "memory", "m0");
}
__device__ __forceinline__ void copy4s_to_lds(const void* sbase, uint32_t voff, uint32_t lds_wave_base) {
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
                 :
                 : "v"(voff), "s"(sbase), "s"(lds_wave_base)
                 : "memory", "m0");
}

// The wait states after the rank-r MFMA chains (see rank_mfma2): they cover
// the matrix-result -> VALU-read latency of T and keep the A fragments
// allocated until the matrix core has consumed them.
template <int RK, int NB>
__device__ __forceinline__ void rank_wait(f32x16 (&T)[NB], const bf16x8 (&a)[RK]) {
    static_assert(NB == 1 || NB == 2, "one or two 32-wide blocks");
    static_assert(RK >= 1 && RK <= 4, "ranks up to 64");
    if constexpr (NB == 2) {
        if constexpr (RK == 1)
            asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 2" : "+v"(T[0]), "+v"(T[1]) : "v"(a[0]));
        else if constexpr (RK == 2)
            asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 2" : "+v"(T[0]), "+v"(T[1]) : "v"(a[0]), "v"(a[1]));
        else if constexpr (RK == 3)
            asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 2" : "+v"(T[0]), "+v"(T[1]) : "v"(a[0]), "v"(a[1]), "v"(a[2]));
        else
            asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 2"
                         : "+v"(T[0]), "+v"(T[1])
                         : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]));
    } else {
        if constexpr (RK == 1)
            asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 2" : "+v"(T[0]) : "v"(a[0]));
        else if constexpr (RK == 2)
            asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 2" : "+v"(T[0]) : "v"(a[0]), "v"(a[1]));
        else if constexpr (RK == 3)
            asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 2" : "+v"(T[0]) : "v"(a[0]), "v"(a[1]), "v"(a[2]));
        else
            asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 2" : "+v"(T[0]) : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]));
    }
}

// T[nb] = sum over c of mfma(a[c], b[nb][c]) for nb < NB (two 32-wide blocks,
// or one for a tile of half the features), with T in VGPRs.
// The main accumulators fill the accumulation registers, so results that the
// VALU consumes are produced by inline-assembly MFMAs writing VGPRs directly
// (chained accumulation into the same registers needs no wait states).  The
// final s_nop block covers the matrix-result -> VALU-read latency; it also
// keeps the A fragments allocated until the matrix core has consumed them.
template <int RK, int NB>
__device__ __forceinline__ void rank_mfma2(f32x16 (&T)[NB], const bf16x8 (&a)[RK], const bf16x8 (&b)[NB][RK]) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(T[nb]) : "v"(a[0]), "v"(b[nb][0]));
#pragma unroll
        for (int c = 1; c < RK; ++c)
            asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+&v"(T[nb]) : "v"(a[c]), "v"(b[nb][c]));
    }
    rank_wait<RK, NB>(T, a);
}

// The same products accumulated onto T: T[nb] += sum over c of
// mfma(a[c], b[nb][c]).  T is written by VALU instructions just before (it
// holds W when the merge folds W into the matrix product), so each chain
// starts with wait states that cover a VALU write -> matrix source-C read,
// which the compiler cannot see through inline assembly.
template <int RK, int NB>
__device__ __forceinline__ void rank_mfma2_acc(f32x16 (&T)[NB], const bf16x8 (&a)[RK], const bf16x8 (&b)[NB][RK]) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        asm volatile("s_nop 4\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+&v"(T[nb]) : "v"(a[0]), "v"(b[nb][0]));
#pragma unroll
        for (int c = 1; c < RK; ++c)
            asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+&v"(T[nb]) : "v"(a[c]), "v"(b[nb][c]));
    }
    rank_wait<RK, NB>(T, a);
}

// One bf16 pair of W' = select(M, W + s.T, 0): raw holds the two bf16 of W,
// t0/t1 the rank-r sums, sel the 32-bit select mask of the pair.
__device__ __forceinline__ uint32_t merge_pair(uint32_t raw, float t0, float t1, float s, uint32_t sel) {
    return pack_bf16x2(fmaf(s, t0, __uint_as_float(raw << 16)), fmaf(s, t1, __uint_as_float(raw & 0xFFFF0000u))) & sel;
}

// Wait until at most N of this wave's vector-memory loads (including the
// LDS copies above) are outstanding, then barrier: afterwards every copy
// issued before the last N of every wave is visible in LDS.
template <int N>
__device__ __forceinline__ void stage_barrier() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" : : "n"(N) : "memory");
}

// Barrier after which LDS written or read before it may be reused.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" : : : "memory");
}

// ds_read_b64_tr_b16: within each group of 16 lanes, lane j supplies the
// address of row j/4, columns 4*(j%4) .. +3 of a 4 x 16 block of 16-bit
// values; lane i receives the 4 values of column i (rows 0..3).
__device__ __forceinline__ u32x2 lds_tr_read(const uint8_t* p) {
    i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p);
    return __builtin_bit_cast(u32x2, v);
}

// Byte offset, inside a swizzled tile whose rows are the MFMA K dimension,
// of this lane's part of the transpose read `t` (0 or 1) that builds the
// 32x32x16 operand of the 32 columns starting at col0 and the 16 rows
// starting at row0.  Lane l ends up with rows row0 + 8*(l/32) + 4t + {0..3}
// of column col0 + l%32, i.e. operand elements 4t .. 4t+3.
__device__ __forceinline__ int tr_frag_off(int lane, int row0, int col0, int t) {
    const int g = lane >> 4, j = lane & 15;
    const int row = row0 + 8 * (g >> 1) + 4 * t + (j >> 2);
    const int col = col0 + 16 * (g & 1) + 4 * (j & 3);
    return tile_off(row, col);
}

__device__ __forceinline__ bf16x8 frag_from_tr(u32x2 lo, u32x2 hi) {
    u32x4 v;
    v[0] = lo[0];
    v[1] = lo[1];
    v[2] = hi[0];
    v[3] = hi[1];
    return as_bf16x8(v);
}

// s_waitcnt vmcnt(n) leaving the LDS/export counters unconstrained (gfx9
// encoding: vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

#pragma clang diagnostic pop

}  // namespace lors
