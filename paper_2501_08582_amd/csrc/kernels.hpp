// Internal launcher interface between the C ABI (abi.cpp) and the kernels.
// Every launcher assumes its arguments were validated by the ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lors {

struct LayerArgs {
    int64_t R, C, L, r;
    float scale;
    bool two_four;          // packed mask layout: 2:4 codes (else bitmap)
    bool sparse_mfma;       // forward on the structured-sparse MFMA (2:4, bf16, r <= 64)
    const void* X;          // L x C
    const void* W;          // R x C
    const uint32_t* M;      // R x ceil(C/32), the caller's layout
    const uint32_t* Mt;     // C x ceil(R/32) transposed bitmap, K-step-major (mt_index; backward only)
    bool reuse_mt;          // Mt already holds the transposed mask
    const void* B;          // R x r
    const void* A;          // r x C
    const void* bias;       // R or nullptr
    const void* dY;         // L x R
    void* Y;                // L x R
    void* dX;               // L x C or nullptr
    float* dB;              // R x r
    float* dA;              // r x C
    float* dbias;           // R or nullptr
    bool ste;               // straight-through adapter gradients (Section 2.3)
    void* ste_ws;           // P, Q, B^T scratch of the straight-through path
    void* b_pad;            // R x roundup8(r) scratch for B when r % 8 != 0 (bf16 backward), else nullptr
    bool clear_grads;       // the bf16 dX launch also clears dB and dA (combined backward)
    int64_t r_grad;         // rank of dB and dA (the caller's r; the dX passes change a.r)
    void* split_ws;         // fp32 partial sums of split tiles (forward, dX), or nullptr: no split
    int64_t split_budget;   // bytes of split_ws the partial sums may use
};

// Split of a grid of `tiles` output tiles whose K-loop has nk steps.  Whole
// waves of tiles (one per CU) run unsplit; a last, partial wave that fills at
// most half of the CUs is cut over K into `split` pieces per tile -- as many
// as fill the CUs, at most 8, each at least 4 K-steps, and no more than the
// pieces whose 256 KiB of fp32 partial sums fit in `max_part_bytes` (a
// kernel whose pieces need no partials passes kNoPartials) -- so that it
// does not leave most of the chip idle.  n_full: the tiles that run whole;
// the grid has n_full + (tiles - n_full) * split workgroups.
struct TailSplit {
    int n_full, split, grid;
};
constexpr int64_t kNoPartials = INT64_MAX;
constexpr int64_t kPieceBytes = 256 * 256 * 4;  // fp32 partials of one piece
TailSplit tail_split(int64_t tiles, int64_t nk, int64_t max_part_bytes);
// Bytes of fp32 partial sums a split grid of 256 x 256 tiles writes.
inline int64_t split_part_bytes(const TailSplit& t) {
    return t.split > 1 ? (int64_t)(t.grid - t.n_full) * kPieceBytes : 0;
}
// A short last wave of 256 x 256 tiles cut into thin tiles instead: each of
// its `tail` tiles becomes q thin tiles (q = 2, 4 or 8, as many as fill the
// CUs; q = 1: not cut) -- its two halves of 128 output features, each cut
// over the tokens into q/2 parts of 512/q tokens.  A thin tile runs the whole
// K-loop with the same per-element arithmetic as a whole tile, so its
// results are the same bits, and it needs no workspace.  Its waves merge 32
// rows of W' each instead of 64, so the merge shrinks with the tile, though
// less than the matrix work does when the tokens are cut too.  Applies to a
// wave that fills at most half of the CUs, like tail_split.
// n_full: the tiles that run whole (the first n_full in the kernels' order).
struct ThinPlan {
    int n_full, tail, q;
};
ThinPlan thin_plan(int64_t tiles);
// Whether the forward (Y = X.W'^T, tiles over L x R, K = C) and the dX kernel
// (dX = dY.W', tiles over L x C, K = R) take their fixed-offset copies: whole
// 256 x 256 tiles and 64-wide K-steps, and per-lane byte offsets of 256 slab
// rows inside 32 bits.  Thin tiles need them; other shapes run whole tiles
// whose copies check every lane.
inline bool fwd_whole_tiles(int64_t L, int64_t R, int64_t C) {
    return L % 256 == 0 && R % 256 == 0 && C % 64 == 0 && 256 * C * 2 < (1ll << 31);
}
inline bool dx_whole_tiles(int64_t L, int64_t R, int64_t C) {
    return L % 256 == 0 && C % 256 == 0 && R % 64 == 0 && 256 * R * 2 < (1ll << 31) && 64 * C * 2 < (1ll << 31);
}
// out (rows x cols, bf16) on the split tiles = the sum of their pieces'
// partials in piece order (+ bias[col] when bias is not null), rounded once.
// Tile coordinates follow work_coords with the same tiles_m, tiles_n, group_m.
hipError_t launch_split_reduce_bf16(const float* part, int n_full, int split, int tiles_m, int tiles_n,
                                    int group_m, int64_t rows, int cols, const void* bias, void* out,
                                    hipStream_t s);

// bf16 path
hipError_t launch_fwd_bf16(const LayerArgs& a, hipStream_t s);
hipError_t launch_fwd24_bf16(const LayerArgs& a, hipStream_t s);      // 2:4 mask, sparse MFMA, rank <= 64
hipError_t launch_dx_bf16(const LayerArgs& a, hipStream_t s);
// The thin tiles of a short last wave (see ThinPlan): logical tiles first ..
// first+tail-1, each cut into q; single-pass ranks (a.r <= 64), whole-tile
// shapes.  ldb: row stride of B; ra: rows of A that exist; clear: the launch
// also clears dB and dA (it is the first of the dX launches).
hipError_t launch_fwd_thin_bf16(const LayerArgs& a, hipStream_t s, int ldb, int first, int tail, int q);
hipError_t launch_dx_thin_bf16(const LayerArgs& a, hipStream_t s, int ldb, int ra, int first, int tail, int q,
                               bool clear);
hipError_t launch_g_bf16(const LayerArgs& a, hipStream_t s);
hipError_t launch_ste_bf16(const LayerArgs& a, hipStream_t s);  // dB, dA of the straight-through backward
size_t ste_workspace_bytes(int64_t R, int64_t L, int64_t r);
hipError_t launch_dbias_bf16(const LayerArgs& a, hipStream_t s);

// fp32 path
hipError_t launch_fwd_f32(const LayerArgs& a, hipStream_t s);
hipError_t launch_dx_f32(const LayerArgs& a, hipStream_t s);
hipError_t launch_g_f32(const LayerArgs& a, hipStream_t s);
hipError_t launch_dbias_f32(const LayerArgs& a, hipStream_t s);

// helpers
hipError_t launch_zero_f32(float* p, int64_t n, hipStream_t s);
// out (R x rp, bf16) = B (R x r) with its columns r .. rp-1 set to zero
hipError_t launch_pad_cols_bf16(const void* B, int64_t R, int64_t r, int64_t rp, void* out, hipStream_t s);
// clears two fp32 buffers with one launch
hipError_t launch_zero2_f32(float* a, int64_t na, float* b, int64_t nb, hipStream_t s);
hipError_t launch_mask_pack(const uint8_t* dense, int64_t R, int64_t C, bool two_four,
                            uint32_t* packed, int64_t* first_bad, hipStream_t s);
hipError_t launch_mask_from_weight(const void* W, bool w_is_bf16, int64_t R, int64_t C,
                                   bool two_four, uint32_t* packed, int64_t* first_bad,
                                   hipStream_t s);
// Transposed bitmap of a packed mask: word j*ceil(R/32) + i/32, bit i % 32
// is the keep bit of element (i, j).
hipError_t launch_mask_transpose(const uint32_t* packed, int64_t R, int64_t C, bool two_four,
                                 uint32_t* mt, hipStream_t s);
hipError_t launch_mask_unpack(const uint32_t* packed, int64_t R, int64_t C, bool two_four,
                              uint8_t* dense, hipStream_t s);

}  // namespace lors
