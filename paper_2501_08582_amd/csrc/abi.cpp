// C ABI of the sparsity-preserved LoRA linear: argument validation, dispatch
// to the gfx950 kernels, and the host twins of the mask packer.
//
// Validation runs entirely on the host, in a fixed order (null, dtype/format,
// shape/range, alignment, alias, workspace), before any HIP call, so every
// rejected call is free of side effects.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "lors.h"
#include "kernels.hpp"

namespace {

constexpr int64_t kMaxExtent = (int64_t(1) << 31) - 1;
constexpr int64_t kMaxRank = 128;
// Largest byte count of any one argument.  Extents are below 2^31 each, so a
// product of two of them and an element size can exceed int64_t; every byte
// count is therefore checked against this bound before it is formed, and
// sums of a few such counts stay far from overflow.
constexpr int64_t kMaxBytes = int64_t(1) << 60;

// a * b * es when it is at most kMaxBytes (a, b >= 0, es in 1..8), else -1.
int64_t bytes_of(int64_t a, int64_t b, int64_t es) {
    int64_t ab = 0, abe = 0;
    if (a < 0 || b < 0 || __builtin_mul_overflow(a, b, &ab) || __builtin_mul_overflow(ab, es, &abe) ||
        abe > kMaxBytes)
        return -1;
    return abe;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Range {
    uintptr_t lo, hi;  // [lo, hi)
};

Range range_of(const void* p, int64_t bytes) {
    const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return Range{lo, lo + static_cast<uintptr_t>(bytes > 0 ? bytes : 0)};
}

bool overlap(Range a, Range b) {
    if (a.lo == a.hi || b.lo == b.hi) return false;  // empty ranges never overlap
    return a.lo < b.hi && b.lo < a.hi;
}

int64_t words_per_row(int64_t C) { return (C + 31) / 32; }

int64_t elt_size(int32_t dtype) { return dtype == LORS_DTYPE_BF16 ? 2 : 4; }

bool valid_dtype(int32_t d) { return d == LORS_DTYPE_BF16 || d == LORS_DTYPE_F32; }
bool valid_format(int32_t f) { return f == LORS_MASK_BITMAP || f == LORS_MASK_2_4; }

// Problem-level checks shared by forward/backward/workspace query, in the
// documented order (dtype/format, then shape/range).
lors_status_t check_problem(const lors_problem_t* p) {
    if (!valid_dtype(p->dtype)) return LORS_ERR_DTYPE;
    if (!valid_format(p->mask_format)) return LORS_ERR_MASK_FORMAT;
    if (p->R < 1 || p->C < 1 || p->L < 0 || p->r < 1 || p->r > kMaxRank) return LORS_ERR_SHAPE;
    if (p->R > kMaxExtent || p->C > kMaxExtent || p->L > kMaxExtent) return LORS_ERR_SHAPE;
    // every argument's byte count (fp32 outputs are 4 bytes per element
    // whatever the problem dtype) must be representable
    if (bytes_of(p->L, p->C, 4) < 0 || bytes_of(p->L, p->R, 4) < 0 || bytes_of(p->R, p->C, 4) < 0)
        return LORS_ERR_SHAPE;
    if (!std::isfinite(p->scale)) return LORS_ERR_SHAPE;
    if (p->mask_format == LORS_MASK_2_4 && (p->C % 4) != 0) return LORS_ERR_MASK_FORMAT;
    if ((p->flags & ~(LORS_FLAG_REUSE_MASK_T | LORS_FLAG_BWD_STE | LORS_FLAG_FWD_SPARSE_MFMA |
                      LORS_FLAG_SPLIT_LAST_WAVE)) != 0u)
        return LORS_ERR_UNSUPPORTED;
    // the structured-sparse forward exists for bf16 2:4 masks up to rank 64
    if ((p->flags & LORS_FLAG_FWD_SPARSE_MFMA) != 0u &&
        (p->dtype != LORS_DTYPE_BF16 || p->mask_format != LORS_MASK_2_4 || p->r > 64))
        return LORS_ERR_UNSUPPORTED;
    // the straight-through backward exists for bf16 only
    if ((p->flags & LORS_FLAG_BWD_STE) != 0u && p->dtype != LORS_DTYPE_BF16) return LORS_ERR_UNSUPPORTED;
    const int64_t row_align = p->dtype == LORS_DTYPE_BF16 ? 8 : 4;
    if (p->R % row_align != 0 || p->C % row_align != 0) return LORS_ERR_UNSUPPORTED;
    if (p->dtype == LORS_DTYPE_F32) {
        // The fp32 kernels put token tiles of 64 on the second grid axis.
        if ((p->L + 63) / 64 > 65535 || (p->R + 63) / 64 > 65535) return LORS_ERR_UNSUPPORTED;
    }
    // Tile counts of the bf16 kernels must fit a 32-bit grid.
    const int64_t t256 = ((p->L + 255) / 256) * ((p->R + 255) / 256);
    const int64_t t256x = ((p->L + 255) / 256) * ((p->C + 255) / 256);
    const int64_t t256g = ((p->R + 255) / 256) * ((p->C + 255) / 256);
    if (t256 > kMaxExtent || t256x > kMaxExtent || t256g > kMaxExtent) return LORS_ERR_UNSUPPORTED;
    return LORS_OK;
}

lors_status_t from_hip(hipError_t e) { return e == hipSuccess ? LORS_OK : LORS_ERR_HIP; }

}  // namespace

extern "C" {

const char* lors_status_string(int status) {
    switch (status) {
        case LORS_OK: return "LORS_OK";
        case LORS_ERR_NULL: return "LORS_ERR_NULL: a required pointer is NULL";
        case LORS_ERR_DTYPE: return "LORS_ERR_DTYPE: unknown dtype";
        case LORS_ERR_SHAPE: return "LORS_ERR_SHAPE: extent or rank out of range";
        case LORS_ERR_MASK_FORMAT: return "LORS_ERR_MASK_FORMAT: unknown mask format or 2:4 with C % 4 != 0";
        case LORS_ERR_ALIGN: return "LORS_ERR_ALIGN: pointer not 16-byte aligned";
        case LORS_ERR_ALIAS: return "LORS_ERR_ALIAS: an output overlaps an input or another output";
        case LORS_ERR_WORKSPACE: return "LORS_ERR_WORKSPACE: workspace too small";
        case LORS_ERR_UNSUPPORTED: return "LORS_ERR_UNSUPPORTED: valid but unsupported problem";
        case LORS_ERR_NOT_2_4: return "LORS_ERR_NOT_2_4: a group does not keep exactly 2 of 4";
        case LORS_ERR_HIP: return "LORS_ERR_HIP: HIP runtime or kernel launch failure";
        default: return "LORS: unknown status";
    }
}

int lors_version(void) { return 10100; }

size_t lors_mask_packed_bytes(int64_t R, int64_t C) {
    const int64_t n = (C < 0) ? -1 : bytes_of(R, words_per_row(C), 4);
    return n < 0 ? 0 : static_cast<size_t>(n);
}

// bf16 backward workspace, each part rounded up to 256 bytes: the
// transposed bitmap M^T (C rows of ceil(R/32) words); with the
// straight-through flag, the P, Q and B^T buffers of the re-associated
// adapter gradients; for ranks that are not a multiple of 8, a copy of B
// with its rows padded to roundup8(r) zero-filled columns, so that the dX
// kernel copies whole 16-byte chunks.  The forward and the fp32 path need
// nothing.
static size_t mt_bytes(const lors_problem_t* p) {
    const int64_t bytes = p->C * ((p->R + 31) / 32) * 4;
    return static_cast<size_t>((bytes + 255) / 256 * 256);
}
static size_t ste_bytes(const lors_problem_t* p) {
    return (p->flags & LORS_FLAG_BWD_STE) != 0u ? lors::ste_workspace_bytes(p->R, p->L, p->r) : 0;
}
static int64_t padded_rank(int64_t r) { return (r + 7) / 8 * 8; }
static size_t bpad_bytes(const lors_problem_t* p) {
    if (p->r % 8 == 0) return 0;
    return static_cast<size_t>((2 * p->R * padded_rank(p->r) + 255) / 256 * 256);
}
// Bytes the fp32 partial sums of split tiles may use.  With the transposed
// mask and the padded copy of B, the workspace then stays below R*C/4
// bytes, an eighth of the merged weight the layer never stores (the
// straight-through buffers, which grow with L, come on top).  When the
// budget is short the split uses fewer pieces, or none.
static int64_t split_budget(const lors_problem_t* p) {
    const int64_t b = p->R * p->C / 4 - static_cast<int64_t>(mt_bytes(p) + bpad_bytes(p)) - 256;
    return b > 0 ? b : 0;
}
// fp32 partial sums of the forward's or dX's split tiles (the larger of the
// two; the calls run one after the other), with LORS_FLAG_SPLIT_LAST_WAVE.
// Only shapes without whole tiles split over K: on whole-tile shapes the
// same short waves run as thin tiles, which need no partials.
static size_t split_bytes(const lors_problem_t* p) {
    if ((p->flags & LORS_FLAG_SPLIT_LAST_WAVE) == 0u || p->dtype != LORS_DTYPE_BF16 || p->L == 0) return 0;
    const int64_t tl = (p->L + 255) / 256;
    const int64_t budget = split_budget(p);
    int64_t fwd = 0, dx = 0;
    if (p->r <= 64 && (p->flags & LORS_FLAG_FWD_SPARSE_MFMA) == 0u && !lors::fwd_whole_tiles(p->L, p->R, p->C))
        fwd = lors::split_part_bytes(lors::tail_split(tl * ((p->R + 255) / 256), (p->C + 63) / 64, budget));
    if (padded_rank(p->r) <= 64 && !lors::dx_whole_tiles(p->L, p->R, p->C))
        dx = lors::split_part_bytes(lors::tail_split(tl * ((p->C + 255) / 256), (p->R + 63) / 64, budget));
    return static_cast<size_t>(fwd > dx ? fwd : dx);
}
size_t lors_workspace_bytes(const lors_problem_t* p) {
    if (p == nullptr || check_problem(p) != LORS_OK) return static_cast<size_t>(-1);
    if (p->dtype != LORS_DTYPE_BF16) return 0;
    return mt_bytes(p) + ste_bytes(p) + bpad_bytes(p) + split_bytes(p);
}
// The split partials sit after the transposed mask (and the other backward
// scratch), so a workspace shared by the forward and the backward calls
// keeps the transposed mask for LORS_FLAG_REUSE_MASK_T.
static void* split_region(const lors_problem_t* p, void* workspace) {
    if (workspace == nullptr || split_bytes(p) == 0) return nullptr;
    return static_cast<uint8_t*>(workspace) + mt_bytes(p) + ste_bytes(p) + bpad_bytes(p);
}

// ---------------------------------------------------------------------------
// masks
// ---------------------------------------------------------------------------

static lors_status_t check_mask_args(int64_t R, int64_t C, int32_t fmt) {
    if (!valid_format(fmt)) return LORS_ERR_MASK_FORMAT;
    if (R < 0 || C < 0 || R > kMaxExtent || C > kMaxExtent) return LORS_ERR_SHAPE;
    if (bytes_of(R, C, 4) < 0) return LORS_ERR_SHAPE;  // the dense mask and an fp32 weight
    if (fmt == LORS_MASK_2_4 && (C % 4) != 0) return LORS_ERR_MASK_FORMAT;
    return LORS_OK;
}

lors_status_t lors_mask_pack(const uint8_t* dense, int64_t R, int64_t C, int32_t mask_format,
                             uint32_t* packed, int64_t* first_bad, void* stream) {
    if (dense == nullptr || packed == nullptr) return LORS_ERR_NULL;
    if (mask_format == LORS_MASK_2_4 && first_bad == nullptr) return LORS_ERR_NULL;
    lors_status_t st = check_mask_args(R, C, mask_format);
    if (st != LORS_OK) return st;
    if (!aligned16(dense) || !aligned16(packed) || (first_bad && (reinterpret_cast<uintptr_t>(first_bad) & 7u)))
        return LORS_ERR_ALIGN;
    const Range out = range_of(packed, static_cast<int64_t>(lors_mask_packed_bytes(R, C)));
    if (overlap(out, range_of(dense, R * C)) ||
        (first_bad && (overlap(range_of(first_bad, 8), out) || overlap(range_of(first_bad, 8), range_of(dense, R * C)))))
        return LORS_ERR_ALIAS;
    return from_hip(lors::launch_mask_pack(dense, R, C, mask_format == LORS_MASK_2_4, packed, first_bad,
                                           static_cast<hipStream_t>(stream)));
}

lors_status_t lors_mask_unpack(const uint32_t* packed, int64_t R, int64_t C, int32_t mask_format,
                               uint8_t* dense, void* stream) {
    if (dense == nullptr || packed == nullptr) return LORS_ERR_NULL;
    lors_status_t st = check_mask_args(R, C, mask_format);
    if (st != LORS_OK) return st;
    if (!aligned16(dense) || !aligned16(packed)) return LORS_ERR_ALIGN;
    if (overlap(range_of(dense, R * C), range_of(packed, static_cast<int64_t>(lors_mask_packed_bytes(R, C)))))
        return LORS_ERR_ALIAS;
    return from_hip(lors::launch_mask_unpack(packed, R, C, mask_format == LORS_MASK_2_4, dense,
                                             static_cast<hipStream_t>(stream)));
}

lors_status_t lors_mask_from_weight(const void* W, int32_t dtype, int64_t R, int64_t C, int32_t mask_format,
                                    uint32_t* packed, int64_t* first_bad, void* stream) {
    if (W == nullptr || packed == nullptr) return LORS_ERR_NULL;
    if (mask_format == LORS_MASK_2_4 && first_bad == nullptr) return LORS_ERR_NULL;
    if (!valid_dtype(dtype)) return LORS_ERR_DTYPE;
    lors_status_t st = check_mask_args(R, C, mask_format);
    if (st != LORS_OK) return st;
    if (!aligned16(W) || !aligned16(packed) || (first_bad && (reinterpret_cast<uintptr_t>(first_bad) & 7u)))
        return LORS_ERR_ALIGN;
    const Range out = range_of(packed, static_cast<int64_t>(lors_mask_packed_bytes(R, C)));
    const Range w = range_of(W, R * C * elt_size(dtype));
    if (overlap(out, w) || (first_bad && (overlap(range_of(first_bad, 8), out) || overlap(range_of(first_bad, 8), w))))
        return LORS_ERR_ALIAS;
    return from_hip(lors::launch_mask_from_weight(W, dtype == LORS_DTYPE_BF16, R, C, mask_format == LORS_MASK_2_4,
                                                  packed, first_bad, static_cast<hipStream_t>(stream)));
}

lors_status_t lors_mask_pack_host(const uint8_t* dense, int64_t R, int64_t C, int32_t mask_format,
                                  uint32_t* packed, int64_t* first_bad) {
    if ((dense == nullptr || packed == nullptr) && R > 0 && C > 0) return LORS_ERR_NULL;
    lors_status_t st = check_mask_args(R, C, mask_format);
    if (st != LORS_OK) return st;
    const int64_t wpr = words_per_row(C);
    if (first_bad) *first_bad = -1;
    for (int64_t i = 0; i < R; ++i) {
        const uint8_t* row = dense + i * C;
        for (int64_t w = 0; w < wpr; ++w) {
            uint32_t word = 0;
            if (mask_format == LORS_MASK_BITMAP) {
                for (int64_t e = 0; e < 32 && 32 * w + e < C; ++e)
                    if (row[32 * w + e]) word |= 1u << e;
            } else {
                for (int64_t n = 0; n < 8; ++n) {
                    const int64_t g = 8 * w + n;
                    if (g >= C / 4) break;
                    int kept[4] = {0, 0, 0, 0};
                    int nk = 0;
                    for (int q = 0; q < 4; ++q)
                        if (row[4 * g + q]) kept[nk++] = q;
                    if (nk != 2) {
                        if (first_bad) *first_bad = i * (C / 4) + g;
                        return LORS_ERR_NOT_2_4;
                    }
                    word |= static_cast<uint32_t>(kept[0] | (kept[1] << 2)) << (4 * n);
                }
            }
            packed[i * wpr + w] = word;
        }
    }
    return LORS_OK;
}

lors_status_t lors_mask_unpack_host(const uint32_t* packed, int64_t R, int64_t C, int32_t mask_format,
                                    uint8_t* dense) {
    if ((dense == nullptr || packed == nullptr) && R > 0 && C > 0) return LORS_ERR_NULL;
    lors_status_t st = check_mask_args(R, C, mask_format);
    if (st != LORS_OK) return st;
    const int64_t wpr = words_per_row(C);
    for (int64_t i = 0; i < R; ++i) {
        for (int64_t j = 0; j < C; ++j) {
            const uint32_t word = packed[i * wpr + j / 32];
            uint8_t v;
            if (mask_format == LORS_MASK_BITMAP) {
                v = static_cast<uint8_t>((word >> (j % 32)) & 1u);
            } else {
                const uint32_t nib = (word >> (4 * ((j / 4) % 8))) & 0xFu;
                const uint32_t q = static_cast<uint32_t>(j % 4);
                v = static_cast<uint8_t>((nib & 3u) == q || (nib >> 2) == q);
            }
            dense[i * C + j] = v;
        }
    }
    return LORS_OK;
}

// ---------------------------------------------------------------------------
// forward / backward
// ---------------------------------------------------------------------------

lors_status_t lors_forward(const lors_problem_t* p, const void* X, const void* W, const uint32_t* M_packed,
                           const void* B, const void* A, const void* bias, void* Y, void* workspace,
                           size_t workspace_bytes, void* stream) {
    if (p == nullptr) return LORS_ERR_NULL;
    const bool tok = p->L != 0;  // with no tokens the activations may be NULL
    if ((tok && (X == nullptr || Y == nullptr)) || W == nullptr || M_packed == nullptr || B == nullptr ||
        A == nullptr)
        return LORS_ERR_NULL;
    lors_status_t st = check_problem(p);
    if (st != LORS_OK) return st;
    if (!aligned16(X) || !aligned16(W) || !aligned16(M_packed) || !aligned16(B) || !aligned16(A) ||
        !aligned16(Y) || (bias && !aligned16(bias)))
        return LORS_ERR_ALIGN;
    const int64_t es = elt_size(p->dtype);
    const int64_t R = p->R, C = p->C, L = p->L, r = p->r;
    const Range y = range_of(Y, L * R * es);
    const Range ins[] = {range_of(X, L * C * es), range_of(W, R * C * es),
                         range_of(M_packed, static_cast<int64_t>(lors_mask_packed_bytes(R, C))),
                         range_of(B, R * r * es), range_of(A, r * C * es),
                         bias ? range_of(bias, R * es) : Range{0, 0}};
    for (const Range& in : ins)
        if (overlap(y, in)) return LORS_ERR_ALIAS;
    // scratch only for the split partial sums (LORS_FLAG_SPLIT_LAST_WAVE)
    const size_t need = split_bytes(p) ? lors_workspace_bytes(p) : 0;
    if (need) {
        if (workspace == nullptr || workspace_bytes < need) return LORS_ERR_WORKSPACE;
        if (!aligned16(workspace)) return LORS_ERR_ALIGN;
        const Range w = range_of(workspace, static_cast<int64_t>(need));
        if (overlap(w, y)) return LORS_ERR_ALIAS;
        for (const Range& in : ins)
            if (overlap(w, in)) return LORS_ERR_ALIAS;
    }

    lors::LayerArgs a{};
    a.R = R; a.C = C; a.L = L; a.r = r;
    a.scale = p->scale;
    a.two_four = p->mask_format == LORS_MASK_2_4;
    a.sparse_mfma = (p->flags & LORS_FLAG_FWD_SPARSE_MFMA) != 0u;
    a.X = X; a.W = W; a.M = M_packed; a.B = B; a.A = A; a.bias = bias; a.Y = Y;
    a.split_ws = need ? split_region(p, workspace) : nullptr;
    a.split_budget = split_budget(p);
    hipStream_t s = static_cast<hipStream_t>(stream);
    return from_hip(p->dtype == LORS_DTYPE_BF16 ? lors::launch_fwd_bf16(a, s) : lors::launch_fwd_f32(a, s));
}

namespace {

// Shared validation of the three backward entry points.  Null pointers of
// optional outputs have been mapped to nullptr by the caller.
lors_status_t check_backward(const lors_problem_t* p, const void* dY, const void* X, const void* W,
                             const uint32_t* M_packed, const void* B, const void* A, void* dX, float* dB,
                             float* dA, float* dbias, const void* workspace, size_t workspace_bytes) {
    lors_status_t st = check_problem(p);
    if (st != LORS_OK) return st;
    const size_t need = lors_workspace_bytes(p);
    const void* all[] = {dY, X, W, M_packed, B, A, dX, dB, dA, dbias, need ? workspace : nullptr};
    for (const void* q : all)
        if (q && !aligned16(q)) return LORS_ERR_ALIGN;
    const int64_t es = elt_size(p->dtype);
    const int64_t R = p->R, C = p->C, L = p->L, r = p->r;
    const Range ins[] = {range_of(dY, L * R * es), X ? range_of(X, L * C * es) : Range{0, 0},
                         W ? range_of(W, R * C * es) : Range{0, 0},
                         range_of(M_packed, static_cast<int64_t>(lors_mask_packed_bytes(R, C))),
                         range_of(B, R * r * es), range_of(A, r * C * es)};
    const Range outs[] = {dX ? range_of(dX, L * C * es) : Range{0, 0}, dB ? range_of(dB, R * r * 4) : Range{0, 0},
                          dA ? range_of(dA, r * C * 4) : Range{0, 0}, dbias ? range_of(dbias, R * 4) : Range{0, 0},
                          (need && workspace) ? range_of(workspace, static_cast<int64_t>(need)) : Range{0, 0}};
    for (int o = 0; o < 5; ++o) {
        for (const Range& in : ins)
            if (overlap(outs[o], in)) return LORS_ERR_ALIAS;
        for (int o2 = o + 1; o2 < 5; ++o2)
            if (overlap(outs[o], outs[o2])) return LORS_ERR_ALIAS;
    }
    if (need && (workspace == nullptr || workspace_bytes < need)) return LORS_ERR_WORKSPACE;
    return LORS_OK;
}

lors::LayerArgs layer_args(const lors_problem_t* p, const void* dY, const void* X, const void* W,
                           const uint32_t* M_packed, const void* B, const void* A, void* dX, float* dB,
                           float* dA, float* dbias, void* workspace) {
    lors::LayerArgs a{};
    a.R = p->R; a.C = p->C; a.L = p->L; a.r = p->r;
    a.r_grad = p->r;
    a.scale = p->scale;
    a.two_four = p->mask_format == LORS_MASK_2_4;
    a.X = X; a.W = W; a.M = M_packed; a.B = B; a.A = A; a.dY = dY;
    a.dX = dX; a.dB = dB; a.dA = dA; a.dbias = dbias;
    a.Mt = (p->dtype == LORS_DTYPE_BF16) ? static_cast<const uint32_t*>(workspace) : nullptr;
    a.reuse_mt = (p->flags & LORS_FLAG_REUSE_MASK_T) != 0u;
    a.ste = (p->flags & LORS_FLAG_BWD_STE) != 0u;
    a.ste_ws = (a.ste && workspace) ? static_cast<uint8_t*>(workspace) + mt_bytes(p) : nullptr;
    a.b_pad = (p->dtype == LORS_DTYPE_BF16 && bpad_bytes(p) && workspace)
                  ? static_cast<uint8_t*>(workspace) + mt_bytes(p) + ste_bytes(p)
                  : nullptr;
    a.split_ws = split_region(p, workspace);
    a.split_budget = split_budget(p);
    return a;
}

// M^T into the workspace (bf16 problems with tokens only, unless the caller
// says the workspace already holds it).
hipError_t build_mt(const lors::LayerArgs& a, bool bf16, hipStream_t s) {
    if (!bf16 || a.L == 0 || a.reuse_mt) return hipSuccess;
    return lors::launch_mask_transpose(a.M, a.R, a.C, a.two_four, const_cast<uint32_t*>(a.Mt), s);
}

hipError_t run_weight(const lors::LayerArgs& a, bool bf16, hipStream_t s) {
    // the straight-through launches clear dB and dA themselves, and so does
    // the dX launch of the combined backward (a.clear_grads)
    hipError_t e = a.ste          ? lors::launch_ste_bf16(a, s)
                   : a.clear_grads ? hipSuccess
                                   : lors::launch_zero2_f32(a.dB, a.R * a.r, a.dA, a.r * a.C, s);
    if (e == hipSuccess && !a.ste) e = bf16 ? lors::launch_g_bf16(a, s) : lors::launch_g_f32(a, s);
    if (e == hipSuccess) e = bf16 ? lors::launch_dbias_bf16(a, s) : lors::launch_dbias_f32(a, s);
    return e;
}

}  // namespace

lors_status_t lors_backward(const lors_problem_t* p, const void* dY, const void* X, const void* W,
                            const uint32_t* M_packed, const void* B, const void* A, void* dX, float* dB,
                            float* dA, float* dbias, void* workspace, size_t workspace_bytes, void* stream) {
    if (p == nullptr) return LORS_ERR_NULL;
    const bool tok = p->L != 0;
    if ((tok && (dY == nullptr || X == nullptr)) || W == nullptr || M_packed == nullptr || B == nullptr ||
        A == nullptr || dB == nullptr || dA == nullptr)
        return LORS_ERR_NULL;
    lors_status_t st = check_backward(p, dY, X, W, M_packed, B, A, dX, dB, dA, dbias, workspace, workspace_bytes);
    if (st != LORS_OK) return st;
    lors::LayerArgs a = layer_args(p, dY, X, W, M_packed, B, A, dX, dB, dA, dbias, workspace);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool bf16 = p->dtype == LORS_DTYPE_BF16;
    // the bf16 dX kernel clears dB and dA for the weight gradient's atomics,
    // which saves the separate clearing launch
    a.clear_grads = bf16 && !a.ste && dX != nullptr && tok;
    hipError_t e = build_mt(a, bf16, s);
    if (e == hipSuccess && dX) e = bf16 ? lors::launch_dx_bf16(a, s) : lors::launch_dx_f32(a, s);
    if (e == hipSuccess) e = run_weight(a, bf16, s);
    return from_hip(e);
}

lors_status_t lors_backward_data(const lors_problem_t* p, const void* dY, const void* W, const uint32_t* M_packed,
                                 const void* B, const void* A, void* dX, void* workspace, size_t workspace_bytes,
                                 void* stream) {
    if (p == nullptr) return LORS_ERR_NULL;
    const bool tok = p->L != 0;
    if ((tok && (dY == nullptr || dX == nullptr)) || W == nullptr || M_packed == nullptr || B == nullptr ||
        A == nullptr)
        return LORS_ERR_NULL;
    lors_status_t st = check_backward(p, dY, nullptr, W, M_packed, B, A, dX, nullptr, nullptr, nullptr, workspace,
                                      workspace_bytes);
    if (st != LORS_OK) return st;
    const lors::LayerArgs a = layer_args(p, dY, nullptr, W, M_packed, B, A, dX, nullptr, nullptr, nullptr, workspace);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool bf16 = p->dtype == LORS_DTYPE_BF16;
    hipError_t e = build_mt(a, bf16, s);
    if (e == hipSuccess) e = bf16 ? lors::launch_dx_bf16(a, s) : lors::launch_dx_f32(a, s);
    return from_hip(e);
}

lors_status_t lors_backward_weight(const lors_problem_t* p, const void* dY, const void* X, const uint32_t* M_packed,
                                   const void* B, const void* A, float* dB, float* dA, float* dbias, void* workspace,
                                   size_t workspace_bytes, void* stream) {
    if (p == nullptr) return LORS_ERR_NULL;
    const bool tok = p->L != 0;
    if ((tok && (dY == nullptr || X == nullptr)) || M_packed == nullptr || B == nullptr || A == nullptr ||
        dB == nullptr || dA == nullptr)
        return LORS_ERR_NULL;
    lors_status_t st = check_backward(p, dY, X, nullptr, M_packed, B, A, nullptr, dB, dA, dbias, workspace,
                                      workspace_bytes);
    if (st != LORS_OK) return st;
    const lors::LayerArgs a = layer_args(p, dY, X, nullptr, M_packed, B, A, nullptr, dB, dA, dbias, workspace);
    const bool bf16 = p->dtype == LORS_DTYPE_BF16;
    hipStream_t s = static_cast<hipStream_t>(stream);
    // the straight-through adapter gradients do not read the mask
    hipError_t e = a.ste ? hipSuccess : build_mt(a, bf16, s);
    if (e == hipSuccess) e = run_weight(a, bf16, s);
    return from_hip(e);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// The backward without a caller-provided workspace, for callers that cannot
// allocate device memory.  Its scratch is one file-scope device array per
// GPU, shared by every call on that GPU.
// ---------------------------------------------------------------------------
namespace {

static __device__ __align__(256) uint8_t scratch[LORS_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_of[kMaxDevices];  // device address of `scratch` per device, once looked up

// The device whose queue `stream` feeds (the current device for the null
// stream), and that device's address of `scratch`.  In host code the
// array's name stands for a host-side shadow, not device memory, so the
// device address is looked up -- once per device, with that device current --
// and only that address is handed to kernels.
hipError_t scratch_of_stream(hipStream_t stream, void** out) {
    int dev = 0;
    hipError_t e = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_of[dev] == nullptr) {
        int cur = -1;
        if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev) {
            const hipError_t e2 = hipSetDevice(cur);
            if (e == hipSuccess) e = e2;
        }
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        g_scratch_of[dev] = p;
    }
    *out = g_scratch_of[dev];
    return hipSuccess;
}

}  // namespace

extern "C" lors_status_t lors_backward_noalloc(const lors_problem_t* p, const void* dY, const void* X,
                                               const void* W, const uint32_t* M_packed, const void* B,
                                               const void* A, void* dX, float* dB, float* dA, float* dbias,
                                               void* stream) {
    if (p == nullptr) return LORS_ERR_NULL;
    const bool tok = p->L != 0;
    if ((tok && (dY == nullptr || X == nullptr)) || W == nullptr || M_packed == nullptr || B == nullptr ||
        A == nullptr || dB == nullptr || dA == nullptr)
        return LORS_ERR_NULL;
    lors_status_t st = check_backward(p, dY, X, W, M_packed, B, A, dX, dB, dA, dbias, nullptr, 0);
    // the only failure that a workspace would have avoided: the scratch size
    if (st == LORS_ERR_WORKSPACE) st = LORS_OK;
    if (st != LORS_OK) return st;
    // the scratch keeps the previous call's contents, whoever made it
    if ((p->flags & LORS_FLAG_REUSE_MASK_T) != 0u) return LORS_ERR_UNSUPPORTED;
    const size_t need = lors_workspace_bytes(p);
    if (need > LORS_NOALLOC_SCRATCH_BYTES) return LORS_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    void* ws = nullptr;
    if (need > 0) {
        const hipError_t e = scratch_of_stream(s, &ws);
        if (e != hipSuccess) return LORS_ERR_HIP;
    }
    lors::LayerArgs a = layer_args(p, dY, X, W, M_packed, B, A, dX, dB, dA, dbias, ws);
    const bool bf16 = p->dtype == LORS_DTYPE_BF16;
    a.clear_grads = bf16 && !a.ste && dX != nullptr && tok;
    hipError_t e = build_mt(a, bf16, s);
    if (e == hipSuccess && dX) e = bf16 ? lors::launch_dx_bf16(a, s) : lors::launch_dx_f32(a, s);
    if (e == hipSuccess) e = run_weight(a, bf16, s);
    return from_hip(e);
}
