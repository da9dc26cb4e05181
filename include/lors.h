/*
 * lors.h -- C ABI of the sparsity-preserved LoRA linear for AMD MI355X (gfx950).
 *
 * The layer (LoRS, arXiv 2501.08582) fine-tunes a pruned weight W with a
 * rank-r adapter while keeping W's sparsity pattern M:
 *
 *   forward   Y  = X . W'^T (+ bias),   W' = select(M, W + s.B.A, 0)
 *   backward  dX = dY . W'                          (W' recomputed, never stored)
 *             G  = select(M, dY^T . X, 0)           (never stored)
 *             dB = s . G . A^T,   dA = s . B^T . G,  dbias = sum_tokens dY
 *
 * Sources: the SP-LoRA forward and backward step lists of Section 2.2 (Eq. 3),
 * weight recompute of Section 2.3 (Algorithms 1 and 2), the scale factor and
 * saved context of the Appendix A LoRS listing.  Readings taken where the
 * paper is silent: s multiplies both adapter gradients (it is the exact
 * derivative of the forward); the mask multiplies the whole sum W + s.B.A;
 * masking is a select, so masked entries are +0; the mask stays on the weight
 * gradient (exact gradient).  The paper's straight-through, re-associated
 * backward (Section 2.3) is the LORS_FLAG_BWD_STE variant, and a 2:4 forward
 * on the structured-sparse MFMA is the LORS_FLAG_FWD_SPARSE_MFMA variant.
 *
 * Names: B is R x r and A is r x C.  The paper calls the R x r adapter
 * (calligraphic) A and the r x C adapter (calligraphic) B; this header uses
 * the opposite, PEFT-style names.  The paper stores tokens as columns
 * (X is C x L); here tokens are rows.
 *
 * Shapes and layouts -- every array is row-major and contiguous, and every
 * pointer is 16-byte aligned:
 *   X  L x C   W  R x C   B  R x r   A  r x C   bias R
 *   Y, dY  L x R          dX  L x C
 *   dB  R x r (float32)   dA  r x C (float32)    dbias  R (float32)
 *   packed mask  R x ceil(C/32) uint32 words (layouts below)
 * The problem dtype (bf16 or fp32) applies to X, W, B, A, bias, Y, dY, dX.
 * L (tokens) is the product of all leading dimensions of the activation.
 *
 * Arithmetic (bf16): W + s.B.A is formed in fp32 from the bf16 operands and
 * rounded once to bf16 (nearest-even) before the main product; all products
 * accumulate in fp32; Y and dX are rounded to bf16 (nearest-even); G is
 * rounded to bf16 before the two rank-r products; dA, dB, dbias stay fp32.
 * For 64 < r <= 128 the forward and dX use that the mask
 * distributes over the adapter's rank blocks: Y (and dX) is the bf16 sum of
 * the product with select(M, W + s.B[:, :64].A[:64, :]) and the product with
 * select(M, s.B[:, 64:].A[64:, :]), each merged weight rounded once, so Y and
 * dX take one more bf16 rounding.
 * The fp32 dtype keeps every intermediate in fp32 (a debug/reference path).
 *
 * Ownership: the caller owns every buffer.  The library never allocates
 * device memory; its scratch needs are reported by lors_workspace_bytes.
 * Pointers must stay valid until the work queued on `stream` completes; the
 * library keeps nothing after a call returns.  Inputs are read only.  Outputs
 * are overwritten, never accumulated into, and must not overlap any input or
 * each other (LORS_ERR_ALIAS).  `stream` is a hipStream_t (NULL = default).
 *
 * Errors: every entry point returns a lors_status_t; nothing prints, throws or
 * aborts.  Arguments are validated on the host in the order
 *   null -> dtype/format -> shape/range -> alignment -> alias -> workspace
 * before any HIP call, so a rejected call has no side effect.  With L == 0
 * the token-sized arrays (X, Y, dY, dX) may be NULL.  Kernel-launch
 * failures return LORS_ERR_HIP.  Compute calls are asynchronous on `stream`.
 */
#ifndef LORS_H
#define LORS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum lors_status {
    LORS_OK = 0,
    LORS_ERR_NULL = 1,          /* a required pointer is NULL */
    LORS_ERR_DTYPE = 2,         /* unknown dtype */
    LORS_ERR_SHAPE = 3,         /* negative/zero extent where not allowed, r out of range */
    LORS_ERR_MASK_FORMAT = 4,   /* unknown mask format, or 2:4 with C % 4 != 0 */
    LORS_ERR_ALIGN = 5,         /* a pointer is not 16-byte aligned */
    LORS_ERR_ALIAS = 6,         /* an output overlaps an input or another output */
    LORS_ERR_WORKSPACE = 7,     /* workspace smaller than lors_workspace_bytes */
    LORS_ERR_UNSUPPORTED = 8,   /* valid but unsupported: see lors_problem_t */
    LORS_ERR_NOT_2_4 = 9,       /* host packer: a group does not keep exactly 2 of 4 */
    LORS_ERR_HIP = 10           /* a HIP runtime call or kernel launch failed */
} lors_status_t;

typedef enum lors_dtype {
    LORS_DTYPE_BF16 = 0,
    LORS_DTYPE_F32 = 1
} lors_dtype_t;

/*
 * Packed mask layouts (the paper keeps M as a dense boolean, `weight != 0`;
 * the packing is this library's own).  Both use ceil(C/32) uint32 words per
 * row, i.e. C/8 bytes per row when C % 32 == 0.
 *   LORS_MASK_BITMAP: element (i, j) is bit j % 32 (least significant first)
 *     of word i*ceil(C/32) + j/32.  Padding bits past C must be 0.
 *   LORS_MASK_2_4: needs C % 4 == 0.  Group g of row i (columns 4g..4g+3)
 *     keeps exactly two positions p0 < p1 and stores the nibble p0 | p1 << 2
 *     at bits 4*(g % 8) of word i*ceil(C/32) + g/8.  Unused nibbles are 0.
 */
typedef enum lors_mask_format {
    LORS_MASK_BITMAP = 0,
    LORS_MASK_2_4 = 1
} lors_mask_format_t;

/* Backward calls: the straight-through, re-associated adapter gradients of
 * Section 2.3 (Algorithm 2) instead of the exact masked ones.  The mask is
 * dropped from the weight gradient, which then never forms:
 *   P = X . A^T, Q = dY . B (L x r, bf16 in the workspace),
 *   dB = s . dY^T . P, dA = s . Q^T . X.
 * dX is unchanged (exact, with the recomputed masked weight).  bf16 only
 * (fp32: LORS_ERR_UNSUPPORTED).  The workspace grows by the P, Q and B^T
 * buffers (lors_workspace_bytes accounts for them). */
#define LORS_FLAG_BWD_STE 0x1u

/* Backward calls only: the workspace already holds the transposed mask that
 * an earlier backward call wrote for the same M_packed, R and C (its
 * contents were not touched since), so it is not rebuilt.  The mask of a
 * sparse layer is frozen during fine-tuning, so a training loop can pass
 * this flag from the second step on, or between lors_backward_data and
 * lors_backward_weight of one step. */
#define LORS_FLAG_REUSE_MASK_T 0x2u

/* Forward only: with a 2:4 mask, multiply on gfx950's structured-sparse MFMA
 * (the 2:4 pattern of Section 3.1): each merged W' tile is compressed in
 * registers to its two kept values per group of 4, indexed by the packed
 * mask codes, so the matrix cores do half the work of the dense product.
 * Same result as the dense forward up to rounding order.  bf16, 2:4 masks
 * and r <= 64 only (otherwise LORS_ERR_UNSUPPORTED).  Not the default: the
 * fused forward is bound by its merge and operand traffic rather than by
 * the matrix cores, so it is not faster today. */
#define LORS_FLAG_FWD_SPARSE_MFMA 0x4u

/* Forward and backward calls: when the forward's or dX's grid of 256 x 256
 * output tiles ends in a partial wave that fills at most half of the GPU's
 * compute units (e.g. 320 tiles on 256 CUs), that wave is spread over more
 * CUs.  On shapes of whole tiles (L and the output features multiples of
 * 256, the contraction a multiple of 64) this happens with or without the
 * flag and needs no workspace: each tile of the wave is cut over its tokens
 * into 2, 4 or 8 thin tiles, which compute the same bits as the whole tile.
 * On other shapes, with this flag, the tiles of that wave are cut
 * along their contraction (K) into up to 8 pieces, one per CU.  Each piece
 * writes its fp32 partial sums (256 KiB) to the workspace; a small reduction
 * launch adds a tile's pieces in a fixed order, adds the bias and rounds
 * once to bf16, so results stay bitwise reproducible.  The partials are
 * bounded so that the whole workspace (transposed mask, padded B copy and
 * partials) stays below R*C/4 bytes, an eighth of the bf16 merged weight
 * the layer exists not to store: when that budget cannot hold two pieces of
 * every tile of the short wave, fewer pieces are used, or none (the call
 * then runs as without the flag).  lors_workspace_bytes accounts for the
 * partials, and lors_forward requires a workspace when there are any.  No
 * effect for fp32; applies to ranks up to 64 (above, the layer already runs
 * as two passes).  The weight gradient always splits such a wave, with no
 * workspace: its pieces' partial G tiles go through the same rank-r products
 * and atomics as whole tiles. */
#define LORS_FLAG_SPLIT_LAST_WAVE 0x8u

/*
 * Problem description.
 *   R (out features) >= 1, C (in features) >= 1, L (tokens) >= 0,
 *   1 <= r <= 128, every extent < 2^31, scale finite, and every argument's
 *   byte count (products L*C, L*R, R*C times 4) at most 2^60; otherwise
 *   LORS_ERR_SHAPE.
 *   bf16: R % 8 == 0 and C % 8 == 0;  fp32: R % 4 == 0 and C % 4 == 0
 *   (16-byte rows); otherwise LORS_ERR_UNSUPPORTED.
 */
typedef struct lors_problem {
    int64_t R;
    int64_t C;
    int64_t L;
    int64_t r;
    float scale;
    int32_t dtype;        /* lors_dtype_t */
    int32_t mask_format;  /* lors_mask_format_t */
    uint32_t flags;       /* 0 or LORS_FLAG_* bits (REUSE_MASK_T, BWD_STE, FWD_SPARSE_MFMA,
                             SPLIT_LAST_WAVE) */
} lors_problem_t;

/* Human-readable name of a status code (static storage). */
const char* lors_status_string(int status);

/* ABI version: major * 10000 + minor * 100 + patch. */
int lors_version(void);

/* Bytes of a packed R x C mask (either layout): 4 * R * ceil(C/32). */
size_t lors_mask_packed_bytes(int64_t R, int64_t C);

/*
 * Device mask packing.  `dense` is an R x C uint8 device array (nonzero =
 * kept); `packed` receives lors_mask_packed_bytes(R, C) bytes.  For
 * LORS_MASK_2_4, `first_bad` (device, one int64) is required and receives the
 * linear index i*(C/4)+g of the first group that does not keep exactly two
 * entries, or -1 if every group is valid; for the bitmap it may be NULL (it is
 * then left untouched) or receives -1.  Asynchronous on `stream`: the call
 * returns LORS_OK once the work is queued and never LORS_ERR_NOT_2_4; the
 * caller reads *first_bad after the stream work completes.  When it is >= 0
 * the packed words are unspecified (an invalid group is not representable
 * in the 2:4 layout) and must not be passed to the compute calls.
 * The mask M is the one of Section 2.1 and Algorithm 1 (kept = nonzero).
 */
lors_status_t lors_mask_pack(const uint8_t* dense, int64_t R, int64_t C,
                             int32_t mask_format, uint32_t* packed,
                             int64_t* first_bad, void* stream);

/* Device unpacking: packed -> dense uint8 0/1 (R x C).  Asynchronous. */
lors_status_t lors_mask_unpack(const uint32_t* packed, int64_t R, int64_t C,
                               int32_t mask_format, uint8_t* dense, void* stream);

/*
 * Device mask derivation M = (W != 0) from the weight itself, as the paper's
 * algorithms and listing do (`weight != 0`); -0 counts as zero and NaN as
 * nonzero (IEEE comparison).  W has dtype `dtype`.  `first_bad` as for
 * lors_mask_pack, with the same asynchronous contract.
 */
lors_status_t lors_mask_from_weight(const void* W, int32_t dtype, int64_t R,
                                    int64_t C, int32_t mask_format,
                                    uint32_t* packed, int64_t* first_bad,
                                    void* stream);

/* Host twins of lors_mask_pack / lors_mask_unpack on host memory.  The
 * packer returns LORS_ERR_NOT_2_4 (and *first_bad, if non-NULL, the group
 * index) for an invalid 2:4 mask; `packed` is then unspecified. */
lors_status_t lors_mask_pack_host(const uint8_t* dense, int64_t R, int64_t C,
                                  int32_t mask_format, uint32_t* packed,
                                  int64_t* first_bad);
lors_status_t lors_mask_unpack_host(const uint32_t* packed, int64_t R, int64_t C,
                                    int32_t mask_format, uint8_t* dense);

/* Device scratch bytes the backward calls (lors_backward, lors_backward_data,
 * lors_backward_weight) need for problem p: for bf16 the transposed bitmap of
 * the mask, 4 * C * ceil(R/32) bytes rounded up to 256 (about R*C/8, i.e.
 * 1/16 of W), plus with LORS_FLAG_BWD_STE the P and Q buffers (2*L*rp
 * bytes each, rp = r rounded up to a multiple of 32) and B^T (2*r*R bytes),
 * plus, when r is not a multiple of 8, a copy of B whose rows are padded with
 * zeros to r8 = r rounded up to a multiple of 8 (2*R*r8 bytes), plus with
 * LORS_FLAG_SPLIT_LAST_WAVE the fp32 partial sums of split tiles (forward and
 * dX; the forward uses only this last part, so a workspace shared by all
 * calls keeps the transposed mask), each part rounded up to 256; 0 for fp32.
 * Without the straight-through flag the total stays below R*C/4 whenever the
 * transposed mask and the padded B alone do (every shape with R*C >= 64 R r8).
 * (size_t)-1 if p is invalid.  The workspace must be
 * 16-byte aligned, must not overlap any argument, and is overwritten; its
 * contents on return are unspecified.  lors_forward needs one only with
 * LORS_FLAG_SPLIT_LAST_WAVE. */
size_t lors_workspace_bytes(const lors_problem_t* p);

/*
 * Forward: Y = X . W'^T (+ bias), W' = select(M, W + s.B.A, 0)
 * (Eq. 3 and Algorithm 1; W' exists only tile by tile in on-chip memory).
 * `bias` may be NULL.  Inputs X, W, M_packed, B, A are what a training
 * framework keeps for the backward (the listing saves x and the parameters;
 * W' and a dense mask are not kept).
 */
lors_status_t lors_forward(const lors_problem_t* p, const void* X,
                           const void* W, const uint32_t* M_packed,
                           const void* B, const void* A, const void* bias,
                           void* Y, void* workspace, size_t workspace_bytes,
                           void* stream);

/*
 * Backward (SP-LoRA backward list of Section 2.2 with the weight recompute of
 * Algorithm 2): dX = dY . W' (skipped if dX is NULL), G = select(M, dY^T.X, 0),
 * dB = s.G.A^T, dA = s.B^T.G, dbias = column sums of dY (skipped if NULL).
 * dB, dA, dbias are fp32 and are overwritten.  Their summation order across
 * tiles is not fixed (fp32 atomics), so they can differ run to run in the
 * last bits; dX is bitwise reproducible.
 */
lors_status_t lors_backward(const lors_problem_t* p, const void* dY,
                            const void* X, const void* W,
                            const uint32_t* M_packed, const void* B,
                            const void* A, void* dX, float* dB, float* dA,
                            float* dbias, void* workspace,
                            size_t workspace_bytes, void* stream);

/*
 * The two halves of lors_backward as separate calls, for callers that need
 * only one of them (a frozen first layer needs no dX; frozen adapters need no
 * dB/dA) or that schedule them on different streams.  Arguments, layouts and
 * errors as for lors_backward; dX is required by lors_backward_data, dB and
 * dA by lors_backward_weight.
 *   lors_backward_data:   dX = dY . W'  (W' recomputed tile by tile;
 *                         the dX step of Section 2.2, Algorithm 2)
 *   lors_backward_weight: G = select(M, dY^T.X, 0) (I_w^4, I_w^5 of Section
 *                         2.2), dB = s.G.A^T, dA = s.B^T.G, dbias
 */
lors_status_t lors_backward_data(const lors_problem_t* p, const void* dY,
                                 const void* W, const uint32_t* M_packed,
                                 const void* B, const void* A, void* dX,
                                 void* workspace, size_t workspace_bytes,
                                 void* stream);
lors_status_t lors_backward_weight(const lors_problem_t* p, const void* dY,
                                   const void* X, const uint32_t* M_packed,
                                   const void* B, const void* A, float* dB,
                                   float* dA, float* dbias, void* workspace,
                                   size_t workspace_bytes, void* stream);

/*
 * lors_backward without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same computation, arguments (less
 * the workspace), layouts, results and errors as lors_backward, with its
 * scratch in a file-scope device array of LORS_NOALLOC_SCRATCH_BYTES that
 * each GPU the library runs on holds from the library's first use on it until
 * the process ends.  The call allocates nothing (no hipMalloc, no allocating
 * library routine); the caller still passes every input and output.
 *   - Problems whose lors_workspace_bytes exceeds LORS_NOALLOC_SCRATCH_BYTES
 *     return LORS_ERR_WORKSPACE (validation happens on the host first, as
 *     for every entry point).
 *   - Every call on one GPU shares that GPU's array, which keeps the last
 *     call's contents: LORS_FLAG_REUSE_MASK_T is refused
 *     (LORS_ERR_UNSUPPORTED), the transposed mask is rebuilt on every call,
 *     and nothing in the array needs to start at zero.  Calls that overlap
 *     in time on one GPU (different streams or host threads) race on the
 *     array: serialise them.
 *   - The array is the one of the device `stream` belongs to (the current
 *     device for the null stream); its device address is looked up once per
 *     device, on the first call there (LORS_ERR_HIP if that fails).
 */
#define LORS_NOALLOC_SCRATCH_BYTES (32u << 20)
lors_status_t lors_backward_noalloc(const lors_problem_t* p, const void* dY,
                                    const void* X, const void* W,
                                    const uint32_t* M_packed, const void* B,
                                    const void* A, void* dX, float* dB,
                                    float* dA, float* dbias, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LORS_H */
