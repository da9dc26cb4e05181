"""The library's rules for a short last wave of output tiles (as documented in
include/lors.h), restated for the tests: on whole-tile shapes its tiles are
cut over their tokens into thin tiles; on other shapes, with
LORS_FLAG_SPLIT_LAST_WAVE, they are split over K -- which shapes split, into
how many pieces, and which output tiles run in pieces."""


def up256(n):
    return -(-n // 256) * 256


def split_budget(R, C, r):
    """Bytes the split partials may use: the workspace (transposed mask,
    padded copy of B, partials) stays below R*C/4."""
    mt = up256(C * -(-R // 32) * 4)
    bpad = up256(2 * R * (-(-r // 8) * 8)) if r % 8 else 0
    return max(0, R * C // 4 - mt - bpad - 256)


def pieces(tiles, nk, budget, cus=256):
    """Pieces per tile of the short last wave (1: no split)."""
    tail = tiles % cus
    if tail == 0 or 2 * tail > cus:
        return 1
    s = min(8, cus // tail, nk // 4, budget // (tail * 256 * 256 * 4))
    return s if s >= 2 else 1


def split_bytes(tiles, nk, budget, cus=256):
    s = pieces(tiles, nk, budget, cus)
    return (tiles % cus) * s * 256 * 256 * 4 if s > 1 else 0


def split_tiles(rows, cols, cus=256, group_m=4):
    """(row0, col0) of the output tiles that run in pieces, given that the
    grid splits: the logical tiles past the whole waves, mapped to tiles in
    the kernels' grouped order (group_m tile rows at a time, column-major
    inside a group)."""
    tm_n, tn_n = -(-rows // 256), -(-cols // 256)
    tiles = tm_n * tn_n
    out = []
    for t in range(tiles - tiles % cus, tiles):
        per_group = group_m * tn_n
        g = t // per_group
        first = g * group_m
        gsz = min(tm_n - first, group_m)
        within = t - g * per_group
        out.append((256 * (first + within % gsz), 256 * (within // gsz)))
    return out


def fwd_whole_tiles(L, R, C):
    """The forward's fixed-offset copies: whole 256 x 256 tiles over L x R,
    64-wide K-steps over C, 256 slab rows of C bf16 addressed in 32 bits."""
    return L % 256 == 0 and R % 256 == 0 and C % 64 == 0 and 256 * C * 2 < 2**31


def dx_whole_tiles(L, R, C):
    """The same for dX: tiles over L x C, K-steps over R."""
    return L % 256 == 0 and C % 256 == 0 and R % 64 == 0 and 256 * R * 2 < 2**31 and 64 * C * 2 < 2**31


def thin_q(tiles, cus=256):
    """Thin tiles per tile of the short last wave (1: not cut): the largest
    of 2, 4, 8 whose thin tiles fit on the CUs."""
    tail = tiles % cus
    if tail == 0 or 2 * tail > cus:
        return 1
    q = 2
    while q < 8 and 2 * q * tail <= cus:
        q *= 2
    return q
