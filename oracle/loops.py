"""Pure-Python loop twin of the oracle, for tiny shapes (test infrastructure only).

Each output element is written as its own sum, straight from the element-wise
definition of the masked merged weight (Eq. 3, Section 2.2) and of the exact
gradients (SP-LoRA backward, Section 2.2), with the scale of the Appendix A
listing.  It uses no numpy arithmetic at all: inputs are converted to nested
Python float lists first.
"""
from __future__ import annotations


def _lst(a):
    return [[float(v) for v in row] for row in a.tolist()] if hasattr(a, "tolist") else a


def merged(W, M, B, A, s):
    W, M, B, A = _lst(W), _lst(M), _lst(B), _lst(A)
    R, C, r = len(W), len(W[0]), len(A)
    out = [[0.0] * C for _ in range(R)]
    for i in range(R):
        for j in range(C):
            if M[i][j]:
                acc = 0.0
                for k in range(r):
                    acc += B[i][k] * A[k][j]
                out[i][j] = W[i][j] + s * acc
    return out


def forward(X, W, M, B, A, s, bias=None):
    X = _lst(X)
    Wp = merged(W, M, B, A, s)
    L, R, C = len(X), len(Wp), len(X[0]) if X else 0
    Y = [[0.0] * R for _ in range(L)]
    for t in range(L):
        for i in range(R):
            acc = 0.0
            for j in range(C):
                acc += X[t][j] * Wp[i][j]
            Y[t][i] = acc + (float(bias[i]) if bias is not None else 0.0)
    return Y


def backward(dY, X, W, M, B, A, s):
    dY, X, Mm, Bm, Am = _lst(dY), _lst(X), _lst(M), _lst(B), _lst(A)
    Wp = merged(W, M, B, A, s)
    L, R, C, r = len(dY), len(Wp), len(Wp[0]), len(Am)
    dX = [[0.0] * C for _ in range(L)]
    for t in range(L):
        for j in range(C):
            acc = 0.0
            for i in range(R):
                acc += dY[t][i] * Wp[i][j]
            dX[t][j] = acc
    G = [[0.0] * C for _ in range(R)]
    for i in range(R):
        for j in range(C):
            if Mm[i][j]:
                acc = 0.0
                for t in range(L):
                    acc += dY[t][i] * X[t][j]
                G[i][j] = acc
    dB = [[0.0] * r for _ in range(R)]
    for i in range(R):
        for k in range(r):
            acc = 0.0
            for j in range(C):
                acc += G[i][j] * Am[k][j]
            dB[i][k] = s * acc
    dA = [[0.0] * C for _ in range(r)]
    for k in range(r):
        for j in range(C):
            acc = 0.0
            for i in range(R):
                acc += Bm[i][k] * G[i][j]
            dA[k][j] = s * acc
    dbias = [sum(dY[t][i] for t in range(L)) for i in range(R)]
    return dX, dB, dA, dbias


def pack_bitmap(M):
    """Pure-Python bitmap packer: bit j%32 of word i*ceil(C/32) + j//32."""
    M = _lst(M)
    R, C = len(M), len(M[0]) if M else 0
    wpr = (C + 31) // 32
    words = [0] * (R * wpr)
    for i in range(R):
        for j in range(C):
            if M[i][j]:
                words[i * wpr + j // 32] |= 1 << (j % 32)
    return words


def pack_2_4(M):
    """Pure-Python 2:4 packer: nibble p0 | p1 << 2 of group g at bits 4*(g%8)."""
    M = _lst(M)
    R, C = len(M), len(M[0]) if M else 0
    wpr = (C + 31) // 32
    words = [0] * (R * wpr)
    for i in range(R):
        for g in range(C // 4):
            kept = [p for p in range(4) if M[i][4 * g + p]]
            if len(kept) != 2:
                raise ValueError(f"row {i} group {g} keeps {len(kept)} of 4")
            nib = kept[0] | (kept[1] << 2)
            words[i * wpr + g // 8] |= nib << (4 * (g % 8))
    return words
