"""Pure-Python brute force for tiny shapes -- TEST INFRASTRUCTURE.

A second, independent spelling of the convolution of Sec. 2.1 in plain Python
integers (no numpy arithmetic, no C), used to cross-check the C oracle's
indexing and its ctypes marshalling on tiny inputs.  It builds the lowered
(im2col) matrix of Sec. 2.1 explicitly -- one row per output pixel holding the
R*S*C window values, padding as zero -- and multiplies it by the filter
matrix, which is the other way of writing the same sum.
"""
from __future__ import annotations


def lowered_rows(x, n, h, w, c, r, s, sh, sw, ph, pw):
    """im2col of an N x H x W x C nested-list tensor: list of (N*P*Q) rows of R*S*C values."""
    p = (h + 2 * ph - r) // sh + 1
    q = (w + 2 * pw - s) // sw + 1
    rows = []
    for ni in range(n):
        for pi in range(p):
            for qi in range(q):
                row = []
                for ri in range(r):
                    for si in range(s):
                        yy, xx = pi * sh - ph + ri, qi * sw - pw + si
                        inside = 0 <= yy < h and 0 <= xx < w
                        for ci in range(c):
                            row.append(x[ni][yy][xx][ci] if inside else 0)
                rows.append(row)
    return rows, p, q


def conv2d(x, wt, stride=(1, 1), pad=(0, 0)):
    """x: N x H x W x C nested lists of ints; wt: K x R x S x C.  Returns N x P x Q x K."""
    n, h, w, c = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    k, r, s = len(wt), len(wt[0]), len(wt[0][0])
    rows, p, q = lowered_rows(x, n, h, w, c, r, s, stride[0], stride[1], pad[0], pad[1])
    cols = [[wt[ko][ri][si][ci] for ri in range(r) for si in range(s) for ci in range(c)] for ko in range(k)]
    out = [[[[0] * k for _ in range(q)] for _ in range(p)] for _ in range(n)]
    for m, row in enumerate(rows):
        ni, rem = divmod(m, p * q)
        pi, qi = divmod(rem, q)
        for ko in range(k):
            out[ni][pi][qi][ko] = sum(a * b for a, b in zip(row, cols[ko]))
    return out
