"""Brute-force loops for tiny shapes, used to pin ``oracle.column``.

TEST INFRASTRUCTURE (see ``oracle/column.py``).

Every output element is computed straight from its definition with scalar
Python loops: no padding arrays, no slicing, no library products.
"""
from __future__ import annotations

import math


def conv(x, w, sh, sw, ph, pw):
    """out[b][y][x][o] = sum over (i, j, c) of w[o][i][j][c] * x[b][y*sh-ph+i]
    [x*sw-pw+j][c], with terms outside the image omitted (zero padding)."""
    B, H, W, C = x.shape
    Co, kh, kw, _ = w.shape
    Ho = (H + 2 * ph - kh) // sh + 1
    Wo = (W + 2 * pw - kw) // sw + 1
    out = [[[[0.0] * Co for _ in range(Wo)] for _ in range(Ho)] for _ in range(B)]
    for b in range(B):
        for y in range(Ho):
            for xx in range(Wo):
                for o in range(Co):
                    s = 0.0
                    for i in range(kh):
                        for j in range(kw):
                            r, q = y * sh - ph + i, xx * sw - pw + j
                            if 0 <= r < H and 0 <= q < W:
                                for c in range(C):
                                    s += float(w[o, i, j, c]) * float(x[b, r, q, c])
                    out[b][y][xx][o] = s
    return out


def maxpool(x, kh, kw, sh, sw, ph, pw):
    """(value, first row-major argmax) of every window; positions outside the
    image are skipped, and the index counts them as window positions."""
    B, H, W, C = x.shape
    Ho = (H + 2 * ph - kh) // sh + 1
    Wo = (W + 2 * pw - kw) // sw + 1
    val = [[[[0.0] * C for _ in range(Wo)] for _ in range(Ho)] for _ in range(B)]
    idx = [[[[0] * C for _ in range(Wo)] for _ in range(Ho)] for _ in range(B)]
    for b in range(B):
        for y in range(Ho):
            for xx in range(Wo):
                for c in range(C):
                    best, bi = -math.inf, -1
                    for i in range(kh):
                        for j in range(kw):
                            r, q = y * sh - ph + i, xx * sw - pw + j
                            if 0 <= r < H and 0 <= q < W:
                                v = float(x[b, r, q, c])
                                if bi < 0 or v > best:
                                    best, bi = v, i * kw + j
                    val[b][y][xx][c] = best
                    idx[b][y][xx][c] = bi
    return val, idx


def dependency_rows(ksp_chain, h_in, out_rows):
    """Set of input rows that the given output rows of a chain of windowed
    ops depend on, found by enumerating every window (tiny shapes only).
    ``ksp_chain`` lists (k, s, p) from input to output."""
    sizes = [h_in]
    for k, s, p in ksp_chain:
        sizes.append((sizes[-1] + 2 * p - k) // s + 1)
    need = set(out_rows)
    for (k, s, p), hin in zip(reversed(ksp_chain), reversed(sizes[:-1])):
        nxt = set()
        for y in need:
            for i in range(k):
                r = y * s - p + i
                if 0 <= r < hin:
                    nxt.add(r)
        need = nxt
    return need
