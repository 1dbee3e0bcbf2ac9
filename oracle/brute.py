"""Pure-Python brute force for tiny shapes.  TEST INFRASTRUCTURE ONLY.

Used to pin oracle.direct: the same definitions written as nested Python
loops over Python floats (fp64), with explicit bounds tests for padding.
"""

from __future__ import annotations


def conv2d(x, w, bias, stride, pad, relu=False):
    """x[n][c][h][w], w[o][c][r][s] nested lists -> y[n][o][oh][ow]."""
    N, C, H, W = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    O, KH, KW = len(w), len(w[0][0]), len(w[0][0][0])
    sh, sw = stride
    ph, pw = pad
    HO = (H + 2 * ph - KH) // sh + 1
    WO = (W + 2 * pw - KW) // sw + 1
    y = [[[[0.0] * WO for _ in range(HO)] for _ in range(O)] for _ in range(N)]
    for n in range(N):
        for o in range(O):
            for oh in range(HO):
                for ow in range(WO):
                    acc = 0.0 if bias is None else float(bias[o])
                    for c in range(C):
                        for r in range(KH):
                            for s in range(KW):
                                ih, iw = oh * sh - ph + r, ow * sw - pw + s
                                if 0 <= ih < H and 0 <= iw < W:
                                    acc += float(w[o][c][r][s]) * float(x[n][c][ih][iw])
                    if relu and acc < 0.0:
                        acc = 0.0
                    y[n][o][oh][ow] = acc
    return y


def linear(x, w, bias, relu=False):
    """x[k][b] feature-major, w[o][k] -> y[o][b]."""
    K, B, O = len(x), len(x[0]), len(w)
    y = [[0.0] * B for _ in range(O)]
    for o in range(O):
        for b in range(B):
            acc = 0.0 if bias is None else float(bias[o])
            for k in range(K):
                acc += float(w[o][k]) * float(x[k][b])
            if relu and acc < 0.0:
                acc = 0.0
            y[o][b] = acc
    return y
