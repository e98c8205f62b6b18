"""Pure-Python brute force for tiny shapes: nested loops over Python integers (unbounded), written
from the definitions of IntConv2D / IntLinear (section 3.2.1, Tab. 1: 3x3, stride 1, pad 1) and of
their adjoints. Used only to pin the oracle's C contractions; shares no code with them."""


def conv_fwd(x, w):
    N, H, W, C = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    CO = len(w)
    out = [[[[0] * CO for _ in range(W)] for _ in range(H)] for _ in range(N)]
    for n in range(N):
        for h in range(H):
            for q in range(W):
                for co in range(CO):
                    t = 0
                    for r in range(3):
                        for s in range(3):
                            hh, qq = h + r - 1, q + s - 1
                            if 0 <= hh < H and 0 <= qq < W:
                                for ci in range(C):
                                    t += int(x[n][hh][qq][ci]) * int(w[co][r][s][ci])
                    out[n][h][q][co] = t
    return out


def conv_dx(g, w):
    """dx[n][h][q][ci] = sum over every output position (ho, qo) and tap (r, s) that reads input
    (h, q) = (ho + r - 1, qo + s - 1) of g[n][ho][qo][co] * w[co][r][s][ci] (scatter form)."""
    N, H, W, CO = len(g), len(g[0]), len(g[0][0]), len(g[0][0][0])
    C = len(w[0][0][0])
    out = [[[[0] * C for _ in range(W)] for _ in range(H)] for _ in range(N)]
    for n in range(N):
        for ho in range(H):
            for qo in range(W):
                for r in range(3):
                    for s in range(3):
                        h, q = ho + r - 1, qo + s - 1
                        if 0 <= h < H and 0 <= q < W:
                            for co in range(CO):
                                for ci in range(C):
                                    out[n][h][q][ci] += int(g[n][ho][qo][co]) * int(w[co][r][s][ci])
    return out


def conv_dw(g, x):
    N, H, W, CO = len(g), len(g[0]), len(g[0][0]), len(g[0][0][0])
    C = len(x[0][0][0])
    out = [[[[0] * C for _ in range(3)] for _ in range(3)] for _ in range(CO)]
    for n in range(N):
        for h in range(H):
            for q in range(W):
                for r in range(3):
                    for s in range(3):
                        hh, qq = h + r - 1, q + s - 1
                        if 0 <= hh < H and 0 <= qq < W:
                            for co in range(CO):
                                for ci in range(C):
                                    out[co][r][s][ci] += int(g[n][h][q][co]) * int(x[n][hh][qq][ci])
    return out


def linear_fwd(x, w):
    return [[sum(int(x[n][k]) * int(w[m][k]) for k in range(len(x[0]))) for m in range(len(w))]
            for n in range(len(x))]


def linear_dx(e, w):
    K = len(w[0])
    return [[sum(int(e[n][m]) * int(w[m][k]) for m in range(len(w))) for k in range(K)]
            for n in range(len(e))]


def linear_dw(e, x):
    M, K = len(e[0]), len(x[0])
    return [[sum(int(e[n][m]) * int(x[n][k]) for n in range(len(e))) for k in range(K)]
            for m in range(M)]


def maxpool(a):
    """2x2/2 max-pool; returns (pooled, index of the first maximum in (0,0),(0,1),(1,0),(1,1))."""
    N, H, W, C = len(a), len(a[0]), len(a[0][0]), len(a[0][0][0])
    P = [[[[0] * C for _ in range(W // 2)] for _ in range(H // 2)] for _ in range(N)]
    I = [[[[0] * C for _ in range(W // 2)] for _ in range(H // 2)] for _ in range(N)]
    for n in range(N):
        for i in range(H // 2):
            for j in range(W // 2):
                for c in range(C):
                    win = [a[n][2 * i][2 * j][c], a[n][2 * i][2 * j + 1][c],
                           a[n][2 * i + 1][2 * j][c], a[n][2 * i + 1][2 * j + 1][c]]
                    best = 0
                    for t in range(1, 4):
                        if win[t] > win[best]:
                            best = t
                    P[n][i][j][c] = win[best]
                    I[n][i][j][c] = best
    return P, I


def maxpool_window(a, kh, kw):
    """kh x kw max-pool, stride (kh, kw): scan each window row by row and keep the first strict
    maximum; returns (pooled, index of the winner within its window)."""
    N, H, W, C = len(a), len(a[0]), len(a[0][0]), len(a[0][0][0])
    P = [[[[0] * C for _ in range(W // kw)] for _ in range(H // kh)] for _ in range(N)]
    I = [[[[0] * C for _ in range(W // kw)] for _ in range(H // kh)] for _ in range(N)]
    for n in range(N):
        for i in range(H // kh):
            for j in range(W // kw):
                for c in range(C):
                    best, arg = None, 0
                    for t in range(kh * kw):
                        v = int(a[n][i * kh + t // kw][j * kw + t % kw][c])
                        if best is None or v > best:
                            best, arg = v, t
                    P[n][i][j][c] = best
                    I[n][i][j][c] = arg
    return P, I


def philox4x64_10(ctr, key):
    """Philox4x64 with 10 rounds, written from its published definition (Salmon et al., SC'11):
    each round multiplies counter words 0 and 2 by two fixed 64-bit constants, and recombines the
    128-bit products' halves with words 1 and 3 and the key; the key is bumped by two Weyl
    constants between rounds. Python integers, so nothing wraps that should not."""
    mask = (1 << 64) - 1
    m0, m1 = 0xD2E7470EE14C6C93, 0xCA5A826395121157
    w0, w1 = 0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B
    c, k = list(ctr), list(key)
    for _ in range(10):
        p0, p1 = m0 * c[0], m1 * c[2]
        c = [(p1 >> 64) ^ c[1] ^ k[0], p1 & mask, (p0 >> 64) ^ c[3] ^ k[1], p0 & mask]
        k = [(k[0] + w0) & mask, (k[1] + w1) & mask]
    return c
