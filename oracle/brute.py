"""Pure-Python brute force for tiny convolutions (test infrastructure only).

Written independently of ``mec_oracle.c`` and sharing nothing with it, so the
two can check each other. Inputs are nested Python lists (or anything
indexable the same way) holding Python numbers; integers stay exact.
"""


def out_dim(i, k, s):
    """Eq. (1) with the floor reading: (i - k) // s + 1."""
    return (i - k) // s + 1


def conv2d(I, K, s_h, s_w):
    """Direct convolution by its definition (Section 3.1, Fig. 1(a)).

    I[n][h][w][c] (n-h-w-c) and K[a][b][c][m]; returns O[n][y][x][m] with
    O[n][y][x][m] = sum over a, b, c of I[n][y*s_h+a][x*s_w+b][c] * K[a][b][c][m].
    """
    i_n, i_h, i_w, i_c = len(I), len(I[0]), len(I[0][0]), len(I[0][0][0])
    k_h, k_w, k_c = len(K), len(K[0]), len(K[0][0][0])
    o_h, o_w = out_dim(i_h, k_h, s_h), out_dim(i_w, k_w, s_w)
    O = [[[[0 for _ in range(k_c)] for _ in range(o_w)] for _ in range(o_h)] for _ in range(i_n)]
    for n in range(i_n):
        for y in range(o_h):
            for x in range(o_w):
                for m in range(k_c):
                    total = 0
                    for a in range(k_h):
                        for b in range(k_w):
                            for c in range(i_c):
                                total += I[n][y * s_h + a][x * s_w + b][c] * K[a][b][c][m]
                    O[n][y][x][m] = total
    return O


def mec_lower(I, k_w, s_w):
    """MEC lowering (Algorithm 2's first loop) by element-wise assignment.

    Returns L[n][w][h][b][c] = I[n][h][s_w*w + b][c].
    """
    i_n, i_h, i_w, i_c = len(I), len(I[0]), len(I[0][0]), len(I[0][0][0])
    o_w = out_dim(i_w, k_w, s_w)
    return [[[[[I[n][h][s_w * w + b][c] for c in range(i_c)] for b in range(k_w)]
              for h in range(i_h)] for w in range(o_w)] for n in range(i_n)]


def dgrad(G, K, i_h, i_w, s_h, s_w):
    """dI by linearity: the convolution is linear in I, so dI[p] is the inner
    product of G with the output of the basis image that is 1 at pixel p and 0
    elsewhere. Uses only conv2d above."""
    i_n, k_c = len(G), len(G[0][0][0])
    k_h, k_w, i_c = len(K), len(K[0]), len(K[0][0])
    dI = [[[[0 for _ in range(i_c)] for _ in range(i_w)] for _ in range(i_h)] for _ in range(i_n)]
    for n in range(i_n):
        for h in range(i_h):
            for x in range(i_w):
                for c in range(i_c):
                    E = [[[[1 if (h2, x2, c2) == (h, x, c) else 0 for c2 in range(i_c)]
                           for x2 in range(i_w)] for h2 in range(i_h)]]
                    O = conv2d(E, K, s_h, s_w)[0]
                    dI[n][h][x][c] = sum(O[y][xx][m] * G[n][y][xx][m] for y in range(len(O))
                                         for xx in range(len(O[0])) for m in range(k_c))
    return dI


def wgrad(I, G, k_h, k_w, s_h, s_w):
    """dK by linearity in K: dK[q] is the inner product of G with the output
    of I under the basis kernel that is 1 at q. Uses only conv2d above."""
    i_c, k_c = len(I[0][0][0]), len(G[0][0][0])
    dK = [[[[0 for _ in range(k_c)] for _ in range(i_c)] for _ in range(k_w)] for _ in range(k_h)]
    for a in range(k_h):
        for b in range(k_w):
            for c in range(i_c):
                for m in range(k_c):
                    E = [[[[1 if (a2, b2, c2, m2) == (a, b, c, m) else 0 for m2 in range(k_c)]
                           for c2 in range(i_c)] for b2 in range(k_w)] for a2 in range(k_h)]
                    O = conv2d(I, E, s_h, s_w)
                    dK[a][b][c][m] = sum(O[n][y][x][mm] * G[n][y][x][mm] for n in range(len(O))
                                         for y in range(len(O[0])) for x in range(len(O[0][0]))
                                         for mm in range(k_c))
    return dK
