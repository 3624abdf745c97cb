"""Exact brute-force conv2d for tiny shapes -- TEST INFRASTRUCTURE ONLY.

It uses the *scatter* form of the operator in exact rational arithmetic
(``fractions.Fraction``): every input pixel x[n, c, h, w] is multiplied by
every filter tap of every output channel of its group, and the product is
added into the output pixel it lands on, if that pixel exists. This walks the
operator in the opposite direction from the gather loop of ``conv2d_ref.c``,
so an index mistake in either does not cancel out. Padding enters only
through which output a product lands on: (h + ph - r*dh) must be a
non-negative multiple of the stride below OH*sh.

Layouts and the operator definition are those of the fp64 oracle
(paper, section 2.1; cross-correlation, zero padding, floor output size).
"""
from __future__ import annotations

from fractions import Fraction


def conv2d_scatter(x, w, N, C, H, W, K, R, S, stride=(1, 1), pad=(0, 0), dil=(1, 1),
                   groups=1):
    """x: nested lists [N][C][H][W]; w: [K][C/groups][R][S]. Returns [N][K][OH][OW] Fractions."""
    sh, sw = stride
    ph, pw = pad
    dh, dw = dil
    OH = (H + 2 * ph - dh * (R - 1) - 1) // sh + 1
    OW = (W + 2 * pw - dw * (S - 1) - 1) // sw + 1
    OH, OW = max(OH, 0), max(OW, 0)
    Cg, Kg = C // groups, K // groups
    y = [[[[Fraction(0) for _ in range(OW)] for _ in range(OH)] for _ in range(K)] for _ in range(N)]
    for n in range(N):
        for c in range(C):
            g = c // Cg
            cl = c - g * Cg
            for h in range(H):
                for wi in range(W):
                    xv = Fraction(x[n][c][h][wi])
                    if xv == 0:
                        continue
                    for k in range(g * Kg, (g + 1) * Kg):
                        for r in range(R):
                            num_h = h + ph - r * dh
                            if num_h < 0 or num_h % sh:
                                continue
                            p = num_h // sh
                            if p >= OH:
                                continue
                            for t in range(S):
                                num_w = wi + pw - t * dw
                                if num_w < 0 or num_w % sw:
                                    continue
                                q = num_w // sw
                                if q >= OW:
                                    continue
                                y[n][k][p][q] += xv * Fraction(w[k][cl][r][t])
    return y
