"""The I420 row kernel stages three chroma rows per plane and output row,
r0, r1 for luma row y0 and r1, r2 for y1 = min(y0 + 1, H - 1). That works
because the vertical chroma taps of two consecutive luma rows always share
y0's second chroma row: y1's taps either move on by one row (y1's first row
is y0's second) or stay on y0's pair (y1's second row is y0's second), in
which case y1 reads (r1, r2) = (its second, its first) row with the weight
4 - f. Checked here for every frame height up to 64 chroma rows, with the
taps written from the definition (centred siting: luma row y sits at chroma
coordinate y/2 - 1/4, clamped at both ends), in exact rationals."""
from fractions import Fraction
import math


def taps(y: int, n: int):
    u = Fraction(y, 2) - Fraction(1, 4)
    if u <= 0:
        return 0, 0, Fraction(0)
    f = math.floor(u)
    if f >= n - 1:
        return n - 1, n - 1, Fraction(0)
    return f, f + 1, u - f


def test_consecutive_luma_rows_share_the_second_chroma_row():
    for H in range(1, 129):
        n = (H + 1) // 2
        for y0 in range(H):
            y1 = min(y0 + 1, H - 1)
            a0, a1, wa = taps(y0, n)
            b0, b1, wb = taps(y1, n)
            nxt = b0 == a1
            assert nxt or b1 == a1, (H, y0)
            r2 = b1 if nxt else b0
            f1 = 4 * wb if nxt else 4 - 4 * wb
            # y1 read as rows (r1, r2) with weight f1 / 4 on r2 equals its taps
            # on any row values (distinct rows get distinct values)
            for k in (3, 17, 101):
                v = lambda r: k * r + 5
                want = (1 - wb) * v(b0) + wb * v(b1)
                got = (1 - f1 / 4) * v(a1) + f1 / 4 * v(r2)
                assert want == got, (H, y0)
