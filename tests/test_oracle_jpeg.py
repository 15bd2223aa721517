"""Pins for the oracle's partial JPEG decoding: the 8 x 8 inverse DCT against
the T.81 formula evaluated in double, round trips through a double-precision
forward DCT, and Algorithm 1's MCU-aligned rectangle against hand-worked
values and exact-rational tap footprints.

Runs without a GPU.
"""
from __future__ import annotations

import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "jpeg_mcu_rect.txt")


def _basis(u: int, v: int) -> np.ndarray:
    """T.81 A.3.3 basis in double: 1/4 C(u) C(v) cos((2x+1)u pi/16) cos((2y+1)v pi/16),
    indexed [y, x]."""
    cu = 1 / math.sqrt(2) if u == 0 else 1.0
    cv = 1 / math.sqrt(2) if v == 0 else 1.0
    x = np.arange(8)
    cx = np.cos((2 * x + 1) * u * math.pi / 16)
    cy = np.cos((2 * x + 1) * v * math.pi / 16)
    return 0.25 * cu * cv * np.outer(cy, cx)


def _round_half_even_clamp(a: np.ndarray) -> np.ndarray:
    return np.clip(np.rint(a), 0, 255)


def test_dc_only_block_is_flat():
    """A DC coefficient d (times its table entry q) gives 128 + d q / 8 at every
    pixel; d q a multiple of 8 keeps it an integer."""
    for d, q in [(0, 1), (40, 1), (-64, 2), (10, 16), (-127, 8)]:
        c = np.zeros(64, np.int16)
        c[0] = d
        qt = np.ones(64, np.uint16)
        qt[0] = q
        exp = np.clip(128 + d * q / 8, 0, 255)
        assert np.all(oracle.idct_block(c, qt) == exp), (d, q)


@pytest.mark.parametrize("amp", [1, 7, -13, 50])
def test_every_basis_function(amp):
    """A single coefficient at (u, v) reproduces the double-precision basis
    function (orientation: u horizontal, v vertical), rounded, except where
    the double value lies within 1e-3 of a rounding boundary."""
    q = np.ones(64, np.uint16)
    for v in range(8):
        for u in range(8):
            c = np.zeros(64, np.int16)
            c[v * 8 + u] = amp
            exact = 128 + amp * _basis(u, v)
            got = oracle.idct_block(c, q).astype(np.float64)
            frac = np.abs(exact - np.floor(exact) - 0.5)
            sure = frac > 1e-3
            assert np.array_equal(got[sure], _round_half_even_clamp(exact)[sure]), (u, v)
            assert np.max(np.abs(got - exact)) <= 0.5 + 1e-3


def test_dequantisation_multiplies():
    """Coefficient c with table entry q equals coefficient c q with entry 1."""
    rng = np.random.default_rng(3)
    c = rng.integers(-20, 21, 64).astype(np.int16)
    q = rng.integers(1, 12, 64).astype(np.uint16)
    assert np.array_equal(oracle.idct_block(c, q),
                          oracle.idct_block((c.astype(np.int32) * q).astype(np.int16),
                                            np.ones(64, np.uint16)))


def test_round_trip_through_forward_dct():
    """Smooth 8 x 8 blocks: forward DCT in double, coefficients rounded to
    integers, then the oracle's inverse: within 1 of the original, mostly
    exact."""
    rng = np.random.default_rng(4)
    B = np.stack([_basis(u, v) for v in range(8) for u in range(8)])  # [k, y, x]
    diffs = []
    for _ in range(200):
        a, b, c0 = rng.uniform(-6, 6), rng.uniform(-6, 6), rng.uniform(40, 215)
        yy, xx = np.mgrid[0:8, 0:8]
        x = np.clip(np.rint(c0 + a * xx + b * yy + rng.integers(-2, 3, (8, 8))), 0, 255)
        # orthonormal: F = sum (x - 128) * basis
        F = np.rint(np.tensordot(B, x - 128, axes=([1, 2], [0, 1]))).astype(np.int16)
        back = oracle.idct_block(F, np.ones(64, np.uint16)).astype(np.int64)
        diffs.append(np.abs(back - x))
    d = np.stack(diffs)
    assert d.max() <= 1
    assert np.mean(d == 0) > 0.9


def _golden():
    rows = []
    for line in open(GOLDEN):
        line = line.split("#")[0].split()
        if line:
            rows.append([int(v) for v in line])
    return rows


def test_mcu_rect_golden():
    for W, H, S, Ch, Cw, x, y, w, h in _golden():
        assert oracle.jpeg_mcu_rect(W, H, S, Ch, Cw) == (x, y, w, h)


def _exact_tap(x: int, n_in: int, n_out: int) -> tuple[int, int]:
    num = Fraction((2 * x + 1) * n_in - n_out, 2 * n_out)
    if num <= 0:
        return 0, 0
    x0 = math.floor(num)
    return (n_in - 1, n_in - 1) if x0 >= n_in - 1 else (x0, x0 + 1)


def _exact_chroma(x: int, n: int) -> tuple[int, int]:
    u = Fraction(x, 2) - Fraction(1, 4)
    if u <= 0:
        return 0, 0
    f = math.floor(u)
    return (n - 1, n - 1) if f >= n - 1 else (f, f + 1)


@pytest.mark.parametrize("W,H,S,C", [(1920, 1080, 224, 224), (641, 359, 128, 112),
                                     (333, 517, 256, 224), (17, 33, 16, 8), (1000, 200, 300, 150)])
def test_mcu_rect_holds_every_sample_and_is_minimal(W, H, S, C):
    """Every luma and chroma sample any output pixel reads lies inside the
    rectangle; it is 16-aligned (or ends at the frame); dropping an MCU
    column or row from any side loses a sample."""
    x, y, w, h = oracle.jpeg_mcu_rect(W, H, S, C, C)
    Wr, Hr, left, top = oracle.output_geometry(W, H, S, C, C)
    xs = [t for c in range(C) for t in _exact_tap(left + c, W, Wr)]
    ys = [t for r in range(C) for t in _exact_tap(top + r, H, Hr)]
    Wc, Hc = (W + 1) // 2, (H + 1) // 2
    cxs = [2 * t + d for lx in set(xs) for t in _exact_chroma(lx, Wc) for d in (0, 1)]
    cys = [2 * t + d for ly in set(ys) for t in _exact_chroma(ly, Hc) for d in (0, 1)]
    lo_x, hi_x = min(xs + [v for v in cxs]), min(max(xs + cxs), W - 1)
    lo_y, hi_y = min(ys + cys), min(max(ys + cys), H - 1)
    assert x % 16 == 0 and y % 16 == 0
    assert (x + w) % 16 == 0 or x + w == W
    assert (y + h) % 16 == 0 or y + h == H
    assert x <= lo_x and hi_x < x + w and y <= lo_y and hi_y < y + h
    assert lo_x < x + 16 and hi_x >= x + w - 16 and lo_y < y + 16 and hi_y >= y + h - 16


def test_partial_decode_equals_full_decode_inside_the_rect():
    """Decoding only the rectangle's blocks gives the full decode's samples
    inside it (chroma over the matching half-resolution range) and leaves
    the rest untouched."""
    rng = np.random.default_rng(5)
    W, H = 203, 77
    coef = rng.integers(-40, 41, oracle.jpeg_coef_count(W, H)).astype(np.int16)
    qy = rng.integers(1, 9, 64).astype(np.uint16)
    qc = rng.integers(1, 9, 64).astype(np.uint16)
    full = oracle.jpeg_decode_i420(coef, qy, qc, W, H, fill=7)
    rect = (48, 16, 112, 48)
    part = oracle.jpeg_decode_i420(coef, qy, qc, W, H, rect, fill=7)
    x, y, w, h = rect
    assert np.array_equal(part[0][y:y + h, x:x + w], full[0][y:y + h, x:x + w])
    for k in (1, 2):
        assert np.array_equal(part[k][y // 2:(y + h) // 2, x // 2:(x + w) // 2],
                              full[k][y // 2:(y + h) // 2, x // 2:(x + w) // 2])
    outside = np.ones((H, W), bool)
    outside[y:y + h, x:x + w] = False
    assert np.all(part[0][outside] == 7)
    # blocks along the right and bottom frame edges are clipped, not skipped
    edge = oracle.jpeg_decode_i420(coef, qy, qc, W, H, (192, 64, 11, 13), fill=7)
    assert np.array_equal(edge[0][64:, 192:], full[0][64:, 192:])


def test_dense_blocks_match_the_double_formula():
    """Blocks with every coefficient nonzero (Laplacian terms falling off with
    frequency, as in coded photographs, and full-range noise): the oracle's
    output equals T.81's formula evaluated in double and rounded, except
    where the double value lies within 1e-3 of a rounding boundary or of the
    clamp, and is never more than 1/2 + 1e-3 from it before clamping. This
    pins the sum as a whole: a dropped or doubled term, a sign error in the
    parity split or a transposed pass all move pixels by far more."""
    rng = np.random.default_rng(24)
    B = np.stack([_basis(u, v) for v in range(8) for u in range(8)])  # [k, y, x]
    q = np.ones(64, np.uint16)
    for trial in range(300):
        if trial % 2:
            c = rng.integers(-300, 301, 64)
        else:
            uu, vv = np.meshgrid(np.arange(8), np.arange(8))
            c = np.rint(rng.laplace(0, 60 / (1 + uu + vv))).reshape(64)
            c[0] = rng.integers(-400, 400)
        c = np.clip(c, -1024, 1023).astype(np.int16)
        exact = 128 + np.tensordot(c.astype(np.float64), B, axes=(0, 0))
        got = oracle.idct_block(c, q).astype(np.float64)
        inside = (exact > 0.001) & (exact < 254.999)
        frac = np.abs(exact - np.floor(exact) - 0.5)
        sure = inside & (frac > 1e-3)
        assert np.array_equal(got[sure], np.rint(exact[sure])), trial
        assert np.all(np.abs(got[inside] - exact[inside]) <= 0.5 + 1e-3), trial
