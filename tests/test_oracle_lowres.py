"""Pins for the oracle's uint8 output and its low-resolution augmentation
(the reduce-to-r-then-preprocess op) against closed forms computed here in
integer arithmetic or from separately pinned oracle calls.

Runs without a GPU.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle

F32, F16, U8 = oracle.OUT_F32, oracle.OUT_F16, oracle.OUT_U8
MEAN = np.array([123.675, 116.28, 103.53], np.float32)
STD = np.array([58.395, 57.12, 57.375], np.float32)


def _flat(imgs):
    flat = np.concatenate([im.reshape(-1) for im in imgs])
    offs = np.cumsum([0] + [im.size for im in imgs[:-1]]).astype(np.int64)
    return flat, offs, [im.shape[1] for im in imgs], [im.shape[0] for im in imgs]


def _u8(imgs, S, Ch, Cw, mode=oracle.RESIZE_SHORT_CROP, layout=oracle.NHWC):
    flat, offs, ws, hs = _flat(imgs)
    return oracle.preprocess_batch_ex(flat, offs, ws, hs, None, None, S, Ch, Cw, np.zeros(3),
                                      np.ones(3), U8, mode, layout)


def _box2_rounded(a: np.ndarray) -> np.ndarray:
    """2 x 2 block means of an integer image rounded to nearest, ties to even,
    in integer arithmetic: sum = 4q + rem; rem 2 is the tie."""
    a = a.astype(np.int64)
    s = a[0::2, 0::2] + a[0::2, 1::2] + a[1::2, 0::2] + a[1::2, 1::2]
    q, rem = np.divmod(s, 4)
    return (q + (rem == 3) + ((rem == 2) & (q % 2 == 1))).astype(np.uint8)


@pytest.mark.parametrize("layout", [oracle.NCHW, oracle.NHWC])
def test_u8_2x_downscale_is_rounded_box_mean(layout):
    """A 2x direct downscale puts every output pixel at a 2 x 2 block centre
    with exact weights 1/2, so the uint8 output is the block mean rounded to
    nearest with ties to even."""
    rng = np.random.default_rng(21)
    img = rng.integers(0, 256, (30, 44, 3), dtype=np.uint8)
    out = _u8([img], 1, 15, 22, oracle.RESIZE_DIRECT, layout)[0]
    got = out if layout == oracle.NHWC else np.transpose(out, (1, 2, 0))
    assert got.dtype == np.uint8
    assert np.array_equal(got, _box2_rounded(img))


def test_u8_rounding_ties_go_to_even():
    """Block means 0.5, 1.5, 2.5 and 3.5 round to 0, 2, 2 and 4."""
    blocks = [(0, 1), (1, 2), (2, 3), (3, 4)]
    img = np.zeros((2, 8, 3), np.uint8)
    for k, (a, b) in enumerate(blocks):
        img[:, 2 * k, :] = a
        img[:, 2 * k + 1, :] = b
    out = _u8([img], 1, 1, 4, oracle.RESIZE_DIRECT)[0]
    assert out[0, :, 0].tolist() == [0, 2, 2, 4]


def test_u8_same_size_is_identity():
    """Short side S equal to the image's and a crop of the whole image: every
    tap has weight 0, the output is the input bytes."""
    rng = np.random.default_rng(22)
    img = rng.integers(0, 256, (23, 37, 3), dtype=np.uint8)
    assert np.array_equal(_u8([img], 23, 23, 37)[0], img)
    nchw = _u8([img], 23, 23, 37, layout=oracle.NCHW)[0]
    assert np.array_equal(np.transpose(nchw, (1, 2, 0)), img)


def _lowres(imgs, r, S, Ch, Cw, dtype=F32, mean=MEAN, std=STD):
    flat, offs, ws, hs = _flat(imgs)
    return oracle.lowres_preprocess_batch(flat, offs, ws, hs, None, r, S, Ch, Cw, mean, std,
                                          dtype)


def test_lowres_of_constant_image_is_constant():
    c = 77
    img = np.full((61, 90, 3), c, np.uint8)
    out = _lowres([img], 19, 40, 32, 32)
    exp = (np.float32(c) - MEAN) / STD
    assert np.array_equal(out[0], np.broadcast_to(exp[:, None, None], (3, 32, 32)))


def test_lowres_at_the_short_side_is_the_central_square():
    """With r equal to the short side the reduction does not resample: it
    keeps the central r x r square (floor((W - r)/2) columns off the left), so
    the op equals steps 2-4 on that square cut out in numpy."""
    rng = np.random.default_rng(23)
    img = rng.integers(0, 256, (41, 70, 3), dtype=np.uint8)
    r = 41
    left = (70 - r) // 2
    sq = np.ascontiguousarray(img[:, left:left + r])
    got = _lowres([img], r, 48, 40, 36, F16)
    flat, offs, ws, hs = _flat([sq])
    exp = oracle.preprocess_batch(flat, offs, ws, hs, None, 48, 40, 36, MEAN, STD, F16)
    assert np.array_equal(got.view(np.uint16), exp.view(np.uint16))


def test_lowres_half_size_is_rounded_box_mean_then_preprocess():
    """A 2r x 2r image reduced to r x r is the rounded 2 x 2 block mean
    (integer closed form above); the op then equals steps 2-4 on that image."""
    rng = np.random.default_rng(24)
    r = 26
    img = rng.integers(0, 256, (2 * r, 2 * r, 3), dtype=np.uint8)
    got = _lowres([img], r, 64, 56, 56, F32)
    low = _box2_rounded(img)
    flat, offs, ws, hs = _flat([low])
    exp = oracle.preprocess_batch(flat, offs, ws, hs, None, 64, 56, 56, MEAN, STD, F32)
    assert np.array_equal(got, exp)


def test_yuv_lowres_is_rounded_conversion_then_preprocess():
    """An r x r I420 frame reduced to r x r is the BT.601 conversion (pinned
    elsewhere) rounded to uint8 with ties to even; the op then equals steps
    2-4 on that RGB image."""
    rng = np.random.default_rng(25)
    r = 30
    y = rng.integers(16, 236, (r, r), dtype=np.uint8)
    cb = rng.integers(16, 241, (r // 2, r // 2), dtype=np.uint8)
    cr = rng.integers(16, 241, (r // 2, r // 2), dtype=np.uint8)
    flat = np.concatenate([y.reshape(-1), cb.reshape(-1), cr.reshape(-1)])
    got = oracle.yuv420_lowres_preprocess_batch(flat, [0], [r * r], [r * r + (r // 2) ** 2], [r],
                                                [r], r, 40, 32, 32, MEAN, STD, F16)
    rgb = np.rint(oracle.yuv420_to_rgb(y, cb, cr)).astype(np.uint8)
    f2, o2, w2, h2 = _flat([rgb])
    exp = oracle.preprocess_batch(f2, o2, w2, h2, None, 40, 32, 32, MEAN, STD, F16)
    assert np.array_equal(got.view(np.uint16), exp.view(np.uint16))


def test_lowres_rejects_bad_arguments():
    img = np.zeros((8, 8, 3), np.uint8)
    with pytest.raises(ValueError):
        _lowres([img], 0, 8, 8, 8)
    with pytest.raises(ValueError):
        flat, offs, ws, hs = _flat([img])
        oracle.lowres_preprocess_batch(flat, offs, ws, hs, None, 4, 8, 8, 8, MEAN, STD, U8)


def test_single_image_entry_points_match_the_batch_calls():
    """The raw-pointer single-image calls (used by the CPU baseline) give the
    batch calls' bytes."""
    rng = np.random.default_rng(26)
    img = rng.integers(0, 256, (45, 62, 3), dtype=np.uint8)
    flat, offs, ws, hs = _flat([img])
    out = np.empty((3, 20, 24), np.uint16)
    rc = oracle.preprocess_image_ex_into(flat.ctypes.data, 62, 45, 186, (5, 3, 40, 30), 1, 20,
                                         24, MEAN, STD, F16, oracle.RESIZE_DIRECT, oracle.NCHW,
                                         out.ctypes.data)
    exp = oracle.preprocess_batch_ex(flat, offs, ws, hs, None, [(5, 3, 40, 30)], 1, 20, 24, MEAN,
                                     STD, F16, oracle.RESIZE_DIRECT, oracle.NCHW)
    assert rc == 0 and np.array_equal(out, exp[0].view(np.uint16))
    o1 = np.empty((3, 28, 28), np.uint16)
    rc = oracle.lowres_preprocess_image_into(flat.ctypes.data, 62, 45, 186, 17, 32, 28, 28, MEAN,
                                             STD, F16, o1.ctypes.data)
    exp = oracle.lowres_preprocess_batch(flat, offs, ws, hs, None, 17, 32, 28, 28, MEAN, STD, F16)
    assert rc == 0 and np.array_equal(o1, exp[0].view(np.uint16))

    W, H = 33, 21
    y = rng.integers(16, 236, (H, W), dtype=np.uint8)
    cb = rng.integers(16, 241, ((H + 1) // 2, (W + 1) // 2), dtype=np.uint8)
    cr = rng.integers(16, 241, ((H + 1) // 2, (W + 1) // 2), dtype=np.uint8)
    o2 = np.empty((10, 12, 3), np.float32)
    rc = oracle.yuv420_preprocess_image_ex_into(y.ctypes.data, cb.ctypes.data, cr.ctypes.data, W,
                                                H, (1, 1, 30, 19), 1, 10, 12, MEAN, STD, F32,
                                                oracle.RESIZE_DIRECT, oracle.NHWC,
                                                oracle.CHROMA_LEFT, o2.ctypes.data)
    yuv = np.concatenate([y.reshape(-1), cb.reshape(-1), cr.reshape(-1)])
    exp = oracle.yuv420_preprocess_batch_ex(yuv, [0], [W * H], [W * H + cb.size], [W], [H],
                                            [(1, 1, 30, 19)], 1, 10, 12, MEAN, STD, F32,
                                            oracle.RESIZE_DIRECT, oracle.NHWC, oracle.CHROMA_LEFT)
    assert rc == 0 and np.array_equal(o2, exp[0])
    o3 = np.empty((3, 16, 16), np.float32)
    rc = oracle.yuv420_lowres_preprocess_image_into(y.ctypes.data, cb.ctypes.data, cr.ctypes.data,
                                                    W, H, 9, 20, 16, 16, MEAN, STD, F32,
                                                    o3.ctypes.data)
    exp = oracle.yuv420_lowres_preprocess_batch(yuv, [0], [W * H], [W * H + cb.size], [W], [H], 9,
                                                20, 16, 16, MEAN, STD, F32)
    assert rc == 0 and np.array_equal(o3, exp[0])
