"""Pins for the oracle's variants -- region of interest, direct resize,
channels-last output, left-sited chroma -- against closed forms and
properties that do not come from the oracle itself.

Runs without a GPU.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle

F32, F16 = oracle.OUT_F32, oracle.OUT_F16
ZERO, ONE = np.zeros(3, np.float32), np.ones(3, np.float32)
KR, KB = 0.299, 0.114


def _rgb_batch(imgs):
    """Flat buffer + tables for a list of H x W x 3 uint8 images."""
    flat = np.concatenate([im.reshape(-1) for im in imgs])
    offs = np.cumsum([0] + [im.size for im in imgs[:-1]]).astype(np.int64)
    return flat, offs, [im.shape[1] for im in imgs], [im.shape[0] for im in imgs]


def _run_rgb(imgs, rois, S, Ch, Cw, mode, layout, dtype=F32, mean=ZERO, std=ONE):
    flat, offs, ws, hs = _rgb_batch(imgs)
    return oracle.preprocess_batch_ex(flat, offs, ws, hs, None, rois, S, Ch, Cw, mean, std, dtype,
                                      mode, layout)


def _box2(a: np.ndarray) -> np.ndarray:
    """Mean of each 2 x 2 block of an H x W x 3 array (H, W even)."""
    a = a.astype(np.float64)
    return (a[0::2, 0::2] + a[0::2, 1::2] + a[1::2, 0::2] + a[1::2, 1::2]) / 4


@pytest.mark.parametrize("layout", [oracle.NCHW, oracle.NHWC])
def test_roi_direct_2x_downscale_is_box_mean(layout):
    """Direct resize of a 2Cw x 2Ch ROI to Cw x Ch: the half-pixel map puts every
    output pixel at the centre of a 2 x 2 block (weights 1/2, exact), so the
    output is the block mean of the ROI -- at the ROI's offset in the image, in
    the requested layout. A wrong ROI origin, a swapped axis, the short-side
    geometry used by mistake or a wrong layout index all fail."""
    rng = np.random.default_rng(7)
    img = rng.integers(0, 256, (37, 45, 3), dtype=np.uint8)
    Ch, Cw, rx, ry = 6, 9, 11, 5
    roi = [(rx, ry, 2 * Cw, 2 * Ch)]
    out = _run_rgb([img], roi, 1, Ch, Cw, oracle.RESIZE_DIRECT, layout)[0]
    exp = _box2(img[ry:ry + 2 * Ch, rx:rx + 2 * Cw])
    got = out.astype(np.float64) if layout == oracle.NHWC else np.transpose(out, (1, 2, 0))
    assert np.array_equal(got, exp)


def test_roi_direct_2x_upscale_closed_form():
    """Direct resize of a ROI to twice its size: output index x maps to
    (2x - 1)/4, so interior weights are 1/4 and 3/4 and the edges clamp; with
    integer pixels every lerp is exact and the closed form below is the
    result bit for bit."""
    rng = np.random.default_rng(8)
    img = rng.integers(0, 256, (20, 30, 3), dtype=np.uint8)
    rx, ry, w, h = 4, 3, 7, 5
    out = _run_rgb([img], [(rx, ry, w, h)], 1, 2 * h, 2 * w, oracle.RESIZE_DIRECT,
                   oracle.NHWC)[0].astype(np.float64)
    roi = img[ry:ry + h, rx:rx + w].astype(np.float64)

    def taps(n_out, n_in):
        u = (2 * np.arange(n_out) - 1) / 4.0
        u = np.clip(u, 0, n_in - 1)
        x0 = np.minimum(np.floor(u).astype(int), n_in - 1)
        x1 = np.minimum(x0 + 1, n_in - 1)
        return x0, x1, u - x0

    y0, y1, wy = taps(2 * h, h)
    x0, x1, wx = taps(2 * w, w)
    top = roi[y0][:, x0] + wx[None, :, None] * (roi[y0][:, x1] - roi[y0][:, x0])
    bot = roi[y1][:, x0] + wx[None, :, None] * (roi[y1][:, x1] - roi[y1][:, x0])
    exp = top + wy[:, None, None] * (bot - top)
    assert np.array_equal(out, exp)


def test_roi_short_side_equals_cut_image():
    """Short-side resize and central crop of a ROI equal the same call on a
    separate copy of the ROI's pixels (the ROI is cut first; taps clamp at the
    ROI's edges, never reading outside it)."""
    rng = np.random.default_rng(9)
    img = rng.integers(0, 256, (90, 120, 3), dtype=np.uint8)
    rx, ry, w, h = 17, 9, 71, 53
    a = _run_rgb([img], [(rx, ry, w, h)], 48, 40, 44, oracle.RESIZE_SHORT_CROP, oracle.NCHW,
                 F16)[0]
    cut = np.ascontiguousarray(img[ry:ry + h, rx:rx + w])
    b = _run_rgb([cut], None, 48, 40, 44, oracle.RESIZE_SHORT_CROP, oracle.NCHW, F16)[0]
    assert np.array_equal(a.view(np.uint16), b.view(np.uint16))


def test_nhwc_is_a_transpose_of_nchw():
    """The layouts hold the same numbers: NHWC[n, y, x, c] == NCHW[n, c, y, x]."""
    rng = np.random.default_rng(10)
    imgs = [rng.integers(0, 256, (h, w, 3), dtype=np.uint8) for h, w in [(31, 40), (50, 33)]]
    args = (None, 24, 20, 22, oracle.RESIZE_SHORT_CROP)
    a = _run_rgb(imgs, *args, oracle.NCHW, F16, np.full(3, 120, np.float32),
                 np.full(3, 60, np.float32))
    b = _run_rgb(imgs, *args, oracle.NHWC, F16, np.full(3, 120, np.float32),
                 np.full(3, 60, np.float32))
    assert np.array_equal(np.transpose(a, (0, 2, 3, 1)).view(np.uint16), b.view(np.uint16))


def test_direct_resize_ignores_aspect_and_crops_nothing():
    """Direct resize geometry: the resized size is the output size, no crop."""
    assert oracle.output_geometry(640, 480, 256, 112, 96, oracle.RESIZE_DIRECT) == (96, 112, 0, 0)
    assert oracle.output_geometry(640, 480, 256, 224, 224) == (341, 256, 58, 16)


@pytest.mark.parametrize("roi", [(-1, 0, 4, 4), (0, 0, 0, 4), (2, 0, 9, 4), (0, 3, 4, 6)])
def test_roi_outside_the_image_is_rejected(roi):
    img = np.zeros((8, 10, 3), np.uint8)
    with pytest.raises(ValueError):
        _run_rgb([img], [roi], 4, 2, 2, oracle.RESIZE_DIRECT, oracle.NCHW)


def test_left_siting_on_ramps():
    """Left (co-sited) 4:2:0: chroma sample k sits at luma column 2k, so a
    horizontal chroma ramp a + b k reaches luma column x as a + b x / 2 (and
    clamps past the last sample); rows stay centred (y/2 - 1/4)."""
    W, H = 64, 40
    Wc, Hc = W // 2, H // 2
    y = np.full((H, W), 128, np.uint8)
    cb = np.tile((40 + 4 * np.arange(Wc)).astype(np.uint8)[None, :], (Hc, 1))
    cr = np.tile((60 + 5 * np.arange(Hc)).astype(np.uint8)[:, None], (1, Wc))
    rgb = oracle.yuv420_to_rgb_sited(y, cb, cr, oracle.CHROMA_LEFT).astype(np.float64)
    x = np.arange(W, dtype=np.float64)
    cbx = np.clip(40 + 4 * (x / 2), 40, 40 + 4 * (Wc - 1))
    yy = np.arange(H, dtype=np.float64)
    cry = np.clip(60 + 5 * (yy / 2 - 0.25), 60, 60 + 5 * (Hc - 1))
    b_exp = np.clip(128 + 2 * (1 - KB) * (cbx - 128), 0, 255)
    r_exp = np.clip(128 + 2 * (1 - KR) * (cry - 128), 0, 255)
    assert np.max(np.abs(rgb[:, :, 2] - b_exp[None, :])) < 1e-4
    assert np.max(np.abs(rgb[:, :, 0] - r_exp[:, None])) < 1e-4
    # the centred siting differs from it by a quarter chroma sample
    c = oracle.yuv420_to_rgb_sited(y, cb, cr, oracle.CHROMA_CENTER)
    assert np.array_equal(c, oracle.yuv420_to_rgb(y, cb, cr))
    assert not np.array_equal(c[:, :, 2], rgb[:, :, 2].astype(np.float32))


@pytest.mark.parametrize("siting", [oracle.CHROMA_CENTER, oracle.CHROMA_LEFT])
def test_yuv_roi_converts_the_frame_then_cuts(siting):
    """An I420 ROI at odd luma coordinates: the frame is converted first (chroma
    taps in frame coordinates), then the ROI is cut and box-averaged by a direct
    2x downscale. The expected value is the 2 x 2 lerp-form mean of the
    converted frame's pixels, evaluated here in numpy fp32."""
    rng = np.random.default_rng(11)
    W, H = 41, 29
    Wc, Hc = (W + 1) // 2, (H + 1) // 2
    yp = rng.integers(16, 236, (H, W), dtype=np.uint8)
    cb = rng.integers(16, 241, (Hc, Wc), dtype=np.uint8)
    cr = rng.integers(16, 241, (Hc, Wc), dtype=np.uint8)
    flat = np.concatenate([yp.reshape(-1), cb.reshape(-1), cr.reshape(-1)])
    rx, ry, Ch, Cw = 7, 3, 9, 11
    out = oracle.yuv420_preprocess_batch_ex(flat, [0], [W * H], [W * H + Wc * Hc], [W], [H],
                                            [(rx, ry, 2 * Cw, 2 * Ch)], 1, Ch, Cw, ZERO, ONE, F32,
                                            oracle.RESIZE_DIRECT, oracle.NHWC, siting)[0]
    rgb = oracle.yuv420_to_rgb_sited(yp, cb, cr, siting)[ry:ry + 2 * Ch, rx:rx + 2 * Cw]
    h = np.float32(0.5)
    p00, p01 = rgb[0::2, 0::2], rgb[0::2, 1::2]
    p10, p11 = rgb[1::2, 0::2], rgb[1::2, 1::2]
    top = p00 + h * (p01 - p00)
    bot = p10 + h * (p11 - p10)
    exp = top + h * (bot - top)
    assert np.array_equal(out, exp)
