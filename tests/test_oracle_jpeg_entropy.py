"""Pins of the oracle's baseline JPEG entropy decoding (ITU-T T.81, Annex F;
the CPU step ahead of section 6.4's partial decode) against what neither the
oracle nor this library wrote: libjpeg, through PIL, as the encoder of every
stream and as an independent decoder, and the closed form of the DCT of a
constant block.

- Tables: PIL takes quantisation tables in natural order and the stream
  stores them in zig-zag order, so reading back the tables given to the
  encoder pins the oracle's zig-zag.
- Pixels: libjpeg's own decode (its integer inverse DCT is within one level
  of the exact transform) agrees with the oracle's coefficients passed
  through the oracle's exact inverse DCT to within two levels, nearly all
  exactly; chroma compared after libjpeg's triangle (3:1) upsampling,
  rebuilt here as bilinear interpolation with centred samples.
- Restart intervals change the stream, not the coefficients.
- A block-constant image at quality 100 (all table entries 1) decodes to
  DC = 8 (level - 128) and no AC terms: the DCT of a constant block.
"""
from __future__ import annotations

import io

import numpy as np
import pytest

import oracle
from paper_2007_13005_amd import synthetic

SIZES = [(203, 77), (64, 48), (33, 21), (1, 1), (17, 3), (640, 480), (16, 16), (31, 47)]


def _libjpeg_ycbcr(data: bytes) -> np.ndarray:
    from PIL import Image
    im = Image.open(io.BytesIO(data))
    im.draft("YCbCr", im.size)
    assert im.mode == "YCbCr"
    return np.asarray(im).astype(np.int64)


def _centred_upsample(c: np.ndarray, W: int, H: int) -> np.ndarray:
    """Bilinear 2x upsampling with centred samples, clamped at the edges:
    output sample x sits at chroma coordinate (x + 1/2)/2 - 1/2."""
    Hc, Wc = c.shape
    xs, ys = (np.arange(W) + 0.5) / 2 - 0.5, (np.arange(H) + 0.5) / 2 - 0.5
    x0, y0 = np.floor(xs).astype(int), np.floor(ys).astype(int)
    fx, fy = xs - x0, (ys - y0)[:, None]
    cx0, cx1 = np.clip(x0, 0, Wc - 1), np.clip(x0 + 1, 0, Wc - 1)
    cy0, cy1 = np.clip(y0, 0, Hc - 1), np.clip(y0 + 1, 0, Hc - 1)
    c = c.astype(np.float64)
    r0 = c[cy0][:, cx0] * (1 - fx) + c[cy0][:, cx1] * fx
    r1 = c[cy1][:, cx0] * (1 - fx) + c[cy1][:, cx1] * fx
    return r0 * (1 - fy) + r1 * fy


def test_tables_come_back_in_natural_order():
    from PIL import Image
    img = synthetic.photo_ycbcr(np.random.default_rng(1), 40, 24)
    q0 = list(range(1, 65))
    q1 = [200 - 3 * i for i in range(64)]
    b = io.BytesIO()
    Image.fromarray(img, "YCbCr").save(b, "JPEG", qtables=[q0, q1], subsampling=2)
    _, qy, qc, W, H = oracle.jpeg_entropy_decode(b.getvalue())
    assert (W, H) == (40, 24)
    assert qy.tolist() == q0 and qc.tolist() == q1


@pytest.mark.parametrize("quality", [50, 75, 95])
def test_pixels_agree_with_libjpeg(quality):
    files = synthetic.jpeg_files(SIZES, 60 + quality, quality)
    for (W, H), data in zip(SIZES, files):
        coef, qy, qc, w, h = oracle.jpeg_entropy_decode(data)
        assert (w, h) == (W, H)
        y, cb, cr = oracle.jpeg_decode_i420(coef, qy, qc, W, H)
        ref = _libjpeg_ycbcr(data)
        d = np.abs(y.astype(np.int64) - ref[..., 0])
        assert d.max() <= 2 and (d == 0).mean() >= 0.95, ((W, H), d.max(), (d == 0).mean())
        for k, c in ((1, cb), (2, cr)):
            e = np.abs(_centred_upsample(c, W, H) - ref[..., k])
            assert e.max() <= 2.0 and e.mean() < 0.5, ((W, H), k, e.max(), e.mean())


@pytest.mark.parametrize("blocks", [1, 3, 7])
def test_restart_intervals_change_nothing(blocks):
    sizes = [(203, 77), (640, 480), (33, 21)]
    plain = synthetic.jpeg_files(sizes, 70, 80)
    marked = synthetic.jpeg_files(sizes, 70, 80, restart_blocks=blocks)
    for a, b in zip(plain, marked):
        assert a != b and b.count(b"\xff\xdd") == 1
        ca, cb_ = oracle.jpeg_entropy_decode(a), oracle.jpeg_entropy_decode(b)
        assert np.array_equal(ca[0], cb_[0])


def test_block_constant_image_is_dc_only():
    from PIL import Image
    rng = np.random.default_rng(5)
    W, H = 48, 32
    levels = rng.integers(0, 256, size=(H // 16, W // 16, 3))
    img = np.repeat(np.repeat(levels, 16, 0), 16, 1).astype(np.uint8)
    b = io.BytesIO()
    Image.fromarray(img, "YCbCr").save(b, "JPEG", quality=100, subsampling=2)
    coef, qy, qc, w, h = oracle.jpeg_entropy_decode(b.getvalue())
    assert (qy == 1).all() and (qc == 1).all()
    bw, bh = 2 * ((W + 15) // 16), 2 * ((H + 15) // 16)
    blk = coef.reshape(-1, 64)
    luma, cb, cr = blk[:bw * bh], blk[bw * bh:bw * bh + bw * bh // 4], blk[bw * bh + bw * bh // 4:]
    assert not luma[:, 1:].any() and not cb[:, 1:].any() and not cr[:, 1:].any()
    lv = np.repeat(np.repeat(levels[..., 0], 2, 0), 2, 1).reshape(-1)
    assert np.array_equal(luma[:, 0], 8 * (lv.astype(np.int64) - 128))
    assert np.array_equal(cb[:, 0], 8 * (levels[..., 1].reshape(-1).astype(np.int64) - 128))
    assert np.array_equal(cr[:, 0], 8 * (levels[..., 2].reshape(-1).astype(np.int64) - 128))


def _encode(mode="YCbCr", **kw) -> bytes:
    from PIL import Image
    img = synthetic.photo_ycbcr(np.random.default_rng(3), 48, 32)
    im = Image.fromarray(img, "YCbCr")
    if mode == "L":
        im = im.getchannel(0)
    b = io.BytesIO()
    im.save(b, "JPEG", **kw)
    return b.getvalue()


@pytest.mark.parametrize("data", [
    _encode(progressive=True, subsampling=2),   # progressive (SOF2)
    _encode(subsampling=0),                     # 4:4:4
    _encode(subsampling=1),                     # 4:2:2
    _encode("L"),                               # one component
    _encode(subsampling=2)[:300],               # cut inside the headers
    _encode(subsampling=2)[:-60],               # cut inside the scan
    b"\x00" + _encode(subsampling=2)[1:],        # no SOI
])
def test_rejects_streams_outside_the_subset(data):
    with pytest.raises(ValueError):
        oracle.jpeg_entropy_decode(data)
