"""Host entropy decoding (``smol_jpeg_entropy_decode_batch``, T.81 Annex F)
against the oracle's decoder, bit for bit: whole streams, restart intervals,
partial decoding of rectangles (only the MCUs the rectangle spans are
written; restart intervals before it are skipped), thread counts, and the
error paths. Host code only: these run without a GPU."""
from __future__ import annotations

import ctypes
import io

import numpy as np
import pytest

import oracle
from paper_2007_13005_amd import smol, synthetic

SIZES = [(203, 77), (64, 48), (33, 21), (1, 1), (17, 3), (640, 480), (16, 16), (31, 47),
         (1280, 720)]
SENTINEL = 0x5A5A


def _decode_raw(files, rects=None, threads=0, fill=SENTINEL, layout=smol.JPEG_COEF_FRAME):
    """The C call on a sentinel-filled buffer: (rc, message, coef, offsets,
    qtables)."""
    n = len(files)
    sizes = np.asarray([len(f) for f in files], np.int64)
    offs = np.concatenate([[0], np.cumsum(sizes)[:-1]]).astype(np.int64)
    data = np.frombuffer(b"".join(files), np.uint8)
    counts = []
    for k, f in enumerate(files):
        try:
            i = smol.jpeg_read_info(f)
            counts.append(smol.jpeg_window_coef_count(i.width, i.height, rects[k])
                          if layout == smol.JPEG_COEF_WINDOW else
                          smol.jpeg_coef_count(i.width, i.height))
        except smol.SmolError:
            counts.append(64)
    co = np.concatenate([[0], np.cumsum(counts)[:-1]]).astype(np.int64)
    coef = np.full(int(np.sum(counts)), fill, np.int16)
    q = np.zeros((n, 2, 64), np.uint16)
    r = None if rects is None else np.ascontiguousarray(rects, np.int32)
    rc = smol.lib().smol_jpeg_entropy_decode_batch(
        data.ctypes.data, data.size, offs.ctypes.data, sizes.ctypes.data, n,
        None if r is None else r.ctypes.data, coef.ctypes.data, coef.size, co.ctypes.data,
        layout, q.ctypes.data, threads)
    return rc, smol.lib().smol_last_error().decode(), coef, co, q


def _blocks(c, W, H):
    """Per-component block arrays (luma (bh, bw, 64), Cb and Cr (bh/2, bw/2,
    64)) of one frame's coefficients."""
    bw, bh = 2 * ((W + 15) // 16), 2 * ((H + 15) // 16)
    y = c[:64 * bw * bh].reshape(bh, bw, 64)
    k = 64 * (bw // 2) * (bh // 2)
    cb = c[64 * bw * bh:64 * bw * bh + k].reshape(bh // 2, bw // 2, 64)
    cr = c[64 * bw * bh + k:64 * bw * bh + 2 * k].reshape(bh // 2, bw // 2, 64)
    return y, cb, cr


@pytest.mark.parametrize("restart", [0, 1, 5, 40])
def test_whole_streams_bit_exact(restart):
    files = synthetic.jpeg_files(SIZES, 80 + restart, [50, 75, 90, 95, 75, 60, 100, 85, 75],
                                 restart_blocks=restart)
    rc, msg, coef, co, q = _decode_raw(files, threads=4)
    assert rc == 0, msg
    for i, f in enumerate(files):
        c, qy, qc, W, H = oracle.jpeg_entropy_decode(f)
        info = smol.jpeg_read_info(f)
        assert (info.width, info.height, info.restart_interval) == (W, H, restart)
        assert np.array_equal(coef[co[i]:co[i] + c.size], c), (i, SIZES[i])
        assert np.array_equal(q[i, 0], qy) and np.array_equal(q[i, 1], qc)


def _random_rects(rng, sizes):
    out = []
    for W, H in sizes:
        x, y = int(rng.integers(0, W)), int(rng.integers(0, H))
        out.append((x, y, int(rng.integers(1, W - x + 1)), int(rng.integers(1, H - y + 1))))
    return out


@pytest.mark.parametrize("restart", [0, 1, 3])
def test_partial_streams_write_only_their_mcus(restart):
    rng = np.random.default_rng(90 + restart)
    files = synthetic.jpeg_files(SIZES, 90, 75, restart_blocks=restart)
    rects = _random_rects(rng, SIZES)
    rc, msg, coef, co, _ = _decode_raw(files, rects, threads=3)
    assert rc == 0, msg
    for i, f in enumerate(files):
        c, _, _, W, H = oracle.jpeg_entropy_decode(f)
        x, y, w, h = rects[i]
        mx0, mx1, my0, my1 = x // 16, (x + w - 1) // 16, y // 16, (y + h - 1) // 16
        got, exp = _blocks(coef[co[i]:co[i] + c.size], W, H), _blocks(c, W, H)
        inside = (slice(2 * my0, 2 * my1 + 2), slice(2 * mx0, 2 * mx1 + 2))
        assert np.array_equal(got[0][inside], exp[0][inside]), (i, rects[i])
        for k in (1, 2):
            sl = (slice(my0, my1 + 1), slice(mx0, mx1 + 1))
            assert np.array_equal(got[k][sl], exp[k][sl]), (i, rects[i], k)
        # everything else untouched
        mask = np.ones(got[0].shape[:2], bool)
        mask[inside] = False
        assert (got[0][mask] == SENTINEL).all(), (i, rects[i])


@pytest.mark.parametrize("restart", [0, 3])
def test_window_layout_holds_the_mcu_window(restart):
    """The window layout stores exactly the frame layout's blocks of the
    rectangle's MCU window, packed."""
    rng = np.random.default_rng(96 + restart)
    files = synthetic.jpeg_files(SIZES, 96, 75, restart_blocks=restart)
    rects = _random_rects(rng, SIZES)
    rc, msg, coef, co, _ = _decode_raw(files, rects, threads=3, layout=smol.JPEG_COEF_WINDOW)
    assert rc == 0, msg
    for i, f in enumerate(files):
        c, _, _, W, H = oracle.jpeg_entropy_decode(f)
        x, y, w, h = rects[i]
        mx0, mx1, my0, my1 = x // 16, (x + w - 1) // 16, y // 16, (y + h - 1) // 16
        nx, ny = mx1 - mx0 + 1, my1 - my0 + 1
        exp = _blocks(c, W, H)
        k = smol.jpeg_window_coef_count(W, H, rects[i])
        assert k == 64 * 6 * nx * ny
        win = coef[co[i]:co[i] + k]
        luma = win[:64 * 4 * nx * ny].reshape(2 * ny, 2 * nx, 64)
        cb = win[64 * 4 * nx * ny:64 * 5 * nx * ny].reshape(ny, nx, 64)
        cr = win[64 * 5 * nx * ny:].reshape(ny, nx, 64)
        assert np.array_equal(luma, exp[0][2 * my0:2 * my1 + 2, 2 * mx0:2 * mx1 + 2]), i
        assert np.array_equal(cb, exp[1][my0:my1 + 1, mx0:mx1 + 1]), i
        assert np.array_equal(cr, exp[2][my0:my1 + 1, mx0:mx1 + 1]), i


def test_algorithm1_rectangles_feed_the_block_decoder():
    """With Algorithm 1's rectangles, the partial entropy decode followed by
    the oracle's partial block decode equals the whole decode on every pixel
    the rectangle holds."""
    sizes = [(640, 480), (1280, 720), (333, 517)]
    files = synthetic.jpeg_files(sizes, 91, 80, restart_blocks=2)
    p = smol.make_params(256, 224, 224, [0, 0, 0], [1, 1, 1], smol.OUT_F16)
    rects = [smol.jpeg_mcu_rect(W, H, p) for W, H in sizes]
    rc, msg, coef, co, q = _decode_raw(files, rects, fill=0)
    assert rc == 0, msg
    for i, f in enumerate(files):
        c, qy, qc, W, H = oracle.jpeg_entropy_decode(f)
        x, y, w, h = rects[i]
        part = oracle.jpeg_decode_i420(coef[co[i]:co[i] + c.size], q[i, 0], q[i, 1], W, H,
                                       rects[i], fill=0)
        full = oracle.jpeg_decode_i420(c, qy, qc, W, H)
        assert np.array_equal(part[0][y:y + h, x:x + w], full[0][y:y + h, x:x + w])
        cs = (slice(y // 2, (y + h - 1) // 2 + 1), slice(x // 2, (x + w - 1) // 2 + 1))
        assert np.array_equal(part[1][cs], full[1][cs]) and np.array_equal(part[2][cs],
                                                                          full[2][cs])


def test_thread_counts_agree():
    files = synthetic.jpeg_files(SIZES * 3, 92, 70)
    ref = _decode_raw(files, threads=1)
    assert ref[0] == 0, ref[1]
    for t in (2, 7, 64, 0, -1):
        got = _decode_raw(files, threads=t)
        assert got[0] == 0 and np.array_equal(got[2], ref[2]), t


def test_binding_returns_batch():
    files = synthetic.jpeg_files([(64, 48), (33, 21)], 93, [60, 90])
    b = smol.jpeg_entropy_decode_batch(files)
    assert b.n == 2 and list(b.widths) == [64, 33] and list(b.heights) == [48, 21]
    assert b.qtables.shape == (2, 2, 64) and not np.array_equal(b.qtables[0], b.qtables[1])


def _encode(mode="YCbCr", **kw) -> bytes:
    from PIL import Image
    im = Image.fromarray(synthetic.photo_ycbcr(np.random.default_rng(3), 48, 32), "YCbCr")
    if mode == "L":
        im = im.getchannel(0)
    b = io.BytesIO()
    im.save(b, "JPEG", **kw)
    return b.getvalue()


@pytest.mark.parametrize("data,code,needle", [
    (_encode(progressive=True, subsampling=2), smol.ERR_UNSUPPORTED, "progressive"),
    (_encode(subsampling=0), smol.ERR_UNSUPPORTED, "4:2:0"),
    (_encode(subsampling=1), smol.ERR_UNSUPPORTED, "4:2:0"),
    (_encode("L"), smol.ERR_UNSUPPORTED, "components"),
    (_encode(subsampling=2)[:300], smol.ERR_INVALID_ARG, ""),
    (_encode(subsampling=2)[:-60], smol.ERR_INVALID_ARG, "ends inside"),
    (b"\x00" + _encode(subsampling=2)[1:], smol.ERR_INVALID_ARG, "SOI"),
])
def test_streams_outside_the_subset_fail(data, code, needle):
    good = _encode(subsampling=2)
    rc, msg, *_ = _decode_raw([good, data])
    assert rc == code and msg.startswith("image 1:") and needle in msg, (rc, msg)


def test_argument_errors():
    f = synthetic.jpeg_files([(16, 16)], 94, 75)[0]
    data = np.frombuffer(f, np.uint8)
    coef = np.zeros(smol.jpeg_coef_count(16, 16), np.int16)
    z = np.zeros(1, np.int64)

    def call(size=len(f), coef_elems=coef.size, n=1, rect=None, layout=0):
        s = np.asarray([size], np.int64)
        r = None if rect is None else np.asarray(rect, np.int32)
        rc = smol.lib().smol_jpeg_entropy_decode_batch(
            data.ctypes.data, data.size, z.ctypes.data, s.ctypes.data, n,
            None if r is None else r.ctypes.data, coef.ctypes.data, coef_elems, z.ctypes.data,
            layout, None, 1)
        return rc, smol.lib().smol_last_error().decode()

    assert call()[0] == 0
    assert call(size=len(f) + 1) == (smol.ERR_INVALID_ARG, "image 0: stream outside data")
    rc, msg = call(coef_elems=coef.size - 1)
    assert rc == smol.ERR_INVALID_ARG and "outside coef" in msg
    rc, msg = call(rect=(8, 8, 9, 8))
    assert rc == smol.ERR_INVALID_ARG and "rectangle" in msg
    rc, msg = call(layout=1)
    assert rc == smol.ERR_INVALID_ARG and "needs rects" in msg
    rc, msg = call(layout=3, rect=(0, 0, 16, 16))
    assert rc == smol.ERR_INVALID_ARG and "coef_layout 3" in msg
    assert call(layout=1, rect=(0, 0, 16, 16), coef_elems=6 * 64)[0] == 0
    rc, msg = call(layout=1, rect=(0, 0, 16, 16), coef_elems=6 * 64 - 1)
    assert rc == smol.ERR_INVALID_ARG and "outside coef" in msg
    assert call(n=-1)[0] == smol.ERR_INVALID_ARG
    assert call(n=0)[0] == 0
    info = smol.JpegInfo()
    assert smol.lib().smol_jpeg_read_info(None, 0, ctypes.byref(info)) == smol.ERR_INVALID_ARG


def test_corrupt_streams_fail_cleanly():
    """Bytes flipped inside the scan: the library accepts exactly the
    streams the oracle accepts (some flips still leave a decodable bit
    sequence) and then yields the oracle's coefficients; it never reads or
    writes out of bounds."""
    rng = np.random.default_rng(95)
    base = synthetic.jpeg_files([(96, 64)], 95, 75, restart_blocks=2)[0]
    scan = smol.jpeg_read_info(base).scan_offset
    counts = {True: 0, False: 0}
    for _ in range(200):
        b = bytearray(base)
        for _ in range(int(rng.integers(1, 4))):
            b[int(rng.integers(scan, len(b) - 2))] = int(rng.integers(0, 256))
        b = bytes(b)
        rc, msg, coef, co, _ = _decode_raw([b], fill=0)
        try:
            c = oracle.jpeg_entropy_decode(b)[0]
        except ValueError:
            c = None
        assert (rc == 0) == (c is not None), msg
        if c is not None:
            assert np.array_equal(coef[:c.size], c)
        counts[c is not None] += 1
    assert counts[True] >= 20 and counts[False] >= 20, counts


def test_widest_and_tallest_streams_bit_exact():
    """libjpeg's largest sizes, 65500 x 17 and 17 x 65500, with restart
    intervals of 100 MCUs, whole and through narrow rectangles at the far
    end (most intervals skipped)."""
    sizes = [(65500, 17), (17, 65500)]
    files = synthetic.jpeg_files(sizes, 111, 75, restart_blocks=100)
    rects = [(65400, 2, 60, 13), (3, 65400, 12, 90)]
    for rr in (None, rects):
        rc, msg, coef, co, _ = _decode_raw(files, rr, threads=2)
        assert rc == 0, msg
        for i, f in enumerate(files):
            c, _, _, W, H = oracle.jpeg_entropy_decode(f)
            got, exp = _blocks(coef[co[i]:co[i] + c.size], W, H), _blocks(c, W, H)
            if rr is None:
                assert np.array_equal(coef[co[i]:co[i] + c.size], c), sizes[i]
                continue
            x, y, w, h = rr[i]
            sl = (slice(2 * (y // 16), 2 * ((y + h - 1) // 16) + 2),
                  slice(2 * (x // 16), 2 * ((x + w - 1) // 16) + 2))
            assert np.array_equal(got[0][sl], exp[0][sl]), sizes[i]
