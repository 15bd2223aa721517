"""GPU parity: the HIP path through the C ABI against the CPU oracle, element
by element, on seeded inputs (marked gpu; run on an MI355X).

Covers the five workloads at full size in the launch configuration the
benchmark uses, both kernel paths (LDS-staged and direct gather) on reduced
batches, and the edge cases: tiny and odd sizes, extreme aspect ratios,
crops that are not multiples of the store width, bands with a ragged tail,
unaligned source pointers and offsets, non-tight pitches, a source buffer
that ends exactly at the last image, determinism, and a non-default stream.
"""
from __future__ import annotations

import numpy as np
import pytest

from paper_2007_13005_amd import smol, synthetic
from tests.gpu_util import assert_parity, note, run_gpu, run_oracle

pytestmark = pytest.mark.gpu

F32, F16 = synthetic.OUT_F32, synthetic.OUT_F16


@pytest.fixture(autouse=True)
def _reset_tuning():
    smol.reset_tuning()
    yield
    smol.reset_tuning()


def _check(wl, **kw):
    ref = run_oracle(wl)
    got = run_gpu(wl, **kw)
    stats = assert_parity(got, ref, wl.out_dtype, wl.name)
    note(f"    {wl.name}: {stats} plan={smol.last_plan()}")
    return got, ref


# ---------------------------------------------------------------------------
# the five workloads, full size, default (benchmark) launch configuration
# ---------------------------------------------------------------------------


_FULL = {}
_REF = {}


def _full(cfg, exact=0):
    """Full-size workload, its oracle output and its GPU output (cached), in
    the default arithmetic or the operation-by-operation one."""
    if (cfg, exact) not in _FULL:
        wl = synthetic.make(cfg)
        if cfg not in _REF:
            _REF[cfg] = run_oracle(wl)
        smol.set_tuning(exact=exact)
        got = run_gpu(wl)
        _FULL[(cfg, exact)] = (wl, _REF[cfg], got, smol.last_plan())
    return _FULL[(cfg, exact)]


@pytest.mark.parametrize("cfg", ["c1", "c2", "c3", "c4", "c5"])
def test_full_config_parity(cfg):
    wl, ref, got, plan = _full(cfg)
    stats = assert_parity(got, ref, wl.out_dtype, wl.name)
    note(f"    {cfg}: {stats} plan={plan}")
    if wl.kind == "rgb":
        assert plan["path"] == smol.PATH_ROWS
    assert plan["uploaded_descriptors"] == (1 if cfg == "c2" else 0)


@pytest.mark.parametrize("cfg", ["c1", "c2", "c3", "c4", "c5"])
def test_full_config_bit_exact(cfg):
    """Stronger than the tolerance: with exact arithmetic selected the kernels
    evaluate the definition's operations in its order with correctly rounded
    results, so every output equals the oracle's bit for bit."""
    wl, ref, got, plan = _full(cfg, exact=1)
    if wl.kind == "rgb":
        assert plan["path"] == smol.PATH_ROWS
    np.testing.assert_array_equal(got.view(np.uint32 if wl.out_dtype == F32 else np.uint16),
                                  ref.view(np.uint32 if wl.out_dtype == F32 else np.uint16))


# ---------------------------------------------------------------------------
# both kernel paths on reduced batches
# ---------------------------------------------------------------------------

SMALL = {"c1": dict(n=6), "c2": dict(n=40), "c3": dict(n=24), "c4": dict(n=3), "c5": dict(n=3)}


@pytest.mark.parametrize("cfg", ["c1", "c2", "c3", "c4"])
@pytest.mark.parametrize("path", [smol.PATH_DIRECT, smol.PATH_LDS, smol.PATH_GATHER,
                                  smol.PATH_ROWS])
def test_rgb_paths(cfg, path):
    smol.set_tuning(path=path)
    wl = synthetic.make(cfg, **SMALL[cfg])
    _check(wl)
    assert smol.last_plan()["path"] == path


@pytest.mark.parametrize("band_rows", [1, 2, 3, 5, 9])
def test_band_rows_with_ragged_tail(band_rows):
    """224 output rows split into bands of R rows (the last band short when R
    does not divide 224)."""
    smol.set_tuning(path=smol.PATH_LDS, band_rows=band_rows, lds_budget=65536)
    wl = synthetic.c2(n=12)
    wl.out_dtype = F32
    _check(wl)
    assert smol.last_plan()["band_rows"] == band_rows


@pytest.mark.parametrize("dtype", [F32, F16])
@pytest.mark.parametrize("sizes,S,C", [
    ([(320, 240)] * 5, 256, 224),       # span 633 B: one 1 KiB chunk group per row
    ([(900, 600), (700, 700)], 256, 224),  # spans 1.6-2.3 KiB: two groups
    ([(1920, 1080)] * 3, 224, 224),     # span 3.2 KiB: four groups
    ([(1200, 400)] * 2, 300, (60, 300)),  # crop 300 wide: four column iterations
], ids=["g1", "g2", "g4", "j4"])
def test_row_streaming_chunk_groups(sizes, S, C, dtype):
    """Staged rows of one, two and four 1 KiB chunk groups, crops needing one
    to four column iterations per lane."""
    smol.set_tuning(path=smol.PATH_ROWS)
    _check(_rgb("groups", sizes, S, C, dtype, seed=11))
    assert smol.last_plan()["path"] == smol.PATH_ROWS


@pytest.mark.parametrize("prefetch", [1, 2])
@pytest.mark.parametrize("cfg", ["c2", "c4"])
def test_row_streaming_prefetch_depths(cfg, prefetch):
    """One or two output rows loaded ahead of the interpolated one."""
    smol.set_tuning(path=smol.PATH_ROWS, band_rows=prefetch)
    _check(synthetic.make(cfg, n=7 if cfg == "c2" else 3))
    assert smol.last_plan()["path"] == smol.PATH_ROWS


@pytest.mark.parametrize("order", [1, 2])
@pytest.mark.parametrize("cfg", ["c1", "c2", "c4", "c5"])
def test_row_streaming_row_orders(cfg, order):
    """Contiguous row ranges and rows interleaved across waves, on uniform
    (incremental vertical taps, wrapping across images) and ragged batches."""
    smol.set_tuning(row_order=order)
    _check(synthetic.make(cfg, n={"c1": 9, "c2": 11, "c4": 3, "c5": 4}[cfg]))
    assert smol.last_plan()["path"] == smol.PATH_ROWS


def test_row_streaming_small_lds_budget():
    """A 1080p span needs 8 KiB of LDS: a 4 KiB budget refuses the forced
    row-streaming plan, the automatic plan takes another kernel."""
    wl = _rgb("budget", [(1920, 1080)] * 2, 224, 224, F16, seed=2)
    smol.set_tuning(path=smol.PATH_ROWS, lds_budget=4096)
    with pytest.raises(smol.SmolError):
        run_gpu(wl)
    smol.set_tuning(lds_budget=4096)
    _check(wl)
    assert smol.last_plan()["path"] != smol.PATH_ROWS


@pytest.mark.parametrize("wg", [1, 2, 5])
def test_row_streaming_few_waves(wg):
    """Few resident waves: each wave walks many rows and several images."""
    smol.set_tuning(path=smol.PATH_ROWS, workgroups_per_cu=wg)
    _check(synthetic.c2(n=30))


def test_row_streaming_single_row_ranges():
    """More waves than rows: ranges of one row (the prologue's second load
    repeats the first row)."""
    smol.set_tuning(path=smol.PATH_ROWS)
    _check(_rgb("one-row", [(64, 48)], 8, (3, 8), F32, seed=12))


def test_c2_aligned_offsets_variant():
    _check(synthetic.c2(n=64, align=256))


# ---------------------------------------------------------------------------
# edge cases
# ---------------------------------------------------------------------------


def _rgb(name, sizes, S, C, out_dtype, seed, align=1, pattern="noise"):
    rng = np.random.default_rng(seed)
    imgs = []
    for w, h in sizes:
        if pattern == "noise":
            imgs.append(rng.integers(0, 256, size=(h, w, 3), dtype=np.uint8))
        else:
            yy, xx = np.mgrid[0:h, 0:w]
            base = (xx * 255 // max(w - 1, 1) + yy * 255 // max(h - 1, 1)) // 2
            imgs.append(np.repeat(base[:, :, None], 3, axis=2).astype(np.uint8))
    return synthetic.rgb_workload(name, imgs, S, C, out_dtype, align)


EDGE = [
    ("1x1", [(1, 1)], 8, 8),
    ("2x2", [(2, 2)], 2, 2),
    ("3x5", [(3, 5)], 4, 3),
    ("identity", [(64, 64)], 64, 64),
    ("2x-down", [(448, 448)], 224, 224),
    ("3x-down", [(21, 21)], 7, 7),
    ("square", [(300, 300)], 256, 224),
    ("extreme-wide", [(2000, 260)], 256, 224),
    ("extreme-tall", [(260, 2000)], 256, 224),
    ("odd-crop", [(640, 480)], 256, (199, 227)),
    ("crop-is-resized", [(50, 37)], 40, (40, 54)),
    ("one-row-crop", [(97, 53)], 30, (1, 30)),
    ("one-col-crop", [(53, 97)], 30, (30, 1)),
    ("upscale-8x", [(16, 12)], 96, 96),
    ("mixed", [(31, 17), (17, 31), (64, 64), (5, 90), (600, 300), (1, 1)], 24, (20, 22)),
]


@pytest.mark.parametrize("dtype", [F32, F16])
@pytest.mark.parametrize("path", [smol.PATH_DIRECT, smol.PATH_AUTO, smol.PATH_GATHER,
                                  smol.PATH_ROWS])
@pytest.mark.parametrize("name,sizes,S,C", EDGE, ids=[e[0] for e in EDGE])
def test_rgb_edge_cases(name, sizes, S, C, path, dtype):
    smol.set_tuning(path=path)
    _check(_rgb(name, sizes, S, C, dtype, seed=len(name)))


@pytest.mark.parametrize("dtype", [F32, F16])
@pytest.mark.parametrize("name,sizes,S,C", EDGE, ids=[e[0] for e in EDGE])
def test_row_streaming_exact_edge_cases(name, sizes, S, C, dtype):
    """Exact arithmetic in the row-streaming kernel: bit-identical to the
    oracle on every edge case."""
    smol.set_tuning(path=smol.PATH_ROWS, exact=1)
    got, ref = _check(_rgb(name, sizes, S, C, dtype, seed=len(name)))
    np.testing.assert_array_equal(got.view(np.uint32 if dtype == F32 else np.uint16),
                                  ref.view(np.uint32 if dtype == F32 else np.uint16))


@pytest.mark.parametrize("path", [smol.PATH_AUTO, smol.PATH_LDS, smol.PATH_ROWS])
def test_wide_spans(path):
    """A crop span too wide to stage in LDS, and wider than the row-streaming
    kernel's 512 columns: forced LDS or row-streaming plans are refused, the
    automatic plan uses the register-gather kernel."""
    smol.set_tuning(path=path)
    wl = _rgb("wide-span", [(20000, 100), (15000, 100)], 100, (2, 12000), F16, seed=3)
    if path in (smol.PATH_LDS, smol.PATH_ROWS):
        with pytest.raises(smol.SmolError):
            run_gpu(wl)
        smol.set_tuning(path=smol.PATH_AUTO)
    _check(wl)
    assert smol.last_plan()["path"] in (smol.PATH_GATHER, smol.PATH_DIRECT)


def test_crop_too_wide_for_gather_tables():
    """Column tap tables of a 30000-wide crop exceed LDS: the automatic plan
    uses the direct kernel, a forced gather plan is refused."""
    wl = _rgb("very-wide", [(31000, 40)], 40, (3, 30000), F32, seed=6)
    _check(wl)
    assert smol.last_plan()["path"] == smol.PATH_DIRECT
    smol.set_tuning(path=smol.PATH_GATHER)
    with pytest.raises(smol.SmolError):
        run_gpu(wl)


def test_gather_prefix_with_direct_tail():
    """In a packed batch the last image's 8-byte windows reach the end of src:
    the gather kernel takes the others and the direct kernel that one."""
    smol.set_tuning(path=smol.PATH_GATHER)
    wl = _rgb("tail", [(128, 128)] * 5, 224, 224, F16, seed=5)
    _check(wl)
    plan = smol.last_plan()
    assert plan["path"] == smol.PATH_GATHER and plan["launches"] == 2


@pytest.mark.parametrize("path", [smol.PATH_AUTO, smol.PATH_GATHER, smol.PATH_ROWS])
def test_image_at_end_of_src_first_in_batch(path):
    """Batch order is the reverse of memory order, so the image whose windows
    reach the end of src comes first: gather and direct launches interleave."""
    import dataclasses
    smol.set_tuning(path=path)
    fwd = _rgb("reversed", [(90, 70), (64, 64), (128, 100), (33, 47)], 48, 40, F16, seed=8)
    wl = dataclasses.replace(fwd, widths=fwd.widths[::-1].copy(),
                             heights=fwd.heights[::-1].copy(), offsets=fwd.offsets[::-1].copy())
    _check(wl)
    assert smol.last_plan()["path"] == (smol.PATH_ROWS if path == smol.PATH_AUTO else path)


@pytest.mark.parametrize("pad", [1, 3, 15])
def test_unaligned_src_pointer(pad):
    wl = synthetic.c1(n=3)
    _check(wl, pad_front=pad)


def test_unaligned_offsets_and_pitch():
    rng = np.random.default_rng(31)
    sizes = [(37, 29), (300, 211), (64, 64), (129, 257)]
    chunks, offs, pitches, cur = [], [], [], 5
    for w, h in sizes:
        p = 3 * w + int(rng.integers(1, 40))
        buf = rng.integers(0, 256, size=(h, p), dtype=np.uint8)
        offs.append(cur)
        pitches.append(p)
        chunks.append(buf.reshape(-1))
        cur += buf.size + int(rng.integers(0, 7))
        chunks.append(rng.integers(0, 256, size=cur - offs[-1] - buf.size, dtype=np.uint8))
    src = np.concatenate([rng.integers(0, 256, size=5, dtype=np.uint8)] + chunks)
    wl = synthetic.Workload("pitched", "rgb", src, np.asarray([w for w, _ in sizes], np.int32),
                            np.asarray([h for _, h in sizes], np.int32), 64, 56, 60, F32,
                            offsets=np.asarray(offs, np.int64),
                            pitches=np.asarray(pitches, np.int32))
    for path in (smol.PATH_DIRECT, smol.PATH_LDS, smol.PATH_GATHER, smol.PATH_ROWS):
        smol.set_tuning(path=path)
        _check(wl)


@pytest.mark.parametrize("path", [smol.PATH_AUTO, smol.PATH_GATHER, smol.PATH_ROWS])
def test_src_ends_at_last_image(path):
    """src_bytes is exactly the packed size (odd), so the last rows' 16-byte
    chunks and 8-byte windows straddle the end of the buffer."""
    smol.set_tuning(path=path)
    wl = _rgb("tight-end", [(33, 21), (41, 20)], 16, 16, F32, seed=4)
    assert wl.src.size % 16 != 0
    _check(wl)


def test_constant_images_are_exact():
    imgs = [np.full((h, w, 3), k, np.uint8) for (w, h), k in [((320, 240), 0), ((97, 301), 131),
                                                              ((1920, 1080), 255)]]
    wl = synthetic.rgb_workload("const", imgs, 224, 224, F32)
    got, _ = _check(wl)
    for i in range(got.shape[0]):
        for c in range(3):
            assert np.all(got[i, c] == got[i, c, 0, 0]), (i, c)


def test_deterministic():
    wl = synthetic.c2(n=16)
    a = run_gpu(wl)
    b = run_gpu(wl)
    np.testing.assert_array_equal(a.view(np.uint16), b.view(np.uint16))


def test_non_default_stream():
    import torch
    s = torch.cuda.Stream()
    wl = synthetic.c3(n=8)
    ref = run_oracle(wl)
    with torch.cuda.stream(s):
        got = run_gpu(wl, stream=s)
    assert_parity(got, ref, wl.out_dtype, "stream")


# ---------------------------------------------------------------------------
# YUV 4:2:0
# ---------------------------------------------------------------------------


def _yuv(name, sizes, S, C, out_dtype, seed, lo=0, hi=256):
    rng = np.random.default_rng(seed)
    planes = []
    for w, h in sizes:
        planes.append((rng.integers(lo, hi, size=(h, w), dtype=np.uint8),
                       rng.integers(lo, hi, size=((h + 1) // 2, (w + 1) // 2), dtype=np.uint8),
                       rng.integers(lo, hi, size=((h + 1) // 2, (w + 1) // 2), dtype=np.uint8)))
    return synthetic.yuv420_workload(name, planes, S, C, out_dtype)


YUV_EDGE = [
    ("1x1", [(1, 1)], 4, 4),
    ("odd", [(33, 21)], 20, (17, 19)),
    ("identity", [(48, 48)], 48, 48),
    ("upscale", [(40, 30)], 120, 112),
    ("ragged", [(1280, 720), (641, 359), (300, 600), (2, 3)], 256, 224),
]


@pytest.mark.parametrize("dtype", [F32, F16])
@pytest.mark.parametrize("path", [smol.PATH_AUTO, smol.PATH_DIRECT, smol.PATH_ROWS])
@pytest.mark.parametrize("name,sizes,S,C", YUV_EDGE, ids=[e[0] for e in YUV_EDGE])
def test_yuv_edge_cases(name, sizes, S, C, path, dtype):
    smol.set_tuning(path=path)
    _check(_yuv(name, sizes, S, C, dtype, seed=len(name)))


@pytest.mark.parametrize("dtype", [F32, F16])
@pytest.mark.parametrize("name,sizes,S,C", YUV_EDGE, ids=[e[0] for e in YUV_EDGE])
def test_yuv_row_streaming_exact(name, sizes, S, C, dtype):
    """Exact arithmetic in the I420 row-streaming kernel: bit-identical to the
    oracle (the frames the direct kernel takes are exact as well)."""
    smol.set_tuning(path=smol.PATH_ROWS, exact=1)
    got, ref = _check(_yuv(name, sizes, S, C, dtype, seed=len(name)))
    np.testing.assert_array_equal(got.view(np.uint32 if dtype == F32 else np.uint16),
                                  ref.view(np.uint32 if dtype == F32 else np.uint16))


# Frames whose row segments all start at one offset per plane (pitches and
# plane offsets multiples of 16: the row kernel's shared-address reads) and
# frames where they do not (luma pitch 1288: consecutive luma rows 8 bytes
# apart in their chunks; chroma pitch 648 likewise), alone and mixed in one
# ragged batch.
YUV_OFFSETS = [
    ("same", [(1280, 720)]),
    ("luma-mixed", [(1288, 720)]),
    ("chroma-mixed", [(1296, 720)]),
    ("all", [(1280, 720), (1288, 720), (1296, 720), (1280, 720)]),
]


@pytest.mark.parametrize("dtype", [F32, F16])
@pytest.mark.parametrize("name,sizes", YUV_OFFSETS, ids=[e[0] for e in YUV_OFFSETS])
def test_yuv_row_segment_offsets_exact(name, sizes, dtype):
    smol.set_tuning(path=smol.PATH_ROWS, exact=1)
    got, ref = _check(_yuv(name, sizes, 256, 224, dtype, seed=len(name)))
    np.testing.assert_array_equal(got.view(np.uint32 if dtype == F32 else np.uint16),
                                  ref.view(np.uint32 if dtype == F32 else np.uint16))


@pytest.mark.parametrize("cb,cr", [(0, 255), (255, 0), (0, 0), (255, 255)])
def test_yuv_extreme_chroma_exact(cb, cr):
    """Chroma planes at 0 and 255: the chroma sums at their extremes (16 x
    (0 - 128) and 16 x (255 - 128)), where the row kernel's conversion of the
    sum to fp32 must still be exact; bit-identical to the oracle."""
    rng = np.random.default_rng(cb * 7 + cr)
    planes = []
    for w, h in [(1280, 720), (641, 359)]:
        ch, cw = (h + 1) // 2, (w + 1) // 2
        planes.append((rng.integers(0, 256, size=(h, w), dtype=np.uint8),
                       np.full((ch, cw), cb, np.uint8), np.full((ch, cw), cr, np.uint8)))
    smol.set_tuning(path=smol.PATH_ROWS, exact=1)
    got, ref = _check(synthetic.yuv420_workload("extreme", planes, 256, 224, F32))
    np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("path", [smol.PATH_AUTO, smol.PATH_ROWS])
def test_yuv_frame_at_end_of_src_first_in_batch(path):
    """Batch order reverses memory order: the frame whose planes end at the
    end of src comes first, so direct and row-streaming launches alternate."""
    import dataclasses
    smol.set_tuning(path=path)
    fwd = _yuv("rev", [(96, 64), (130, 90), (64, 64)], 48, 40, F16, seed=9)
    rev = lambda x: x[::-1].copy()
    wl = dataclasses.replace(fwd, widths=rev(fwd.widths), heights=rev(fwd.heights),
                             y_offsets=rev(fwd.y_offsets), cb_offsets=rev(fwd.cb_offsets),
                             cr_offsets=rev(fwd.cr_offsets))
    _check(wl)
    assert smol.last_plan()["path"] == smol.PATH_ROWS


def test_yuv_wide_span_uses_direct_kernel():
    """A luma span past 2016 bytes: forced row streaming is refused, the
    automatic plan uses the direct kernel."""
    wl = _yuv("wide", [(12000, 100)], 20, (2, 450), F32, seed=10)
    smol.set_tuning(path=smol.PATH_ROWS)
    with pytest.raises(smol.SmolError):
        run_gpu(wl)
    smol.set_tuning(path=smol.PATH_AUTO)
    _check(wl)
    assert smol.last_plan()["path"] == smol.PATH_DIRECT


@pytest.mark.parametrize("dtype", [F32, F16])
def test_yuv_long_luma_rows_stream(dtype):
    """1080p frames at short side 224: luma spans of 1,078 bytes take the
    row-streaming kernel's two-chunk luma segments (and spans of 992 to 2016
    bytes in general, here also a ragged second frame)."""
    wl = _yuv("hd", [(1920, 1080), (1500, 900)], 224, 224, dtype, seed=12)
    _check(wl)
    assert smol.last_plan()["path"] == smol.PATH_ROWS


def test_yuv_neutral_chroma_equals_rgb_path_on_gpu():
    rng = np.random.default_rng(41)
    y = rng.integers(0, 256, size=(123, 201), dtype=np.uint8)
    c = np.full((62, 101), 128, np.uint8)
    wy = synthetic.yuv420_workload("neutral", [(y, c, c)], 100, 90, F32)
    wr = synthetic.rgb_workload("grey", [np.repeat(y[:, :, None], 3, axis=2)], 100, 90, F32)
    a = run_gpu(wy)
    b = run_gpu(wr)
    assert_parity(a, b, F32, "yuv-vs-rgb")
