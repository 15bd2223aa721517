"""GPU parity of uint8 output and of the low-resolution augmentation
(``smol_lowres_preprocess_batch``, ``smol_yuv420_lowres_preprocess_batch``)
against the oracle (marked gpu; run on an MI355X).

uint8 outputs are a rounding decision both sides take in fp32 on bit-identical
values, so they are compared bit for bit; the augmentation's normalised output
to the fp32 / fp16 bar, and its intermediate r x r images bit for bit.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2007_13005_amd import smol, synthetic
from tests.gpu_util import assert_parity, note, run_gpu, run_oracle, upload

pytestmark = pytest.mark.gpu

F32, F16, U8 = synthetic.OUT_F32, synthetic.OUT_F16, synthetic.OUT_U8
SHORT, DIRECT = smol.RESIZE_SHORT_CROP, smol.RESIZE_DIRECT
NCHW, NHWC = smol.LAYOUT_NCHW, smol.LAYOUT_NHWC


@pytest.fixture(autouse=True)
def _reset_tuning():
    smol.reset_tuning()
    yield
    smol.reset_tuning()


def _check(wl):
    ref = run_oracle(wl)
    got = run_gpu(wl)
    assert got.shape == ref.shape
    stats = assert_parity(got, ref, wl.out_dtype, wl.name)
    note(f"    {wl.name}: {stats} plan={smol.last_plan()}")
    return got, ref


SIZES = [(640, 480), (333, 517), (97, 61), (50, 40), (1920, 1080)]
ROIS = [(101, 37, 300, 250), (0, 0, 150, 517), (0, 0, 97, 61), (49, 39, 1, 1),
        (1620, 780, 300, 300)]


def _rgb(name, sizes, S, C, dtype, mode=SHORT, layout=NCHW, rois=None, seed=31):
    rng = np.random.default_rng(seed)
    imgs = [rng.integers(0, 256, size=(h, w, 3), dtype=np.uint8) for w, h in sizes]
    wl = synthetic.rgb_workload(name, imgs, S, C, dtype)
    wl.rois = None if rois is None else np.asarray(rois, np.int32)
    wl.resize_mode, wl.layout = mode, layout
    return wl


def _yuv(name, sizes, S, C, dtype, mode=SHORT, layout=NCHW, siting=0, seed=32):
    rng = np.random.default_rng(seed)
    planes = []
    for w, h in sizes:
        cw, ch = (w + 1) // 2, (h + 1) // 2
        planes.append((rng.integers(16, 236, size=(h, w), dtype=np.uint8),
                       rng.integers(16, 241, size=(ch, cw), dtype=np.uint8),
                       rng.integers(16, 241, size=(ch, cw), dtype=np.uint8)))
    wl = synthetic.yuv420_workload(name, planes, S, C, dtype)
    wl.resize_mode, wl.layout, wl.siting = mode, layout, siting
    return wl


@pytest.mark.parametrize("C", [(36, 40), (35, 41)], ids=["even", "odd"])
@pytest.mark.parametrize("layout", [NCHW, NHWC])
@pytest.mark.parametrize("path", [smol.PATH_AUTO, smol.PATH_DIRECT, smol.PATH_ROWS])
def test_rgb_u8_short_side_crop(path, layout, C):
    """Even crop widths store pixel pairs as 16-bit words, odd ones byte by
    byte; both kernels that write uint8."""
    smol.set_tuning(path=path)
    _check(_rgb("u8-short", SIZES[:4], 41, C, U8, SHORT, layout))
    want = smol.PATH_DIRECT if path == smol.PATH_DIRECT else smol.PATH_ROWS
    assert smol.last_plan()["path"] == want


@pytest.mark.parametrize("layout", [NCHW, NHWC])
def test_rgb_u8_uniform_frames_row_streaming(layout):
    """A uniform batch of long rows (strided row order for fp16) keeps the
    contiguous order with uint8 output."""
    rng = np.random.default_rng(34)
    batch = rng.integers(0, 256, size=(4, 1080, 1920, 3), dtype=np.uint8)
    wl = synthetic.uniform_rgb_workload("u8-frames", batch, 161, 161, U8)
    wl.layout = layout
    _check(wl)
    assert smol.last_plan()["path"] == smol.PATH_ROWS


@pytest.mark.parametrize("layout", [NCHW, NHWC])
def test_rgb_u8_rois_direct_resize(layout):
    """ROIs touching every edge, up- and downscales, a 1 x 1 ROI."""
    _check(_rgb("u8-roi", SIZES, 1, (57, 43), U8, DIRECT, layout, ROIS))


def test_rgb_u8_same_size_is_the_input():
    """Short side unchanged, whole-image crop: the bytes come back."""
    wl = _rgb("u8-id", [(37, 23)] * 3, 23, (23, 37), U8, SHORT, NHWC)
    got, _ = _check(wl)
    assert np.array_equal(got.reshape(-1), wl.src)


@pytest.mark.parametrize("siting", [smol.CHROMA_CENTER, smol.CHROMA_LEFT])
@pytest.mark.parametrize("layout", [NCHW, NHWC])
def test_yuv_u8(layout, siting):
    _check(_yuv("yuv-u8", [(1280, 720), (641, 359), (33, 21)], 24, (20, 24), U8, SHORT, layout,
                siting))


@pytest.mark.parametrize("path", [smol.PATH_LDS, smol.PATH_GATHER])
def test_u8_forced_tiled_paths_are_unsupported(path):
    smol.set_tuning(path=path)
    with pytest.raises(smol.SmolError):
        run_gpu(_rgb("u8-tiled", SIZES[:2], 40, 32, U8))


def test_yuv_u8_forced_rows_path_is_unsupported():
    smol.set_tuning(path=smol.PATH_ROWS)
    with pytest.raises(smol.SmolError):
        run_gpu(_yuv("yuv-u8-rows", [(64, 48)], 24, 20, U8))


def _lowres(name, sizes, r, S, C, dtype, seed=33):
    wl = _rgb(name, sizes, S, C, dtype, seed=seed)
    wl.low_res = r
    return wl


@pytest.mark.parametrize("dtype", [F32, F16])
@pytest.mark.parametrize("r", [1, 31, 161, 700])
def test_lowres_rgb_ragged(r, dtype):
    """Ragged sizes; r from a single pixel to above every image's short side
    (the reduction then upsamples)."""
    _check(_lowres("lowres", [(640, 480), (333, 517), (97, 61), (300, 600), (1920, 1080)], r,
                   224, 224, dtype))


def test_lowres_intermediate_images_are_exact():
    """The workspace holds the r x r uint8 images of the oracle's reduction."""
    import torch
    r = 57
    wl = _lowres("lowres-ws", [(640, 480), (333, 517), (61, 97)], r, 64, 56, F16)
    _, src = upload(wl)
    p = smol.make_params(wl.resize_short, wl.crop_h, wl.crop_w, wl.mean, wl.std, wl.out_dtype)
    ws = torch.zeros(smol.lowres_workspace_bytes(wl.n, r), dtype=torch.uint8, device="cuda:0")
    out = smol.lowres_preprocess_batch(src, wl.offsets, wl.widths, wl.heights, p, r,
                                       workspace=ws)
    torch.cuda.synchronize()
    low = ws.cpu().numpy()[:wl.n * r * r * 3].reshape(wl.n, r, r, 3)
    exp = oracle.preprocess_batch_ex(wl.src, wl.offsets, wl.widths, wl.heights, None, None, r, r,
                                     r, np.zeros(3), np.ones(3), oracle.OUT_U8,
                                     oracle.RESIZE_SHORT_CROP, oracle.NHWC)
    assert np.array_equal(low, exp)
    assert_parity(out.cpu().numpy(), run_oracle(wl), F16, "lowres-ws")


@pytest.mark.parametrize("dtype", [F32, F16])
def test_lowres_yuv(dtype):
    wl = _yuv("lowres-yuv", [(1280, 720), (641, 359), (300, 600)], 256, 224, dtype)
    wl.low_res = 112
    _check(wl)


def test_lowres_c7_small():
    _check(synthetic.c7(n=16))


def test_lowres_c7_full():
    """The augmentation workload at the size the benchmark runs."""
    wl = synthetic.c7()
    _check(wl)
    # the reduction (row-streaming kernel reading the pinned descriptor
    # table, and the direct kernel for an image whose staged rows would cross
    # the end of src), then the second step
    assert smol.last_plan()["launches"] in (2, 3)
