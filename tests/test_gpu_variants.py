"""GPU parity of the variants -- region of interest per image, direct resize,
channels-last output, co-sited chroma -- through the C ABI's _ex calls
against the oracle (marked gpu; run on an MI355X).

Covers every RGB kernel path with ROIs (the ROI is folded into the image
descriptor), the row-streaming and direct kernels with NHWC output (even and
odd crop widths, fp16 and fp32), I420 ROIs at odd frame coordinates with both
chroma sitings on both I420 kernels, uniform and ragged ROI tables, ROIs that
touch every edge of their image, and the detection-crop workload c6.
"""
from __future__ import annotations

import numpy as np
import pytest

from paper_2007_13005_amd import smol, synthetic
from tests.gpu_util import assert_parity, note, run_gpu, run_oracle

pytestmark = pytest.mark.gpu

F32, F16 = synthetic.OUT_F32, synthetic.OUT_F16
SHORT, DIRECT = smol.RESIZE_SHORT_CROP, smol.RESIZE_DIRECT
NCHW, NHWC = smol.LAYOUT_NCHW, smol.LAYOUT_NHWC


@pytest.fixture(autouse=True)
def _reset_tuning():
    smol.reset_tuning()
    yield
    smol.reset_tuning()


def _check(wl, **kw):
    ref = run_oracle(wl)
    got = run_gpu(wl, **kw)
    assert got.shape == wl.out_shape()
    stats = assert_parity(got, ref, wl.out_dtype, wl.name)
    note(f"    {wl.name}: {stats} plan={smol.last_plan()}")
    return got, ref


def _rgb(name, sizes, rois, S, C, out_dtype, mode, layout, seed=1):
    rng = np.random.default_rng(seed)
    imgs = [rng.integers(0, 256, size=(h, w, 3), dtype=np.uint8) for w, h in sizes]
    wl = synthetic.rgb_workload(name, imgs, S, C, out_dtype)
    wl.rois = None if rois is None else np.asarray(rois, np.int32)
    wl.resize_mode, wl.layout = mode, layout
    return wl


def _yuv(name, sizes, rois, S, C, out_dtype, mode, layout, siting, seed=2):
    rng = np.random.default_rng(seed)
    planes = []
    for w, h in sizes:
        cw, ch = (w + 1) // 2, (h + 1) // 2
        planes.append((rng.integers(0, 256, size=(h, w), dtype=np.uint8),
                       rng.integers(0, 256, size=(ch, cw), dtype=np.uint8),
                       rng.integers(0, 256, size=(ch, cw), dtype=np.uint8)))
    wl = synthetic.yuv420_workload(name, planes, S, C, out_dtype)
    wl.rois = None if rois is None else np.asarray(rois, np.int32)
    wl.resize_mode, wl.layout, wl.siting = mode, layout, siting
    return wl


# ROIs of ragged images: interior, touching each edge, the whole image, 1 px
RGB_SIZES = [(640, 480), (333, 517), (1920, 1080), (97, 61), (50, 40)]
RGB_ROIS = [(101, 37, 300, 250), (0, 0, 150, 517), (1620, 780, 300, 300), (0, 0, 97, 61),
            (49, 39, 1, 1)]


@pytest.mark.parametrize("dtype", [F32, F16])
@pytest.mark.parametrize("path", [smol.PATH_AUTO, smol.PATH_DIRECT, smol.PATH_LDS,
                                  smol.PATH_GATHER, smol.PATH_ROWS])
def test_rgb_roi_direct_resize_nchw_all_paths(path, dtype):
    smol.set_tuning(path=path)
    _check(_rgb("roi-direct", RGB_SIZES, RGB_ROIS, 1, (72, 80), dtype, DIRECT, NCHW))


@pytest.mark.parametrize("dtype", [F32, F16])
@pytest.mark.parametrize("path", [smol.PATH_AUTO, smol.PATH_DIRECT, smol.PATH_ROWS])
@pytest.mark.parametrize("C", [(64, 96), (33, 45)], ids=["even", "odd"])
def test_rgb_roi_nhwc(C, path, dtype):
    """NHWC on the row-streaming and direct kernels: even widths store whole
    pixel pairs, odd widths element by element."""
    smol.set_tuning(path=path)
    _check(_rgb("roi-nhwc", RGB_SIZES, RGB_ROIS, 1, C, dtype, DIRECT, NHWC))


@pytest.mark.parametrize("layout", [NCHW, NHWC])
def test_rgb_roi_short_side_crop(layout):
    """ROI then the standard pipeline (short side 96, centre crop 80 x 88)."""
    rois = [(101, 37, 300, 250), (0, 0, 150, 517), (1620, 780, 300, 300), (0, 0, 97, 88),
            (0, 0, 50, 40)]
    sizes = RGB_SIZES[:3] + [(97, 88), (50, 40)]
    _check(_rgb("roi-short", sizes, rois, 96, (80, 88), F16, SHORT, layout))


@pytest.mark.parametrize("layout", [NCHW, NHWC])
def test_rgb_direct_resize_whole_images(layout):
    """Direct resize without ROIs, up and down, extreme aspect."""
    _check(_rgb("direct", [(1920, 1080), (64, 300), (7, 5)], None, 1, (112, 112), F16, DIRECT,
                layout))


def test_rgb_uniform_roi_batch_uses_uniform_descriptor():
    """The same ROI in equal frames: a uniform batch (no descriptor upload)."""
    wl = _rgb("uniform-roi", [(800, 600)] * 6, [(120, 90, 400, 300)] * 6, 1, (112, 112), F16,
              DIRECT, NHWC)
    _check(wl)
    assert smol.last_plan()["uploaded_descriptors"] == 0


def test_rgb_nhwc_matches_nchw_transpose_on_gpu():
    """With exact arithmetic both layouts hold the oracle's bits, so one is the
    other's transpose. (By default the fp16 conversion may or may not fuse
    with the last product, which each kernel's compiler decides: the layouts
    then agree within the 1-ulp bar, not bit for bit.)"""
    smol.set_tuning(exact=1)
    a = _rgb("t", RGB_SIZES, RGB_ROIS, 1, (72, 80), F16, DIRECT, NCHW)
    b = _rgb("t", RGB_SIZES, RGB_ROIS, 1, (72, 80), F16, DIRECT, NHWC)
    ga, gb = run_gpu(a), run_gpu(b)
    np.testing.assert_array_equal(np.transpose(ga, (0, 2, 3, 1)).view(np.uint16),
                                  gb.view(np.uint16))


def test_rgb_nhwc_forced_gather_is_unsupported():
    smol.set_tuning(path=smol.PATH_GATHER)
    with pytest.raises(smol.SmolError):
        run_gpu(_rgb("nhwc-gather", RGB_SIZES, RGB_ROIS, 1, (64, 64), F16, DIRECT, NHWC))


YUV_SIZES = [(1280, 720), (641, 359), (300, 600), (33, 21)]
YUV_ROIS = [(301, 117, 400, 300), (1, 1, 639, 357), (0, 3, 300, 597), (32, 20, 1, 1)]


@pytest.mark.parametrize("siting", [smol.CHROMA_CENTER, smol.CHROMA_LEFT])
@pytest.mark.parametrize("layout", [NCHW, NHWC])
@pytest.mark.parametrize("path", [smol.PATH_AUTO, smol.PATH_DIRECT, smol.PATH_ROWS])
def test_yuv_roi_sitings(path, layout, siting):
    """I420 ROIs at odd frame coordinates: chroma taps in frame coordinates,
    clamped at the frame, sited as asked; both I420 kernels."""
    smol.set_tuning(path=path)
    _check(_yuv("yuv-roi", YUV_SIZES, YUV_ROIS, 1, (56, 72), F16, DIRECT, layout, siting))


@pytest.mark.parametrize("dtype", [F32, F16])
def test_yuv_roi_short_side_left_siting(dtype):
    rois = [(301, 117, 400, 300), (1, 1, 639, 357), (0, 3, 300, 597), (4, 2, 29, 19)]
    _check(_yuv("yuv-roi-short", YUV_SIZES, rois, 64, (48, 56), dtype, SHORT, NCHW,
                smol.CHROMA_LEFT))


def test_yuv_uniform_roi_batch():
    wl = _yuv("yuv-uniform-roi", [(1280, 720)] * 4, [(333, 101, 501, 401)] * 4, 1, (112, 112),
              F16, DIRECT, NHWC, smol.CHROMA_LEFT)
    _check(wl)
    assert smol.last_plan()["uploaded_descriptors"] == 0


def test_yuv_left_siting_whole_frames_nchw():
    """Co-sited chroma alone (no ROI, standard pipeline)."""
    _check(_yuv("yuv-left", [(1280, 720), (641, 359)], None, 256, 224, F16, SHORT, NCHW,
                smol.CHROMA_LEFT))


def test_detection_crops_c6_small():
    """The detection-crop workload at a reduced size (32 ROIs)."""
    wl = synthetic.c6(n=32)
    _check(wl)
    assert smol.last_plan()["path"] == smol.PATH_ROWS


def test_detection_crops_c6_full():
    """The detection-crop workload at the size the benchmark runs."""
    _check(synthetic.c6())


@pytest.mark.parametrize("upload", [0, 1, 2, 3])
def test_descriptor_upload_paths(upload):
    """Every way a ragged table reaches the device (DMA on the copy stream,
    the copy kernel on the caller's stream, or the kernel reading the pinned
    slot itself) gives the oracle's results, over more calls than the staging
    ring has slots."""
    smol.set_tuning(upload=upload)
    wl = synthetic.c6(n=24)
    ref = run_oracle(wl)
    for _ in range(20):
        got = run_gpu(wl)
        assert_parity(got, ref, wl.out_dtype, f"c6 upload={upload}")
    assert smol.last_plan()["uploaded_descriptors"] == 1
    assert smol.last_plan()["launches"] == (2 if upload == 2 else 1)


@pytest.mark.parametrize("upload", [0, 2])
def test_back_to_back_ragged_calls_reuse_the_ring(upload):
    """40 ragged calls enqueued back to back, each on its own images and
    output, with no synchronisation between them (the 16-slot staging ring is
    reused while earlier kernels may still read it): every output matches the
    oracle."""
    import torch
    smol.set_tuning(upload=upload)
    try:
        wls = [synthetic.c6(n=8 + (k % 5)) for k in range(4)]
        refs = [run_oracle(wl) for wl in wls]
        srcs = [torch.from_numpy(wl.src).to("cuda:0") for wl in wls]
        torch.cuda.synchronize()
        outs = []
        for k in range(40):
            outs.append(smol.run_workload(wls[k % 4], srcs[k % 4]))
        torch.cuda.synchronize()
        for k, out in enumerate(outs):
            assert_parity(out.cpu().numpy(), refs[k % 4], wls[k % 4].out_dtype,
                          f"call {k} upload={upload}")
    finally:
        smol.reset_tuning()


@pytest.mark.parametrize("upload", [0, 1, 2])
def test_ring_waits_for_kernels_held_behind_a_busy_stream(upload):
    """The staging ring's reuse wait on kernels that have not started: a
    bounded spin kernel holds the stream while 40 ragged calls are enqueued
    (the ring has 16 slots, so the 17th call must wait for the 1st kernel's
    completion event before it rewrites that slot); every output matches the
    oracle."""
    import torch
    smol.set_tuning(upload=upload)
    try:
        wls = [synthetic.c6(n=8 + (k % 5)) for k in range(4)]
        refs = [run_oracle(wl) for wl in wls]
        srcs = [torch.from_numpy(wl.src).to("cuda:0") for wl in wls]
        torch.cuda.synchronize()
        held = torch.cuda.Event()
        torch.cuda._sleep(200_000_000)
        held.record()
        outs = [smol.run_workload(wls[k % 4], srcs[k % 4]) for k in range(16)]
        # the ring is full and the stream still held: the calls below reuse
        # slots whose kernels have not run yet
        assert not held.query(), "the spin kernel ended before the ring filled"
        outs += [smol.run_workload(wls[k % 4], srcs[k % 4]) for k in range(16, 40)]
        torch.cuda.synchronize()
        for k, out in enumerate(outs):
            assert_parity(out.cpu().numpy(), refs[k % 4], wls[k % 4].out_dtype,
                          f"call {k} upload={upload}")
    finally:
        smol.reset_tuning()
