"""JPEG files end to end on the GPU: the library's host entropy decoding
(partial, Algorithm 1's rectangles), per-frame dequantisation tables, block
decoding and the fused preprocessing, against the oracle's whole-stream
entropy decoding, whole-frame block decoding and preprocessing (marked gpu;
run on an MI355X)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2007_13005_amd import smol, synthetic
from tests.gpu_util import assert_parity, files_workload, note, run_oracle

pytestmark = pytest.mark.gpu

F32, F16 = synthetic.OUT_F32, synthetic.OUT_F16


def test_per_frame_tables_whole_decode():
    """Twenty streams of twenty qualities (more table pairs than one launch
    holds), decoded whole on the GPU with each frame's own tables."""
    import torch
    rng = np.random.default_rng(100)
    sizes = [(int(rng.integers(1, 300)), int(rng.integers(1, 200))) for _ in range(20)]
    quals = [5 * (k + 1) for k in range(20)]
    files = synthetic.jpeg_files(sizes, 100, quals, restart_blocks=4)
    b = smol.jpeg_entropy_decode_batch(files, threads=8)
    assert len({q.tobytes() for q in b.qtables}) == 20
    yo, bo, ro, cur = [], [], [], 0
    for W, H in sizes:
        Wc, Hc = (W + 1) // 2, (H + 1) // 2
        yo.append(cur)
        bo.append(cur + W * H)
        ro.append(cur + W * H + Wc * Hc)
        cur += W * H + 2 * Wc * Hc
    out = torch.full((cur,), 3, dtype=torch.uint8, device="cuda:0")
    coef = torch.from_numpy(b.coef).to("cuda:0")
    smol.jpeg_decode_i420(coef, b.coef_offsets, b.qtables, b.widths, b.heights, out, yo, bo, ro)
    torch.cuda.synchronize()
    flat = out.cpu().numpy()
    for i, f in enumerate(files):
        c, qy, qc, W, H = oracle.jpeg_entropy_decode(f)
        y, cb, cr = oracle.jpeg_decode_i420(c, qy, qc, W, H)
        assert np.array_equal(flat[yo[i]:bo[i]], y.reshape(-1)), (i, sizes[i])
        assert np.array_equal(flat[bo[i]:ro[i]], cb.reshape(-1)), (i, sizes[i])
        assert np.array_equal(flat[ro[i]:ro[i] + cb.size], cr.reshape(-1)), (i, sizes[i])
    note(f"    {len(files)} streams, {len(quals)} table pairs, decoded bit for bit")


def test_window_layout_decode():
    """Coefficients of only each rectangle's MCU window (the layout the file
    path copies to the device) decode to the oracle's pixels inside the
    rectangle and leave the rest of the planes alone; runs share launches."""
    import torch
    rng = np.random.default_rng(103)
    sizes = [(int(rng.integers(1, 400)), int(rng.integers(1, 300))) for _ in range(40)]
    sizes += [(640, 480)] * 8
    files = synthetic.jpeg_files(sizes, 103, 80, restart_blocks=3)
    rects = []
    for W, H in sizes:
        x, y = 2 * int(rng.integers(0, (W + 1) // 2)), 2 * int(rng.integers(0, (H + 1) // 2))
        rects.append((x, y, int(rng.integers(1, W - x + 1)), int(rng.integers(1, H - y + 1))))
    rects[-8:] = [rects[-8]] * 8
    b = smol.jpeg_entropy_decode_batch(files, rects, threads=8,
                                       coef_layout=smol.JPEG_COEF_WINDOW)
    yo, bo, ro, cur = [], [], [], 0
    for W, H in sizes:
        Wc, Hc = (W + 1) // 2, (H + 1) // 2
        yo.append(cur)
        bo.append(cur + W * H)
        ro.append(cur + W * H + Wc * Hc)
        cur += W * H + 2 * Wc * Hc
    out = torch.full((cur,), 7, dtype=torch.uint8, device="cuda:0")
    smol.jpeg_decode_i420(torch.from_numpy(b.coef).to("cuda:0"), b.coef_offsets, b.qtables,
                          b.widths, b.heights, out, yo, bo, ro, rects,
                          coef_layout=smol.JPEG_COEF_WINDOW)
    torch.cuda.synchronize()
    flat = out.cpu().numpy()
    for i, f in enumerate(files):
        c, qy, qc, W, H = oracle.jpeg_entropy_decode(f)
        exp = oracle.jpeg_decode_i420(c, qy, qc, W, H, rects[i], fill=7)
        Wc, Hc = (W + 1) // 2, (H + 1) // 2
        got = (flat[yo[i]:bo[i]].reshape(H, W), flat[bo[i]:ro[i]].reshape(Hc, Wc),
               flat[ro[i]:ro[i] + Wc * Hc].reshape(Hc, Wc))
        for k in range(3):
            assert np.array_equal(got[k], exp[k]), (i, sizes[i], rects[i], k)
    note(f"    {len(files)} frames decoded from their MCU windows")


@pytest.mark.parametrize("layout", [smol.LAYOUT_NCHW, smol.LAYOUT_NHWC])
@pytest.mark.parametrize("dtype", [F32, F16])
@pytest.mark.parametrize("restart", [0, 2])
def test_files_preprocess_end_to_end(dtype, layout, restart):
    sizes = [(640, 480), (333, 517), (1280, 720), (300, 600), (451, 302), (257, 256)]
    files = synthetic.jpeg_files(sizes, 101, [75, 90, 60, 75, 95, 80], restart_blocks=restart)
    p = smol.make_params(256, 224, 224, synthetic.IMAGENET_MEAN_255, synthetic.IMAGENET_STD_255,
                         dtype)
    o = smol.make_options(layout=layout) if layout else None
    got = smol.jpeg_files_preprocess(files, p, o, threads=4)
    import torch
    torch.cuda.synchronize()
    wl = files_workload("jpeg-files", files, 256, 224, dtype)
    wl.layout = layout
    stats = assert_parity(got.cpu().numpy(), run_oracle(wl), dtype, wl.name)
    note(f"    files restart={restart}: {stats}")


def test_files_at_benchmark_size():
    """The file benchmark's batch: 128 streams of 1280x720 at quality 75,
    restart markers every MCU row."""
    files = synthetic.jpeg_file_batch()
    p = smol.make_params(256, 224, 224, synthetic.IMAGENET_MEAN_255, synthetic.IMAGENET_STD_255,
                         F16)
    got = smol.jpeg_files_preprocess(files, p, threads=16)
    import torch
    torch.cuda.synchronize()
    wl = files_workload("jpeg-files-128", files, 256, 224, F16)
    stats = assert_parity(got.cpu().numpy(), run_oracle(wl), F16, wl.name)
    note(f"    {wl.name}: {stats}")


def test_widest_and_tallest_streams():
    """65500 x 17 and 17 x 65500 (libjpeg's largest size): block indices and
    windows near the 16-bit limits of the run table, restart skipping on
    4094-MCU rows; whole frames and Algorithm 1's windows, bit for bit."""
    import torch
    sizes = [(65500, 17), (17, 65500)]
    files = synthetic.jpeg_files(sizes, 111, 75, restart_blocks=100)
    p = smol.make_params(224, 224, 224, synthetic.IMAGENET_MEAN_255, synthetic.IMAGENET_STD_255,
                         F16)
    rects = [smol.jpeg_mcu_rect(W, H, p) for W, H in sizes]
    yo, bo, ro, cur = [], [], [], 0
    for W, H in sizes:
        Wc, Hc = (W + 1) // 2, (H + 1) // 2
        yo.append(cur)
        bo.append(cur + W * H)
        ro.append(cur + W * H + Wc * Hc)
        cur += W * H + 2 * Wc * Hc
    for layout, rr in ((smol.JPEG_COEF_FRAME, None), (smol.JPEG_COEF_WINDOW, rects)):
        b = smol.jpeg_entropy_decode_batch(files, rr, threads=2, coef_layout=layout)
        out = torch.full((cur,), 7, dtype=torch.uint8, device="cuda:0")
        smol.jpeg_decode_i420(torch.from_numpy(b.coef).to("cuda:0"), b.coef_offsets, b.qtables,
                              b.widths, b.heights, out, yo, bo, ro, rr, coef_layout=layout)
        torch.cuda.synchronize()
        flat = out.cpu().numpy()
        for i, f in enumerate(files):
            c, qy, qc, W, H = oracle.jpeg_entropy_decode(f)
            exp = oracle.jpeg_decode_i420(c, qy, qc, W, H, None if rr is None else rr[i], fill=7)
            Wc, Hc = (W + 1) // 2, (H + 1) // 2
            got = (flat[yo[i]:bo[i]].reshape(H, W), flat[bo[i]:ro[i]].reshape(Hc, Wc),
                   flat[ro[i]:ro[i] + Wc * Hc].reshape(Hc, Wc))
            for k in range(3):
                assert np.array_equal(got[k], exp[k]), (layout, sizes[i], k)


def test_side_streams_match_the_current_stream():
    """Calls given a stream other than torch's current one (a torch stream
    or a raw handle) order themselves after the current stream's work and
    keep their temporaries alive: same bytes as on the current stream."""
    import torch
    files = synthetic.jpeg_files([(640, 480), (333, 517), (1280, 720)], 104, 80,
                                 restart_blocks=2)
    p = smol.make_params(256, 224, 224, synthetic.IMAGENET_MEAN_255, synthetic.IMAGENET_STD_255,
                         F16)
    ref = smol.jpeg_files_preprocess(files, p, threads=4)
    wl = synthetic.c7(n=6)
    src = torch.from_numpy(wl.src).to("cuda:0")
    low_ref = smol.run_workload(wl, src)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    for st in (side, side.cuda_stream):
        got = smol.jpeg_files_preprocess(files, p, threads=4, stream=st)
        low = smol.run_workload(wl, src, stream=st)
        torch.cuda.synchronize()
        assert torch.equal(got, ref) and torch.equal(low, low_ref)
        # a caller-supplied output filled on the current stream just before:
        # the side-stream call must overwrite it only after that fill
        out = torch.empty_like(ref)
        out.fill_(7.0)
        got = smol.jpeg_files_preprocess(files, p, threads=4, stream=st, out=out)
        torch.cuda.synchronize()
        assert got.data_ptr() == out.data_ptr() and torch.equal(out, ref)
