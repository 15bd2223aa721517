"""GPU parity of partial JPEG decoding (``include/smol_jpeg.h``): block
decoding bit for bit against the oracle, partial decoding of Algorithm 1's
rectangle, and decode-then-preprocess against the oracle's whole-frame decode
followed by its preprocessing (marked gpu; run on an MI355X)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2007_13005_amd import smol, synthetic
from tests.gpu_util import assert_parity, note, run_gpu, run_oracle

pytestmark = pytest.mark.gpu

F32, F16 = synthetic.OUT_F32, synthetic.OUT_F16
SIZES = [(203, 77), (33, 21), (16, 16), (1, 1), (640, 480), (97, 130)]


def _upload(wl):
    import torch
    return torch.from_numpy(wl.src.copy()).to("cuda:0").view(torch.int16)


def _planes_layout(sizes):
    yo, bo, ro, cur = [], [], [], 0
    for W, H in sizes:
        Wc, Hc = (W + 1) // 2, (H + 1) // 2
        yo.append(cur)
        bo.append(cur + W * H)
        ro.append(cur + W * H + Wc * Hc)
        cur += W * H + 2 * Wc * Hc
    return yo, bo, ro, cur


def _gpu_decode(wl, rects=None, fill=7):
    import torch
    sizes = list(zip(wl.widths.tolist(), wl.heights.tolist()))
    yo, bo, ro, total = _planes_layout(sizes)
    out = torch.full((total,), fill, dtype=torch.uint8, device="cuda:0")
    smol.jpeg_decode_i420(_upload(wl), wl.coef_offsets, wl.qtables, wl.widths, wl.heights, out,
                          yo, bo, ro, rects)
    torch.cuda.synchronize()
    flat = out.cpu().numpy()
    res = []
    for (W, H), y, b, r in zip(sizes, yo, bo, ro):
        Wc, Hc = (W + 1) // 2, (H + 1) // 2
        res.append((flat[y:y + W * H].reshape(H, W), flat[b:b + Wc * Hc].reshape(Hc, Wc),
                    flat[r:r + Wc * Hc].reshape(Hc, Wc)))
    return res


def _oracle_decode(wl, i, rect=None, fill=7):
    W, H = int(wl.widths[i]), int(wl.heights[i])
    k = oracle.jpeg_coef_count(W, H)
    c = wl.src.view(np.int16)[int(wl.coef_offsets[i]):int(wl.coef_offsets[i]) + k]
    return oracle.jpeg_decode_i420(c, *wl.frame_qtables(i), W, H, rect, fill=fill)


def test_whole_frame_decode_bit_exact():
    wl = synthetic.jpeg_workload("jpeg-sizes", SIZES, 16, 8, F16, 51)
    got = _gpu_decode(wl)
    for i in range(wl.n):
        exp = _oracle_decode(wl, i)
        for k in range(3):
            assert np.array_equal(got[i][k], exp[k]), (SIZES[i], k)
    note(f"    decoded {wl.n} frames bit for bit")


def test_rectangle_decode_touches_only_its_blocks():
    sizes = [(203, 77), (640, 480), (97, 130)]
    wl = synthetic.jpeg_workload("jpeg-rect", sizes, 16, 8, F16, 52)
    rects = [(48, 16, 112, 48), (100, 50, 301, 333), (0, 2, 97, 128)]
    got = _gpu_decode(wl, rects, fill=7)
    for i, r in enumerate(rects):
        exp = _oracle_decode(wl, i, r, fill=7)
        for k in range(3):
            assert np.array_equal(got[i][k], exp[k]), (sizes[i], r, k)


def test_ragged_batch_spans_several_launches():
    """Sixty frames in more runs of one geometry than one launch's table
    holds, with and without rectangles, bit for bit."""
    rng = np.random.default_rng(56)
    sizes = []
    while len(sizes) < 60:
        W, H = int(rng.integers(1, 200)), int(rng.integers(1, 150))
        sizes += [(W, H)] * (1 + (len(sizes) % 3 == 0) * int(rng.integers(0, 4)))
    sizes = sizes[:60]
    runs = 1 + sum(a != b for a, b in zip(sizes, sizes[1:]))
    assert runs > 24, runs
    wl = synthetic.jpeg_workload("jpeg-ragged", sizes, 16, 8, F16, 56)
    rects = []
    for W, H in sizes:
        x, y = 2 * int(rng.integers(0, (W + 1) // 2)), 2 * int(rng.integers(0, (H + 1) // 2))
        rects.append((x, y, int(rng.integers(1, W - x + 1)), int(rng.integers(1, H - y + 1))))
    for rr in (None, rects):
        got = _gpu_decode(wl, rr, fill=7)
        for i in range(wl.n):
            exp = _oracle_decode(wl, i, None if rr is None else rr[i], fill=7)
            for k in range(3):
                assert np.array_equal(got[i][k], exp[k]), (i, sizes[i], k)
    note(f"    {wl.n} frames in {runs} runs decoded bit for bit")


@pytest.mark.parametrize("layout", [smol.LAYOUT_NCHW, smol.LAYOUT_NHWC])
@pytest.mark.parametrize("dtype", [F32, F16])
def test_partial_decode_then_preprocess(dtype, layout):
    """Algorithm 1 end to end against the oracle's whole-frame decode and
    preprocessing: decoding only the MCU rectangle changes nothing."""
    sizes = [(640, 480), (333, 517), (1280, 720), (300, 600), (451, 302)]
    wl = synthetic.jpeg_workload("jpeg-roi", sizes, 256, 224, dtype, 53)
    wl.layout = layout
    got = run_gpu(wl)
    stats = assert_parity(got, run_oracle(wl), dtype, wl.name)
    plan = smol.last_plan()
    note(f"    {wl.name}: {stats} plan={plan}")
    # the plan counts the block decoding too (one launch for these five
    # geometries) besides the preprocessing's launches
    assert plan["launches"] >= 2


def test_partial_decode_direct_resize():
    wl = synthetic.jpeg_workload("jpeg-direct", [(640, 480), (97, 130)], 1, (112, 96), F16, 54)
    wl.resize_mode = smol.RESIZE_DIRECT
    assert_parity(run_gpu(wl), run_oracle(wl), F16, wl.name)


def test_partial_equals_whole_decode_on_gpu():
    """The combined call's output equals the library's own whole-frame decode
    followed by smol_yuv420_preprocess_batch, bit for bit."""
    import torch
    wl = synthetic.jpeg_workload("jpeg-eq", [(1280, 720)] * 3, 224, 224, F16, 55)
    a = run_gpu(wl)
    sizes = list(zip(wl.widths.tolist(), wl.heights.tolist()))
    yo, bo, ro, total = _planes_layout(sizes)
    planes = torch.empty(total, dtype=torch.uint8, device="cuda:0")
    smol.jpeg_decode_i420(_upload(wl), wl.coef_offsets, wl.qtables, wl.widths, wl.heights,
                          planes, yo, bo, ro)
    p = smol.make_params(224, 224, 224, wl.mean, wl.std, F16)
    b = smol.yuv420_preprocess_batch(planes, yo, bo, ro, wl.widths, wl.heights, p)
    torch.cuda.synchronize()
    assert np.array_equal(a.view(np.uint16), b.cpu().numpy().view(np.uint16))


def test_jpeg_c8_full():
    """The partial-decoding workload at the size the benchmark runs."""
    wl = synthetic.c8()
    got = run_gpu(wl)
    stats = assert_parity(got, run_oracle(wl), wl.out_dtype, wl.name)
    note(f"    c8: {stats} plan={smol.last_plan()}")


@pytest.mark.parametrize("wg", [1, 3])
def test_block_decoder_walks_many_groups_per_wave(wg):
    """A launch of `wg` one-wave workgroups per compute unit: every wave
    walks many groups of blocks, across runs of different geometries,
    reading each next group's rows while it computes the current one; the
    decodes of the whole-frame and many-runs cases stay bit for bit."""
    smol.set_tuning(workgroups_per_cu=wg)
    try:
        test_whole_frame_decode_bit_exact()
        test_ragged_batch_spans_several_launches()
    finally:
        smol.reset_tuning()
