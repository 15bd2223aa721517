"""GPU checks of the pipelined ingest (``include/smol_pipeline.h``): several
producer threads filling reused pinned slots, copies and preprocessing on
several streams, a consumer behind every batch -- every batch's output
against the oracle (marked gpu; run on an MI355X)."""
from __future__ import annotations

import threading

import numpy as np
import pytest

from paper_2007_13005_amd import smol, synthetic
from tests.gpu_util import assert_parity, note, run_oracle

pytestmark = pytest.mark.gpu

F16 = synthetic.OUT_F16


def _rgb_batches(k: int, n: int, seed: int = 41):
    rng = np.random.default_rng(seed)
    out = []
    for b in range(k):
        sizes = rng.integers(60, 201, size=(n, 2))
        imgs = [rng.integers(0, 256, size=(int(h), int(w), 3), dtype=np.uint8) for w, h in sizes]
        out.append(synthetic.rgb_workload(f"pipe{b}", imgs, 64, 56, F16))
    return out


def _copy_consumer(results):
    """A consumer that copies each batch's output into results[user] on the
    batch's stream (stands in for a DNN reading it)."""
    rt = smol.hip_runtime()

    def consume(user, output, n, stream):
        try:
            dst = results[user or 0]
            return rt.hipMemcpyAsync(dst.data_ptr(), output, dst.numel() * dst.element_size(),
                                     smol.HIP_MEMCPY_DEVICE_TO_DEVICE, stream)
        except Exception:  # noqa: BLE001 -- reported as a failed consumer
            return 1
    return smol.CONSUMER(consume)


def _params(wl):
    return smol.make_params(wl.resize_short, wl.crop_h, wl.crop_w, wl.mean, wl.std, wl.out_dtype)


def test_concurrent_producers_every_batch_matches_the_oracle():
    import torch
    wls = _rgb_batches(5, 12)
    refs = [run_oracle(w) for w in wls]
    threads, per_thread = 4, 6
    jobs = threads * per_thread
    results = [torch.empty(wls[j % 5].out_shape(), dtype=torch.float16, device="cuda:0")
               for j in range(jobs)]
    cb = _copy_consumer(results)
    in_bytes = max(w.src.size for w in wls)
    out_bytes = max(int(np.prod(w.out_shape())) * 2 for w in wls)
    errors = []
    with smol.Pipeline(slots=3, streams=2, input_bytes=in_bytes, output_bytes=out_bytes) as pl:
        def producer(t):
            try:
                for i in range(per_thread):
                    j = t * per_thread + i
                    wl = wls[j % 5]
                    slot, _, _ = pl.acquire()
                    pl.host_view(slot)[:wl.src.size] = wl.src
                    pl.submit(slot, wl.src.size, wl.offsets, wl.widths, wl.heights, _params(wl),
                              consumer=cb, user=j)
            except Exception as e:  # noqa: BLE001
                errors.append(e)
        ts = [threading.Thread(target=producer, args=(t,)) for t in range(threads)]
        for t in ts:
            t.start()
        for t in ts:
            t.join()
        pl.drain()
        st = pl.stats()
    assert not errors, errors
    torch.cuda.synchronize()
    note(f"    pipeline stats {st}")
    assert st["submitted"] == st["completed"] == jobs
    assert st["images"] == sum(wls[j % 5].n for j in range(jobs))
    for j in range(jobs):
        assert_parity(results[j].cpu().numpy(), refs[j % 5], F16, f"batch {j}")


def test_yuv_batches_with_options_through_one_slot():
    """One slot, one stream: each submission waits for the previous one to
    finish; I420 frames with NHWC output and left-sited chroma."""
    import torch
    rng = np.random.default_rng(42)
    wls = []
    for b in range(3):
        planes = []
        for w, h in [(320, 240), (161, 99), (200, 300)]:
            cw, ch = (w + 1) // 2, (h + 1) // 2
            planes.append((rng.integers(16, 236, (h, w), dtype=np.uint8),
                           rng.integers(16, 241, (ch, cw), dtype=np.uint8),
                           rng.integers(16, 241, (ch, cw), dtype=np.uint8)))
        wl = synthetic.yuv420_workload(f"pipe-yuv{b}", planes, 96, 80, F16)
        wl.layout, wl.siting = smol.LAYOUT_NHWC, smol.CHROMA_LEFT
        wls.append(wl)
    results = [torch.empty(w.out_shape(), dtype=torch.float16, device="cuda:0") for w in wls]
    cb = _copy_consumer(results)
    opts = smol.make_options(smol.RESIZE_SHORT_CROP, smol.LAYOUT_NHWC, smol.CHROMA_LEFT)
    with smol.Pipeline(1, 1, max(w.src.size for w in wls),
                       max(int(np.prod(w.out_shape())) * 2 for w in wls)) as pl:
        for j, wl in enumerate(wls):
            slot, _, _ = pl.acquire()
            pl.host_view(slot)[:wl.src.size] = wl.src
            pl.submit_yuv420(slot, wl.src.size, wl.y_offsets, wl.cb_offsets, wl.cr_offsets,
                             wl.widths, wl.heights, _params(wl), options=opts, consumer=cb,
                             user=j)
        pl.drain()
        assert pl.stats()["acquire_waits"] <= 2  # 0 when a batch finished before the next acquire
    torch.cuda.synchronize()
    for j, wl in enumerate(wls):
        assert_parity(results[j].cpu().numpy(), run_oracle(wl), F16, wl.name)


def test_bad_submission_keeps_the_slot_and_failed_consumer_recycles_it():
    wl = _rgb_batches(1, 4)[0]
    with smol.Pipeline(2, 1, wl.src.size, int(np.prod(wl.out_shape())) * 2) as pl:
        slot, _, _ = pl.acquire()
        with pytest.raises(smol.SmolError):
            pl.submit(slot, wl.src.size + 1, wl.offsets, wl.widths, wl.heights, _params(wl))
        pl.host_view(slot)[:wl.src.size] = wl.src
        failing = smol.CONSUMER(lambda user, out, n, stream: 7)
        with pytest.raises(smol.SmolError, match="consumer returned 7"):
            pl.submit(slot, wl.src.size, wl.offsets, wl.widths, wl.heights, _params(wl),
                      consumer=failing)
        with pytest.raises(smol.SmolError):
            pl.release(slot)  # submitted: no longer acquired
        s2, _, _ = pl.acquire()
        pl.release(s2)
        pl.drain()
        st = pl.stats()
        assert st["submitted"] == st["completed"] == 1


def test_jpeg_batches_decoded_into_slots():
    """Producer threads entropy-decode JPEG batches straight into the pinned
    slots they acquired; the copy, partial block decoding and preprocessing
    run in stream order; every batch equals the oracle's chain."""
    import torch
    from tests.gpu_util import files_workload
    rng = np.random.default_rng(43)
    batches = []
    for b in range(4):
        sizes = [(int(rng.integers(200, 700)), int(rng.integers(200, 500))) for _ in range(5)]
        batches.append(synthetic.jpeg_files(sizes, 43 + b, [60, 75, 90, 75, 85],
                                            restart_blocks=b % 3))
    p = smol.make_params(128, 112, 112, synthetic.IMAGENET_MEAN_255,
                         synthetic.IMAGENET_STD_255, F16)
    results = [torch.empty((5, 3, 112, 112), dtype=torch.float16, device="cuda:0")
               for _ in range(8)]
    cb = _copy_consumer(results)
    ws = max(smol.jpeg_workspace_bytes(*zip(*[(smol.jpeg_read_info(f).width,
                                                smol.jpeg_read_info(f).height) for f in bt]))
             for bt in batches)
    errors = []
    with smol.Pipeline(4, 2, 8 << 20, 5 * 3 * 112 * 112 * 2, workspace_bytes=ws) as pl:

        def producer(t):
            try:
                for j in range(t, 8, 2):
                    slot, _, _ = pl.acquire()
                    nb, co, q, w, h = pl.decode_jpeg_into(slot, batches[j % 4], p, threads=2)
                    pl.submit_jpeg(slot, nb, co, q, w, h, p, consumer=cb, user=j)
            except Exception as e:  # noqa: BLE001 -- reported below
                errors.append(e)

        ths = [threading.Thread(target=producer, args=(t,)) for t in range(2)]
        for th in ths:
            th.start()
        for th in ths:
            th.join()
        pl.drain()
        assert pl.stats()["submitted"] == 8
    assert not errors, errors
    torch.cuda.synchronize()
    for j in range(8):
        wl = files_workload(f"pipe-jpeg{j}", batches[j % 4], 128, 112, F16)
        assert_parity(results[j].cpu().numpy(), run_oracle(wl), F16, wl.name)
    note("    8 JPEG batches through the pipeline match the oracle")


def test_jpeg_submission_errors_keep_the_slot():
    """A JPEG submission to a pipeline created without a workspace, or with
    an odd byte count, is rejected before anything is enqueued; the slot
    stays acquired and can be released."""
    p = smol.make_params(64, 56, 56, synthetic.IMAGENET_MEAN_255, synthetic.IMAGENET_STD_255,
                         F16)
    q = np.ones((1, 2, 64), np.uint16)
    for ws, nbytes, needle in ((0, 6 * 128, "no workspace"), (1 << 20, 6 * 128 - 1, "int16")):
        with smol.Pipeline(1, 1, 1 << 16, 3 * 56 * 56 * 2, workspace_bytes=ws) as pl:
            slot, _, _ = pl.acquire()
            with pytest.raises(smol.SmolError, match=needle):
                pl.submit_jpeg(slot, nbytes, [0], q, [16], [16], p,
                               coef_layout=smol.JPEG_COEF_FRAME)
            pl.release(slot)
            assert pl.stats()["submitted"] == 0


def test_jpeg_batch_larger_than_the_slot_is_refused():
    files = synthetic.jpeg_files([(640, 480)], 44, 75)
    p = smol.make_params(256, 224, 224, synthetic.IMAGENET_MEAN_255, synthetic.IMAGENET_STD_255,
                         F16)
    with smol.Pipeline(1, 1, 1 << 10, 3 * 224 * 224 * 2, workspace_bytes=1 << 20) as pl:
        slot, _, _ = pl.acquire()
        with pytest.raises(ValueError, match="exceed the slot"):
            pl.decode_jpeg_into(slot, files, p)
        pl.release(slot)
