"""The pipeline (smol_pipeline.cpp) and the binding's consumer path on the
CPU, against a thread-backed HIP stand-in (tests/csrc/fake_hip): each stream
is a worker thread executing its copies, event records and waits and
"kernels" (tasks of 200 us) in order, host waits block on events, device
memory is host memory. The library's host files are built with g++ against
it, so acquire / submit / the consumer callback / hipEventSynchronize run with
real concurrency and real locks.

What is checked (each scenario in its own process under a time limit, so a
deadlock fails the test instead of hanging it):

- eight Python producer threads and a monitor share six slots and three
  streams; every consumer is a Python callable that holds the GIL for a while,
  re-enters the library (a preprocessing call on the batch's stream), queues
  device work of its own and sleeps; every batch completes and the queues
  drain: no lock order between the GIL, the pipeline's mutex, the ctypes
  callback and the host waits deadlocks;
- a consumer that calls back into its own pipeline's blocking entry points
  (here acquire) is refused by the binding instead of waiting, and its
  submission fails;
- the hazard that guard exists for: through the raw C ABI, producers whose
  consumers wait for a slot of their own pipeline while holding every slot
  never finish (the time limit ends them)."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2007_13005_amd", "csrc")
SOURCES = ["smol_host.cpp", "smol_pipeline.cpp", "smol_jpeg.cpp", "smol_jpeg_entropy.cpp"]


@pytest.fixture(scope="module")
def fake_lib(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("needs g++")
    out = tmp_path_factory.mktemp("fake") / "libsmol_fake.so"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-shared", "-fPIC",
           "-I", os.path.join(ROOT, "tests", "csrc", "fake_hip"),
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           *[os.path.join(CSRC, f) for f in SOURCES],
           os.path.join(ROOT, "tests", "csrc", "fake_hip.cpp"), "-o", str(out), "-lpthread"]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, res.stderr[-4000:]
    return str(out)


PRELUDE = textwrap.dedent("""
    import ctypes, sys, threading, time
    import numpy as np
    sys.path.insert(0, {root!r})
    from paper_2007_13005_amd import smol, synthetic
    L = smol.bind_signatures(ctypes.CDLL({lib!r}), required=False)
    L.fake_hip_task.argtypes = [ctypes.c_void_p, ctypes.c_uint]
    L.fake_hip_pending_ops.restype = ctypes.c_long
    N, SIDE = 8, 64                  # images per batch, 64 x 64 RGB each
    IMG = SIDE * SIDE * 3
    p = smol.make_params(32, 32, 32, synthetic.IMAGENET_MEAN_255,
                         synthetic.IMAGENET_STD_255, smol.OUT_F32)
    OUT = N * 3 * 32 * 32 * 4        # = N * IMG: the output read as N 64 x 64 images
    offs = np.arange(N, dtype=np.int64) * IMG
    cons_offs = np.arange(N, dtype=np.int64) * (OUT // N)
    ws = np.full(N, SIDE, np.int32)
    hs = np.full(N, SIDE, np.int32)
    scratch = np.zeros(OUT, np.uint8)
""")


def _run(fake_lib, body: str, timeout: int):
    code = PRELUDE.format(root=ROOT, lib=fake_lib) + textwrap.dedent(body)
    return subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                          timeout=timeout)


def test_producers_and_reentrant_consumers_complete(fake_lib):
    res = _run(fake_lib, """
        pipe = smol.Pipeline(6, 3, N * IMG, OUT, library=L)
        BATCHES, THREADS = 25, 8
        calls = [0]

        def consumer(output, n, stream):
            calls[0] += 1
            sum(range(5000))                       # hold the GIL a while
            # re-enter the library on the batch's stream: its output read as
            # n RGB images of 64 x 64, resized into a scratch buffer
            rc = L.smol_preprocess_batch(output, OUT, cons_offs.ctypes.data, ws.ctypes.data,
                                         hs.ctypes.data, None, n, ctypes.byref(p),
                                         scratch.ctypes.data, stream)
            assert rc == 0, L.smol_last_error()
            L.fake_hip_task(stream, 300)           # the consumer's own device work
            time.sleep(0.0001)

        errors = []

        def producer(t):
            try:
                for b in range(BATCHES):
                    slot, host, out = pipe.acquire()
                    pipe.host_view(slot)[:N * IMG] = (t + b) % 251
                    pipe.submit(slot, N * IMG, offs, ws, hs, p, consumer=consumer)
            except Exception as e:                 # noqa: BLE001
                errors.append(repr(e))

        stop = threading.Event()

        def monitor():
            while not stop.is_set():
                pipe.stats()
                time.sleep(0.002)

        th = [threading.Thread(target=producer, args=(t,)) for t in range(THREADS)]
        mon = threading.Thread(target=monitor)
        mon.start()
        for x in th:
            x.start()
        for x in th:
            x.join()
        stop.set()
        mon.join()
        pipe.drain()
        st = pipe.stats()
        assert not errors, errors
        assert st["submitted"] == st["completed"] == BATCHES * THREADS, st
        assert calls[0] == BATCHES * THREADS
        pipe.close()
        print("OK", st, "pending", L.fake_hip_pending_ops())
    """, timeout=180)
    assert res.returncode == 0, (res.stdout + res.stderr)[-4000:]
    assert "OK" in res.stdout


def test_consumer_calling_its_own_pipeline_is_refused(fake_lib):
    res = _run(fake_lib, """
        pipe = smol.Pipeline(2, 1, N * IMG, OUT, library=L)
        seen = []

        def greedy(output, n, stream):
            try:
                pipe.acquire()
            except RuntimeError as e:
                seen.append(str(e))
                raise

        slot, host, out = pipe.acquire()
        try:
            pipe.submit(slot, N * IMG, offs, ws, hs, p, consumer=greedy)
            raise SystemExit("the submission should have failed")
        except smol.SmolError as e:
            assert "consumer returned" in str(e), e
        assert seen and "inside a consumer" in seen[0], seen
        pipe.drain()
        assert pipe.stats()["completed"] == 1
        pipe.close()
        print("OK")
    """, timeout=60)
    assert res.returncode == 0, (res.stdout + res.stderr)[-4000:]
    assert "OK" in res.stdout


def test_raw_consumer_waiting_for_a_slot_never_finishes(fake_lib):
    # The hazard the guard refuses, shown through the C ABI with no guard:
    # two producers hold both slots and their consumers wait for a third.
    with pytest.raises(subprocess.TimeoutExpired):
        _run(fake_lib, """
            h = ctypes.c_void_p()
            cfg = smol.PipelineConfig()
            cfg.slots, cfg.streams, cfg.copy_streams = 2, 1, 1
            cfg.input_bytes, cfg.output_bytes = N * IMG, OUT
            assert L.smol_pipeline_create(ctypes.byref(cfg), ctypes.byref(h)) == 0
            barrier = threading.Barrier(2)

            def waits_for_a_slot(user, output, n, stream):
                s, a, b = ctypes.c_int32(), ctypes.c_void_p(), ctypes.c_void_p()
                return L.smol_pipeline_acquire(h, ctypes.byref(s), ctypes.byref(a),
                                               ctypes.byref(b))

            cb = smol.CONSUMER(waits_for_a_slot)

            def producer():
                s, a, b = ctypes.c_int32(), ctypes.c_void_p(), ctypes.c_void_p()
                L.smol_pipeline_acquire(h, ctypes.byref(s), ctypes.byref(a), ctypes.byref(b))
                barrier.wait()                     # both slots are held now
                L.smol_pipeline_submit(h, s.value, N * IMG, offs.ctypes.data, ws.ctypes.data,
                                       hs.ctypes.data, None, None, N, ctypes.byref(p), None,
                                       cb, None)

            th = [threading.Thread(target=producer) for _ in range(2)]
            for x in th:
                x.start()
            for x in th:
                x.join()
            print("finished")
        """, timeout=8)
