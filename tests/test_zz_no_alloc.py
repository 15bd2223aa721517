"""The no-allocation entry point (smol_preprocess_batch_noalloc) on the GPU,
through the C ABI, against smol_preprocess_batch on the same inputs: the
same kernels run, so the outputs must be identical bit for bit (which is
within the parity bar of the regular call: 1e-5 for fp32, one fp16 ulp).

Calls follow one another on one stream with nothing in between, the second
on a smaller ragged batch: its descriptor table overwrites the front of the
fixed device array while the first call's kernel may still be queued, so a
copy that did not keep stream order would corrupt the first output."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest

from paper_2007_13005_amd import smol, synthetic
from tests.gpu_util import assert_parity, note, run_oracle

pytestmark = pytest.mark.gpu


def _tables(wl):
    return (np.ascontiguousarray(wl.offsets, np.int64), np.ascontiguousarray(wl.widths, np.int32),
            np.ascontiguousarray(wl.heights, np.int32))


def _call(name, wl, src, out, stream):
    """Enqueue one call of `name` (a C-ABI symbol) on `stream`."""
    p = smol.make_params(wl.resize_short, wl.crop_h, wl.crop_w, wl.mean, wl.std, wl.out_dtype)
    off, w, h = _tables(wl)
    rc = getattr(smol.lib(), name)(src.data_ptr(), src.numel(), off.ctypes.data, w.ctypes.data,
                                   h.ctypes.data, None, wl.n, ctypes.byref(p), out.data_ptr(),
                                   stream)
    assert rc == 0, smol.lib().smol_last_error().decode()


def _empty_out(wl):
    import torch
    dt = torch.float16 if wl.out_dtype == synthetic.OUT_F16 else torch.float32
    return torch.full(wl.out_shape(), float("nan"), dtype=dt, device="cuda:0")


def _tiny_ragged(n: int, seed: int):
    """n ragged images of 16..48 px a side (S 32, crop 32, fp32)."""
    rng = np.random.default_rng(seed)
    sizes = rng.integers(16, 49, size=(n, 2))
    images = [rng.integers(0, 256, size=(int(h), int(w), 3), dtype=np.uint8) for w, h in sizes]
    return synthetic.rgb_workload(f"tiny{seed}", images, 32, 32, synthetic.OUT_F32)


def _run_pair(first, second):
    """Both workloads through both entry points; returns the four outputs."""
    import torch
    st = torch.cuda.current_stream().cuda_stream
    src1 = torch.from_numpy(first.src).to("cuda:0")
    src2 = torch.from_numpy(second.src).to("cuda:0")
    ref1, ref2 = _empty_out(first), _empty_out(second)
    _call("smol_preprocess_batch", first, src1, ref1, st)
    _call("smol_preprocess_batch", second, src2, ref2, st)
    torch.cuda.synchronize()
    got1, got2 = _empty_out(first), _empty_out(second)
    _call("smol_preprocess_batch_noalloc", first, src1, got1, st)
    _call("smol_preprocess_batch_noalloc", second, src2, got2, st)
    torch.cuda.synchronize()
    return ref1, ref2, got1, got2


def test_two_ragged_calls_in_a_row_second_smaller():
    import torch
    big = synthetic.c2(n=600)
    # the same images in another order, fewer of them: another table
    rng = np.random.default_rng(7)
    idx = rng.permutation(big.n)[:150]
    imgs = [big.src[int(big.offsets[i]):int(big.offsets[i]) + 3 * int(big.widths[i]) *
                    int(big.heights[i])].reshape(int(big.heights[i]), int(big.widths[i]), 3)
            for i in idx]
    small = synthetic.rgb_workload("c2-small", imgs, 256, 224, synthetic.OUT_F16)
    note(f"noalloc: ragged {big.n} then {small.n} images")
    ref1, ref2, got1, got2 = _run_pair(big, small)
    assert torch.equal(got1, ref1)
    assert torch.equal(got2, ref2)
    # and the regular call itself holds the parity bar on the small batch
    assert_parity(got2.cpu().numpy(), run_oracle(small), small.out_dtype, small.name)


def test_largest_table_then_a_smaller_one():
    import torch
    big = _tiny_ragged(4096, 11)
    small = _tiny_ragged(1000, 12)
    note(f"noalloc: ragged {big.n} (the limit) then {small.n} tiny images")
    ref1, ref2, got1, got2 = _run_pair(big, small)
    assert torch.equal(got1, ref1)
    assert torch.equal(got2, ref2)
    assert_parity(got2.cpu().numpy(), run_oracle(small), small.out_dtype, small.name)


def test_uniform_batch_needs_no_table():
    import torch
    wl = synthetic.c4(n=3)
    note("noalloc: uniform 3 x 1080p")
    ref, _, got, _ = _run_pair(wl, synthetic.c1(n=2))
    assert torch.equal(got, ref)


def test_over_the_limit_is_refused_before_anything_runs():
    import torch
    wl = _tiny_ragged(4097, 13)
    src = torch.from_numpy(wl.src).to("cuda:0")
    out = _empty_out(wl)
    p = smol.make_params(32, 32, 32, wl.mean, wl.std, wl.out_dtype)
    off, w, h = _tables(wl)
    rc = smol.lib().smol_preprocess_batch_noalloc(src.data_ptr(), src.numel(), off.ctypes.data,
                                                  w.ctypes.data, h.ctypes.data, None, wl.n,
                                                  ctypes.byref(p), out.data_ptr(), None)
    torch.cuda.synchronize()
    assert rc == smol.ERR_UNSUPPORTED
    assert bool(torch.isnan(out).all())
