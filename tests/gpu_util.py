"""Helpers for the GPU parity tests: run a workload through the C ABI and
through the oracle, and compare to the stated tolerances.

Tolerances: fp32 outputs within 1e-5 absolute of the oracle; fp16 outputs
within 1 unit in the last place of the oracle's round-to-nearest-even fp16
(distance measured on the ordered binary16 encoding); uint8 outputs (a
rounding decision taken in fp32 on both sides) bit for bit.
"""
from __future__ import annotations

import sys

import numpy as np

import oracle
from paper_2007_13005_amd import smol, synthetic

F32_TOL = 1e-5
F16_ULP = 1


def note(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def jpeg_planes(wl: synthetic.Workload):
    """The oracle's whole-frame decode of a jpeg workload as a packed I420
    batch: (flat buffer, y, cb, cr offsets)."""
    coef = wl.src.view(np.int16)
    bufs, yo, bo, ro, cur = [], [], [], [], 0
    for i in range(wl.n):
        W, H = int(wl.widths[i]), int(wl.heights[i])
        k = oracle.jpeg_coef_count(W, H)
        c = coef[int(wl.coef_offsets[i]):int(wl.coef_offsets[i]) + k]
        y, cb, cr = oracle.jpeg_decode_i420(c, *wl.frame_qtables(i), W, H)
        yo.append(cur)
        bo.append(cur + y.size)
        ro.append(cur + y.size + cb.size)
        cur += y.size + cb.size + cr.size
        bufs += [y.reshape(-1), cb.reshape(-1), cr.reshape(-1)]
    return np.concatenate(bufs), yo, bo, ro


def files_workload(name, files, S, C, dtype) -> synthetic.Workload:
    """The oracle's entropy decoding of JPEG streams, packed as a coefficient
    workload (per-frame tables) for the oracle's block decoding and
    preprocessing (``run_oracle``)."""
    coefs, qs, ws, hs = [], [], [], []
    for f in files:
        c, qy, qc, W, H = oracle.jpeg_entropy_decode(f)
        coefs.append(c)
        qs.append(np.stack([qy, qc]))
        ws.append(W)
        hs.append(H)
    offs = np.cumsum([0] + [c.size for c in coefs[:-1]]).astype(np.int64)
    return synthetic.Workload(name=name, kind="jpeg", src=np.concatenate(coefs).view(np.uint8),
                              widths=np.asarray(ws, np.int32), heights=np.asarray(hs, np.int32),
                              resize_short=S, crop_h=C, crop_w=C, out_dtype=dtype,
                              coef_offsets=offs, qtables=np.stack(qs))


def run_oracle(wl: synthetic.Workload) -> np.ndarray:
    if wl.kind == "jpeg":
        flat, yo, bo, ro = jpeg_planes(wl)
        return oracle.yuv420_preprocess_batch_ex(flat, yo, bo, ro, wl.widths, wl.heights, None,
                                                 wl.resize_short, wl.crop_h, wl.crop_w, wl.mean,
                                                 wl.std, wl.out_dtype, wl.resize_mode, wl.layout,
                                                 oracle.CHROMA_CENTER)
    if wl.low_res:
        if wl.kind == "rgb":
            return oracle.lowres_preprocess_batch(wl.src, wl.offsets, wl.widths, wl.heights,
                                                  wl.pitches, wl.low_res, wl.resize_short,
                                                  wl.crop_h, wl.crop_w, wl.mean, wl.std,
                                                  wl.out_dtype)
        return oracle.yuv420_lowres_preprocess_batch(wl.src, wl.y_offsets, wl.cb_offsets,
                                                     wl.cr_offsets, wl.widths, wl.heights,
                                                     wl.low_res, wl.resize_short, wl.crop_h,
                                                     wl.crop_w, wl.mean, wl.std, wl.out_dtype)
    if wl.variant:
        if wl.kind == "rgb":
            return oracle.preprocess_batch_ex(wl.src, wl.offsets, wl.widths, wl.heights,
                                              wl.pitches, wl.rois, wl.resize_short, wl.crop_h,
                                              wl.crop_w, wl.mean, wl.std, wl.out_dtype,
                                              wl.resize_mode, wl.layout)
        return oracle.yuv420_preprocess_batch_ex(wl.src, wl.y_offsets, wl.cb_offsets,
                                                 wl.cr_offsets, wl.widths, wl.heights, wl.rois,
                                                 wl.resize_short, wl.crop_h, wl.crop_w, wl.mean,
                                                 wl.std, wl.out_dtype, wl.resize_mode, wl.layout,
                                                 wl.siting)
    if wl.kind == "rgb":
        return oracle.preprocess_batch(wl.src, wl.offsets, wl.widths, wl.heights, wl.pitches,
                                       wl.resize_short, wl.crop_h, wl.crop_w, wl.mean, wl.std,
                                       wl.out_dtype)
    return oracle.yuv420_preprocess_batch(wl.src, wl.y_offsets, wl.cb_offsets, wl.cr_offsets,
                                          wl.widths, wl.heights, wl.resize_short, wl.crop_h,
                                          wl.crop_w, wl.mean, wl.std, wl.out_dtype)


def upload(wl: synthetic.Workload, pad_front: int = 0):
    """Copy wl.src to the device. pad_front > 0 places it at a byte offset in a
    larger allocation (to exercise unaligned src pointers)."""
    import torch
    buf = torch.empty(wl.src.size + pad_front, dtype=torch.uint8, device="cuda:0")
    view = buf[pad_front:]
    view.copy_(torch.from_numpy(wl.src))
    return buf, view


def run_gpu(wl: synthetic.Workload, pad_front: int = 0, stream=None) -> np.ndarray:
    import torch
    note(f"[gpu] {wl.name}: n={wl.n} kind={wl.kind} S={wl.resize_short} "
         f"crop={wl.crop_h}x{wl.crop_w} dtype={('f32', 'f16', 'u8')[wl.out_dtype]} "
         f"low_res={wl.low_res}")
    _, src = upload(wl, pad_front)
    out = smol.run_workload(wl, src, stream=stream)
    torch.cuda.synchronize()
    res = out.cpu().numpy()
    return res


def f16_ordered(bits: np.ndarray) -> np.ndarray:
    b = bits.astype(np.int32)
    mag = b & 0x7FFF
    return np.where(b & 0x8000, -mag, mag)


def assert_parity(gpu: np.ndarray, ref: np.ndarray, out_dtype: int, what: str = "") -> dict:
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    if out_dtype == smol.OUT_U8:
        assert gpu.dtype == np.uint8 and ref.dtype == np.uint8
        bad = np.argwhere(gpu != ref)
        if bad.size:
            i = tuple(bad[0])
            raise AssertionError(f"{what}: {len(bad)} uint8 outputs differ, first at {i}: "
                                 f"gpu {gpu[i]} oracle {ref[i]}")
        return {"exact_frac": 1.0}
    if out_dtype == smol.OUT_F32:
        assert gpu.dtype == np.float32 and ref.dtype == np.float32
        assert np.all(np.isfinite(gpu)), what
        err = np.abs(gpu.astype(np.float64) - ref.astype(np.float64))
        worst = float(err.max()) if err.size else 0.0
        if worst > F32_TOL:
            i = np.unravel_index(int(err.argmax()), err.shape)
            raise AssertionError(f"{what}: max |gpu - oracle| = {worst:.3e} > {F32_TOL} at {i}: "
                                 f"gpu {gpu[i]!r} oracle {ref[i]!r}")
        return {"max_abs": worst, "exact_frac": float(np.mean(err == 0)) if err.size else 1.0}
    assert gpu.dtype == np.float16 and ref.dtype == np.float16
    d = np.abs(f16_ordered(gpu.view(np.uint16)) - f16_ordered(ref.view(np.uint16)))
    worst = int(d.max()) if d.size else 0
    if worst > F16_ULP:
        i = np.unravel_index(int(d.argmax()), d.shape)
        raise AssertionError(f"{what}: fp16 distance {worst} ulp > {F16_ULP} at {i}: "
                             f"gpu {gpu[i]!r} oracle {ref[i]!r}")
    return {"max_ulp": worst, "exact_frac": float(np.mean(d == 0)) if d.size else 1.0}
