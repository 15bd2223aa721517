"""Plain CPU oracle for fused image preprocessing -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. It wraps ``smol_oracle.c`` (plain scalar
C, fp32, no FMA contraction) through ctypes. It shares no code with the HIP
library in ``paper_2007_13005_amd``; neither imports the other.

What is computed, and which passage each step follows, is documented at the top
of ``smol_oracle.c``: the standard ResNet preprocessing of the paper's section 2
("Breakdown of end-to-end DNN inference", steps 2-4), the crop taken in output
space (section 6.2, reordering rule 3) at Algorithm 1's offsets, and the
colorspace conversion listed in App. A ("Components"); and the variants and
the low-resolution augmentation (section 5.3) described there too.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "smol_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libsmol_oracle.so")

OUT_F32 = 0
OUT_F16 = 1
OUT_U8 = 2
RESIZE_SHORT_CROP = 0
RESIZE_DIRECT = 1
NCHW = 0
NHWC = 1
CHROMA_CENTER = 0
CHROMA_LEFT = 1

# No -ffast-math, no -march: x86-64 SSE arithmetic is exact IEEE binary32, and
# -ffp-contract=off keeps every multiply and add rounded on its own.
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]


def build(verbose: bool = False) -> str:
    """Compile the oracle with gcc into ``oracle/libsmol_oracle.so``."""
    cmd = ["gcc", *CFLAGS, "-o", _LIB_PATH + ".tmp", _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


_lib = None

_i64p = ctypes.POINTER(ctypes.c_int64)
_i32p = ctypes.POINTER(ctypes.c_int32)
_f32p = ctypes.POINTER(ctypes.c_float)
_u8p = ctypes.POINTER(ctypes.c_uint8)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.oracle_resized_dims.argtypes = [ctypes.c_int64] * 3 + [_i64p, _i64p]
    lib.oracle_resized_dims.restype = None
    lib.oracle_crop_offsets.argtypes = [ctypes.c_int64] * 4 + [_i64p, _i64p]
    lib.oracle_crop_offsets.restype = None
    lib.oracle_axis_tap.argtypes = [ctypes.c_int64] * 3 + [_i64p, _i64p, _f32p]
    lib.oracle_axis_tap.restype = None
    lib.oracle_ycbcr_to_rgb.argtypes = [ctypes.c_float] * 3 + [_f32p]
    lib.oracle_ycbcr_to_rgb.restype = None
    lib.oracle_yuv420_to_rgb.argtypes = [ctypes.c_void_p] * 3 + [ctypes.c_int64] * 2 + [
        ctypes.c_void_p
    ]
    lib.oracle_yuv420_to_rgb.restype = None
    lib.oracle_f32_to_f16.argtypes = [ctypes.c_float]
    lib.oracle_f32_to_f16.restype = ctypes.c_uint16
    lib.smol_ref_preprocess_image.argtypes = [ctypes.c_void_p] + [ctypes.c_int32] * 6 + [
        ctypes.c_void_p,
        ctypes.c_void_p,
        ctypes.c_int32,
        ctypes.c_void_p,
    ]
    lib.smol_ref_preprocess_image.restype = ctypes.c_int
    lib.smol_ref_yuv420_preprocess_image.argtypes = [ctypes.c_void_p] * 3 + [
        ctypes.c_int32
    ] * 5 + [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]
    lib.smol_ref_yuv420_preprocess_image.restype = ctypes.c_int
    lib.smol_ref_preprocess_batch.argtypes = [
        ctypes.c_void_p,
        ctypes.c_int64,
        ctypes.c_void_p,
        ctypes.c_void_p,
        ctypes.c_void_p,
        ctypes.c_void_p,
        ctypes.c_int32,
        ctypes.c_int32,
        ctypes.c_int32,
        ctypes.c_int32,
        ctypes.c_void_p,
        ctypes.c_void_p,
        ctypes.c_int32,
        ctypes.c_void_p,
    ]
    lib.smol_ref_preprocess_batch.restype = ctypes.c_int
    lib.smol_ref_yuv420_preprocess_batch.argtypes = [
        ctypes.c_void_p,
        ctypes.c_int64,
        ctypes.c_void_p,
        ctypes.c_void_p,
        ctypes.c_void_p,
        ctypes.c_void_p,
        ctypes.c_void_p,
        ctypes.c_int32,
        ctypes.c_int32,
        ctypes.c_int32,
        ctypes.c_int32,
        ctypes.c_void_p,
        ctypes.c_void_p,
        ctypes.c_int32,
        ctypes.c_void_p,
    ]
    lib.smol_ref_yuv420_preprocess_batch.restype = ctypes.c_int
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.oracle_yuv420_to_rgb_sited.argtypes = [P, P, P, I64, I64, I32, P]
    lib.oracle_yuv420_to_rgb_sited.restype = None
    lib.oracle_output_geometry.argtypes = [I64] * 5 + [I32] + [_i64p] * 4
    lib.oracle_output_geometry.restype = None
    lib.smol_ref_preprocess_batch_ex.argtypes = [P, I64, P, P, P, P, P, I32, I32, I32, I32, P, P,
                                                 I32, I32, I32, P]
    lib.smol_ref_preprocess_batch_ex.restype = ctypes.c_int
    lib.smol_ref_yuv420_preprocess_batch_ex.argtypes = [P, I64, P, P, P, P, P, P, I32, I32, I32,
                                                        I32, P, P, I32, I32, I32, I32, P]
    lib.smol_ref_yuv420_preprocess_batch_ex.restype = ctypes.c_int
    lib.smol_ref_preprocess_image_ex.argtypes = [P] + [I32] * 10 + [P, P, I32, I32, I32, P]
    lib.smol_ref_preprocess_image_ex.restype = ctypes.c_int
    lib.smol_ref_yuv420_preprocess_image_ex.argtypes = [P, P, P] + [I32] * 9 + [P, P, I32, I32,
                                                                                  I32, I32, P]
    lib.smol_ref_yuv420_preprocess_image_ex.restype = ctypes.c_int
    lib.smol_ref_lowres_preprocess_batch.argtypes = [P, I64, P, P, P, P] + [I32] * 5 + [P, P, I32,
                                                                                        P]
    lib.smol_ref_lowres_preprocess_batch.restype = ctypes.c_int
    lib.smol_ref_yuv420_lowres_preprocess_batch.argtypes = [P, I64, P, P, P, P, P] + [I32] * 5 + [
        P, P, I32, P]
    lib.smol_ref_yuv420_lowres_preprocess_batch.restype = ctypes.c_int
    lib.smol_ref_lowres_preprocess_image.argtypes = [P] + [I32] * 7 + [P, P, I32, P]
    lib.smol_ref_lowres_preprocess_image.restype = ctypes.c_int
    lib.smol_ref_yuv420_lowres_preprocess_image.argtypes = [P, P, P] + [I32] * 6 + [P, P, I32, P]
    lib.smol_ref_yuv420_lowres_preprocess_image.restype = ctypes.c_int
    lib.oracle_idct_block.argtypes = [P, P, P, I64, I32, I32]
    lib.oracle_idct_block.restype = None
    lib.oracle_jpeg_coef_count.argtypes = [I32, I32]
    lib.oracle_jpeg_coef_count.restype = I64
    lib.oracle_jpeg_mcu_rect.argtypes = [I32] * 6 + [P]
    lib.oracle_jpeg_mcu_rect.restype = ctypes.c_int
    lib.oracle_jpeg_decode_i420.argtypes = [P, P, P, I32, I32, P, P, P, P]
    lib.oracle_jpeg_decode_i420.restype = ctypes.c_int
    lib.oracle_jpeg_entropy_decode.argtypes = [P, I64, P, I64, P, P, P, P]
    lib.oracle_jpeg_entropy_decode.restype = ctypes.c_int
    _lib = lib
    return lib


def lib():
    """The loaded ctypes library (built on first use)."""
    return _load()


# --------------------------------------------------------------------------
# scalar helpers
# --------------------------------------------------------------------------


def resized_dims(W: int, H: int, S: int) -> tuple[int, int]:
    a, b = ctypes.c_int64(), ctypes.c_int64()
    _load().oracle_resized_dims(W, H, S, ctypes.byref(a), ctypes.byref(b))
    return a.value, b.value


def crop_offsets(Wr: int, Hr: int, Ch: int, Cw: int) -> tuple[int, int]:
    a, b = ctypes.c_int64(), ctypes.c_int64()
    _load().oracle_crop_offsets(Wr, Hr, Ch, Cw, ctypes.byref(a), ctypes.byref(b))
    return a.value, b.value


def axis_tap(x: int, n_in: int, n_out: int) -> tuple[int, int, float]:
    a, b, w = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_float()
    _load().oracle_axis_tap(x, n_in, n_out, ctypes.byref(a), ctypes.byref(b), ctypes.byref(w))
    return a.value, b.value, w.value


def ycbcr_to_rgb(Y: float, Cb: float, Cr: float) -> np.ndarray:
    out = np.zeros(3, np.float32)
    _load().oracle_ycbcr_to_rgb(Y, Cb, Cr, out.ctypes.data_as(_f32p))
    return out


def f32_to_f16_bits(x: float) -> int:
    return int(_load().oracle_f32_to_f16(float(np.float32(x))))


def yuv420_to_rgb(y: np.ndarray, cb: np.ndarray, cr: np.ndarray) -> np.ndarray:
    """Planes as 2-D uint8 arrays (H x W, ceil(H/2) x ceil(W/2)) -> H x W x 3 fp32."""
    H, W = y.shape
    y = np.ascontiguousarray(y, np.uint8)
    cb = np.ascontiguousarray(cb, np.uint8)
    cr = np.ascontiguousarray(cr, np.uint8)
    assert cb.shape == ((H + 1) // 2, (W + 1) // 2) and cr.shape == cb.shape
    out = np.empty((H, W, 3), np.float32)
    _load().oracle_yuv420_to_rgb(y.ctypes.data, cb.ctypes.data, cr.ctypes.data, W, H, out.ctypes.data)
    return out


# --------------------------------------------------------------------------
# whole-image / batch calls
# --------------------------------------------------------------------------


def _out_array(n: int, Ch: int, Cw: int, out_dtype: int) -> np.ndarray:
    if out_dtype not in _ELEM:
        raise ValueError("out_dtype must be OUT_F32, OUT_F16 or OUT_U8")
    return np.empty((n, 3, Ch, Cw), _ELEM[out_dtype])


def _finish(out: np.ndarray, out_dtype: int) -> np.ndarray:
    return out.view(np.float16) if out_dtype == OUT_F16 else out


_ELEM = {OUT_F32: np.float32, OUT_F16: np.uint16, OUT_U8: np.uint8}


def _vec3(v) -> np.ndarray:
    a = np.ascontiguousarray(np.asarray(v, dtype=np.float32).reshape(3))
    return a


def preprocess_image(img: np.ndarray, S: int, Ch: int, Cw: int, mean, std, out_dtype: int,
                     pitch: int | None = None, width: int | None = None,
                     height: int | None = None) -> np.ndarray:
    """One image. ``img`` is H x W x 3 uint8 (any row pitch via ``pitch`` on a
    flat buffer, in which case ``width``/``height`` are required)."""
    if pitch is None:
        img = np.ascontiguousarray(img, np.uint8)
        height, width = img.shape[0], img.shape[1]
        pitch = 3 * width
    m, s = _vec3(mean), _vec3(std)
    out = _out_array(1, Ch, Cw, out_dtype)
    rc = _load().smol_ref_preprocess_image(img.ctypes.data, width, height, pitch, S, Ch, Cw,
                                           m.ctypes.data, s.ctypes.data, out_dtype, out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return _finish(out, out_dtype)[0]


def preprocess_image_into(img_ptr: int, W: int, H: int, pitch: int, S: int, Ch: int, Cw: int,
                          mean: np.ndarray, std: np.ndarray, out_dtype: int, out_ptr: int) -> int:
    """Raw-pointer form used by the threaded CPU baseline (ctypes drops the GIL)."""
    return _load().smol_ref_preprocess_image(img_ptr, W, H, pitch, S, Ch, Cw, mean.ctypes.data,
                                             std.ctypes.data, out_dtype, out_ptr)


def yuv420_preprocess_image_into(y_ptr: int, cb_ptr: int, cr_ptr: int, W: int, H: int, S: int,
                                 Ch: int, Cw: int, mean: np.ndarray, std: np.ndarray,
                                 out_dtype: int, out_ptr: int) -> int:
    return _load().smol_ref_yuv420_preprocess_image(y_ptr, cb_ptr, cr_ptr, W, H, S, Ch, Cw,
                                                    mean.ctypes.data, std.ctypes.data, out_dtype,
                                                    out_ptr)


def preprocess_batch(src: np.ndarray, offsets, widths, heights, pitches, S: int, Ch: int, Cw: int,
                     mean, std, out_dtype: int) -> np.ndarray:
    """Ragged batch of packed HWC RGB uint8 images in the flat buffer ``src``."""
    src = np.ascontiguousarray(src, np.uint8).reshape(-1)
    n = len(offsets)
    off = np.ascontiguousarray(offsets, np.int64)
    w = np.ascontiguousarray(widths, np.int32)
    h = np.ascontiguousarray(heights, np.int32)
    p = None if pitches is None else np.ascontiguousarray(pitches, np.int32)
    m, s = _vec3(mean), _vec3(std)
    out = _out_array(n, Ch, Cw, out_dtype)
    rc = _load().smol_ref_preprocess_batch(src.ctypes.data, src.size, off.ctypes.data,
                                           w.ctypes.data, h.ctypes.data,
                                           None if p is None else p.ctypes.data, n, S, Ch, Cw,
                                           m.ctypes.data, s.ctypes.data, out_dtype,
                                           out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return _finish(out, out_dtype)


def yuv420_preprocess_batch(src: np.ndarray, y_offsets, cb_offsets, cr_offsets, widths, heights,
                            S: int, Ch: int, Cw: int, mean, std, out_dtype: int) -> np.ndarray:
    """Batch of planar I420 frames in the flat buffer ``src``."""
    src = np.ascontiguousarray(src, np.uint8).reshape(-1)
    n = len(y_offsets)
    yo = np.ascontiguousarray(y_offsets, np.int64)
    bo = np.ascontiguousarray(cb_offsets, np.int64)
    ro = np.ascontiguousarray(cr_offsets, np.int64)
    w = np.ascontiguousarray(widths, np.int32)
    h = np.ascontiguousarray(heights, np.int32)
    m, s = _vec3(mean), _vec3(std)
    out = _out_array(n, Ch, Cw, out_dtype)
    rc = _load().smol_ref_yuv420_preprocess_batch(src.ctypes.data, src.size, yo.ctypes.data,
                                                  bo.ctypes.data, ro.ctypes.data, w.ctypes.data,
                                                  h.ctypes.data, n, S, Ch, Cw, m.ctypes.data,
                                                  s.ctypes.data, out_dtype, out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return _finish(out, out_dtype)


# --------------------------------------------------------------------------
# variants: region of interest, direct resize, NHWC, left-sited chroma
# --------------------------------------------------------------------------


def output_geometry(W: int, H: int, S: int, Ch: int, Cw: int,
                    resize_mode: int = RESIZE_SHORT_CROP) -> tuple[int, int, int, int]:
    """(Wr, Hr, left, top) of a W x H image (or ROI)."""
    v = [ctypes.c_int64() for _ in range(4)]
    _load().oracle_output_geometry(W, H, S, Ch, Cw, resize_mode, *[ctypes.byref(x) for x in v])
    return tuple(x.value for x in v)


def yuv420_to_rgb_sited(y: np.ndarray, cb: np.ndarray, cr: np.ndarray,
                        siting: int = CHROMA_CENTER) -> np.ndarray:
    """As ``yuv420_to_rgb`` with the chroma siting chosen."""
    H, W = y.shape
    y = np.ascontiguousarray(y, np.uint8)
    cb = np.ascontiguousarray(cb, np.uint8)
    cr = np.ascontiguousarray(cr, np.uint8)
    assert cb.shape == ((H + 1) // 2, (W + 1) // 2) and cr.shape == cb.shape
    out = np.empty((H, W, 3), np.float32)
    _load().oracle_yuv420_to_rgb_sited(y.ctypes.data, cb.ctypes.data, cr.ctypes.data, W, H,
                                       siting, out.ctypes.data)
    return out


def _out_array_ex(n: int, Ch: int, Cw: int, out_dtype: int, layout: int) -> np.ndarray:
    shape = (n, Ch, Cw, 3) if layout == NHWC else (n, 3, Ch, Cw)
    if out_dtype not in _ELEM:
        raise ValueError("out_dtype must be OUT_F32, OUT_F16 or OUT_U8")
    return np.empty(shape, _ELEM[out_dtype])


def _rois(rois, n: int):
    if rois is None:
        return None
    r = np.ascontiguousarray(rois, np.int32).reshape(n, 4)
    return r


def preprocess_batch_ex(src: np.ndarray, offsets, widths, heights, pitches, rois, S: int,
                        Ch: int, Cw: int, mean, std, out_dtype: int,
                        resize_mode: int = RESIZE_SHORT_CROP, layout: int = NCHW) -> np.ndarray:
    """RGB batch with an optional ROI per image ((x, y, w, h) rows), the
    resize mode and the output layout."""
    src = np.ascontiguousarray(src, np.uint8).reshape(-1)
    n = len(offsets)
    off = np.ascontiguousarray(offsets, np.int64)
    w = np.ascontiguousarray(widths, np.int32)
    h = np.ascontiguousarray(heights, np.int32)
    p = None if pitches is None else np.ascontiguousarray(pitches, np.int32)
    r = _rois(rois, n)
    m, s = _vec3(mean), _vec3(std)
    out = _out_array_ex(n, Ch, Cw, out_dtype, layout)
    rc = _load().smol_ref_preprocess_batch_ex(
        src.ctypes.data, src.size, off.ctypes.data, w.ctypes.data, h.ctypes.data,
        None if p is None else p.ctypes.data, None if r is None else r.ctypes.data, n, S, Ch, Cw,
        m.ctypes.data, s.ctypes.data, out_dtype, resize_mode, layout, out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return _finish(out, out_dtype)


def yuv420_preprocess_batch_ex(src: np.ndarray, y_offsets, cb_offsets, cr_offsets, widths,
                               heights, rois, S: int, Ch: int, Cw: int, mean, std, out_dtype: int,
                               resize_mode: int = RESIZE_SHORT_CROP, layout: int = NCHW,
                               siting: int = CHROMA_CENTER) -> np.ndarray:
    """I420 batch with an optional ROI per frame, resize mode, layout and
    chroma siting."""
    src = np.ascontiguousarray(src, np.uint8).reshape(-1)
    n = len(y_offsets)
    yo = np.ascontiguousarray(y_offsets, np.int64)
    bo = np.ascontiguousarray(cb_offsets, np.int64)
    ro = np.ascontiguousarray(cr_offsets, np.int64)
    w = np.ascontiguousarray(widths, np.int32)
    h = np.ascontiguousarray(heights, np.int32)
    r = _rois(rois, n)
    m, s = _vec3(mean), _vec3(std)
    out = _out_array_ex(n, Ch, Cw, out_dtype, layout)
    rc = _load().smol_ref_yuv420_preprocess_batch_ex(
        src.ctypes.data, src.size, yo.ctypes.data, bo.ctypes.data, ro.ctypes.data, w.ctypes.data,
        h.ctypes.data, None if r is None else r.ctypes.data, n, S, Ch, Cw, m.ctypes.data,
        s.ctypes.data, out_dtype, resize_mode, layout, siting, out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return _finish(out, out_dtype)


def preprocess_image_ex_into(img_ptr: int, W: int, H: int, pitch: int, roi, S: int, Ch: int,
                             Cw: int, mean: np.ndarray, std: np.ndarray, out_dtype: int,
                             resize_mode: int, layout: int, out_ptr: int) -> int:
    """Raw-pointer form of one RGB image with its ROI (x, y, w, h) and options."""
    x, y, w, h = roi
    return _load().smol_ref_preprocess_image_ex(img_ptr, W, H, pitch, x, y, w, h, S, Ch, Cw,
                                                mean.ctypes.data, std.ctypes.data, out_dtype,
                                                resize_mode, layout, out_ptr)


def yuv420_preprocess_image_ex_into(y_ptr: int, cb_ptr: int, cr_ptr: int, W: int, H: int, roi,
                                    S: int, Ch: int, Cw: int, mean: np.ndarray, std: np.ndarray,
                                    out_dtype: int, resize_mode: int, layout: int, siting: int,
                                    out_ptr: int) -> int:
    """Raw-pointer form of one I420 frame with its ROI and options."""
    x, y, w, h = roi
    return _load().smol_ref_yuv420_preprocess_image_ex(y_ptr, cb_ptr, cr_ptr, W, H, x, y, w, h,
                                                       S, Ch, Cw, mean.ctypes.data,
                                                       std.ctypes.data, out_dtype, resize_mode,
                                                       layout, siting, out_ptr)


# --------------------------------------------------------------------------
# low-resolution-aware augmentation (section 5.3)
# --------------------------------------------------------------------------


def lowres_preprocess_batch(src: np.ndarray, offsets, widths, heights, pitches, r: int, S: int,
                            Ch: int, Cw: int, mean, std, out_dtype: int) -> np.ndarray:
    """RGB batch: each image reduced to the r x r uint8 image, then steps 2-4."""
    src = np.ascontiguousarray(src, np.uint8).reshape(-1)
    n = len(offsets)
    off = np.ascontiguousarray(offsets, np.int64)
    w = np.ascontiguousarray(widths, np.int32)
    h = np.ascontiguousarray(heights, np.int32)
    p = None if pitches is None else np.ascontiguousarray(pitches, np.int32)
    m, s = _vec3(mean), _vec3(std)
    out = _out_array(n, Ch, Cw, out_dtype)
    rc = _load().smol_ref_lowres_preprocess_batch(
        src.ctypes.data, src.size, off.ctypes.data, w.ctypes.data, h.ctypes.data,
        None if p is None else p.ctypes.data, n, r, S, Ch, Cw, m.ctypes.data, s.ctypes.data,
        out_dtype, out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return _finish(out, out_dtype)


def yuv420_lowres_preprocess_batch(src: np.ndarray, y_offsets, cb_offsets, cr_offsets, widths,
                                   heights, r: int, S: int, Ch: int, Cw: int, mean, std,
                                   out_dtype: int) -> np.ndarray:
    """I420 batch: each frame converted and reduced to the r x r uint8 RGB
    image, then steps 2-4."""
    src = np.ascontiguousarray(src, np.uint8).reshape(-1)
    n = len(y_offsets)
    yo = np.ascontiguousarray(y_offsets, np.int64)
    bo = np.ascontiguousarray(cb_offsets, np.int64)
    ro = np.ascontiguousarray(cr_offsets, np.int64)
    w = np.ascontiguousarray(widths, np.int32)
    h = np.ascontiguousarray(heights, np.int32)
    m, s = _vec3(mean), _vec3(std)
    out = _out_array(n, Ch, Cw, out_dtype)
    rc = _load().smol_ref_yuv420_lowres_preprocess_batch(
        src.ctypes.data, src.size, yo.ctypes.data, bo.ctypes.data, ro.ctypes.data, w.ctypes.data,
        h.ctypes.data, n, r, S, Ch, Cw, m.ctypes.data, s.ctypes.data, out_dtype, out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return _finish(out, out_dtype)


def lowres_preprocess_image_into(img_ptr: int, W: int, H: int, pitch: int, r: int, S: int,
                                 Ch: int, Cw: int, mean: np.ndarray, std: np.ndarray,
                                 out_dtype: int, out_ptr: int) -> int:
    """Raw-pointer form of one RGB image (the threaded CPU baseline)."""
    return _load().smol_ref_lowres_preprocess_image(img_ptr, W, H, pitch, r, S, Ch, Cw,
                                                    mean.ctypes.data, std.ctypes.data, out_dtype,
                                                    out_ptr)


def yuv420_lowres_preprocess_image_into(y_ptr: int, cb_ptr: int, cr_ptr: int, W: int, H: int,
                                        r: int, S: int, Ch: int, Cw: int, mean: np.ndarray,
                                        std: np.ndarray, out_dtype: int, out_ptr: int) -> int:
    """Raw-pointer form of one I420 frame."""
    return _load().smol_ref_yuv420_lowres_preprocess_image(y_ptr, cb_ptr, cr_ptr, W, H, r, S, Ch,
                                                           Cw, mean.ctypes.data, std.ctypes.data,
                                                           out_dtype, out_ptr)


# --------------------------------------------------------------------------
# partial JPEG decoding (section 6.4, "ROI decoding", Algorithm 1)
# --------------------------------------------------------------------------


def idct_block(coef, q) -> np.ndarray:
    """One 8 x 8 block of int16 coefficients (natural order) dequantised by q
    (uint16), inverse-DCT'd, level-shifted, rounded and clamped: uint8 8 x 8."""
    c = np.ascontiguousarray(coef, np.int16).reshape(64)
    qq = np.ascontiguousarray(q, np.uint16).reshape(64)
    out = np.empty((8, 8), np.uint8)
    _load().oracle_idct_block(c.ctypes.data, qq.ctypes.data, out.ctypes.data, 8, 8, 8)
    return out


def jpeg_coef_count(W: int, H: int) -> int:
    """int16 coefficients of one W x H 4:2:0 frame (MCU-padded block grid)."""
    return int(_load().oracle_jpeg_coef_count(W, H))


def jpeg_mcu_rect(W: int, H: int, S: int, Ch: int, Cw: int,
                  resize_mode: int = RESIZE_SHORT_CROP) -> tuple[int, int, int, int]:
    """Algorithm 1's MCU-aligned rectangle (x, y, w, h) for a W x H frame."""
    r = np.zeros(4, np.int32)
    if _load().oracle_jpeg_mcu_rect(W, H, S, Ch, Cw, resize_mode, r.ctypes.data) != 0:
        raise ValueError("oracle rejected the arguments")
    return tuple(int(v) for v in r)


def jpeg_decode_i420(coef, qy, qc, W: int, H: int, rect=None, fill: int | None = None):
    """Decode the blocks of a frame that meet ``rect`` (None: all) into
    full-size I420 planes (y, cb, cr); pixels outside stay ``fill`` (or
    uninitialised when None)."""
    c = np.ascontiguousarray(coef, np.int16).reshape(-1)
    assert c.size == jpeg_coef_count(W, H)
    qy = np.ascontiguousarray(qy, np.uint16).reshape(64)
    qc = np.ascontiguousarray(qc, np.uint16).reshape(64)
    Wc, Hc = (W + 1) // 2, (H + 1) // 2
    mk = (lambda shape: np.full(shape, fill, np.uint8)) if fill is not None else (
        lambda shape: np.empty(shape, np.uint8))
    y, cb, cr = mk((H, W)), mk((Hc, Wc)), mk((Hc, Wc))
    r = None if rect is None else np.ascontiguousarray(rect, np.int32)
    rc = _load().oracle_jpeg_decode_i420(c.ctypes.data, qy.ctypes.data, qc.ctypes.data, W, H,
                                         None if r is None else r.ctypes.data, y.ctypes.data,
                                         cb.ctypes.data, cr.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return y, cb, cr


def jpeg_entropy_decode(data: bytes):
    """Entropy-decode a whole baseline 4:2:0 JPEG stream (T.81, Annex F):
    (coefficients int16 in the library's block layout, luma table, chroma
    table (natural order, uint16[64] each), W, H). Raises ValueError on a
    stream outside the accepted subset or a corrupt one."""
    buf = np.frombuffer(bytes(data), np.uint8)
    qy, qc = np.zeros(64, np.uint16), np.zeros(64, np.uint16)
    W, H = ctypes.c_int32(0), ctypes.c_int32(0)
    lib_ = _load()
    if lib_.oracle_jpeg_entropy_decode(buf.ctypes.data, buf.size, None, 0, qy.ctypes.data,
                                       qc.ctypes.data, ctypes.byref(W), ctypes.byref(H)) != 0:
        raise ValueError("oracle rejected the stream")
    coef = np.zeros(jpeg_coef_count(W.value, H.value), np.int16)
    if lib_.oracle_jpeg_entropy_decode(buf.ctypes.data, buf.size, coef.ctypes.data, coef.size,
                                       qy.ctypes.data, qc.ctypes.data, ctypes.byref(W),
                                       ctypes.byref(H)) != 0:
        raise ValueError("oracle rejected the stream")
    return coef, qy, qc, W.value, H.value
