"""Thin ctypes binding over libsmol.so (the C ABI declared in include/smol.h).

Argument marshalling only: every step of the preprocessing runs in the HIP
kernels behind the C ABI. torch supplies device memory and the stream. If the
library has not been built this module raises on first use; there is no CPU
fallback.
"""
from __future__ import annotations

import ctypes
import os
import sys
import threading

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsmol.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_UNSUPPORTED = -2
ERR_HIP = -3

OUT_F32 = 0
OUT_F16 = 1
OUT_U8 = 2

PATH_AUTO = 0
PATH_DIRECT = 1
PATH_LDS = 2
PATH_GATHER = 3
PATH_ROWS = 4

RESIZE_SHORT_CROP = 0
RESIZE_DIRECT = 1
LAYOUT_NCHW = 0
LAYOUT_NHWC = 1
JPEG_COEF_FRAME = 0
JPEG_COEF_WINDOW = 1
CHROMA_CENTER = 0
CHROMA_LEFT = 1

MAX_DIM = 65535
MAX_RESIZED = 4194303
MAX_BATCH = 1048576


class Params(ctypes.Structure):
    _fields_ = [("resize_short", ctypes.c_int32), ("crop_h", ctypes.c_int32),
                ("crop_w", ctypes.c_int32), ("out_dtype", ctypes.c_int32),
                ("mean", ctypes.c_float * 3), ("std", ctypes.c_float * 3)]


class Geometry(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in (
        "resized_w", "resized_h", "crop_left", "crop_top", "src_x_first", "src_x_last",
        "src_rows", "chroma_x_first", "chroma_x_last", "chroma_rows")]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_}


class Options(ctypes.Structure):
    _fields_ = [("resize_mode", ctypes.c_int32), ("layout", ctypes.c_int32),
                ("chroma_siting", ctypes.c_int32), ("reserved", ctypes.c_int32 * 5)]


class Tuning(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int32), ("band_rows", ctypes.c_int32),
                ("lds_budget", ctypes.c_int32), ("workgroups_per_cu", ctypes.c_int32),
                ("exact", ctypes.c_int32), ("row_order", ctypes.c_int32),
                ("upload", ctypes.c_int32), ("reserved", ctypes.c_int32 * 1)]


class Plan(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int32), ("band_rows", ctypes.c_int32),
                ("lds_bytes", ctypes.c_int32), ("launches", ctypes.c_int32),
                ("uploaded_descriptors", ctypes.c_int32), ("grid", ctypes.c_int32),
                ("work_items", ctypes.c_int64)]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_}


class PipelineConfig(ctypes.Structure):
    _fields_ = [("slots", ctypes.c_int32), ("streams", ctypes.c_int32),
                ("input_bytes", ctypes.c_int64), ("output_bytes", ctypes.c_int64),
                ("copy_streams", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_int64)]


class PipelineStats(ctypes.Structure):
    _fields_ = [("submitted", ctypes.c_int64), ("completed", ctypes.c_int64),
                ("images", ctypes.c_int64), ("bytes_copied", ctypes.c_int64),
                ("acquire_waits", ctypes.c_int64), ("reserved", ctypes.c_int64 * 3)]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_ if name != "reserved"}


class JpegInfo(ctypes.Structure):
    _fields_ = [("width", ctypes.c_int32), ("height", ctypes.c_int32),
                ("restart_interval", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("scan_offset", ctypes.c_int64), ("qtables", ctypes.c_uint16 * 128)]


# smol_consumer_fn: int (*)(void *user, const void *output, int32_t n, void *stream)
CONSUMER = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                            ctypes.c_void_p)

# Every symbol include/*.h declares, with its ctypes signature.
_vp = ctypes.c_void_p
SIGNATURES = {
    "smol_preprocess_batch": (ctypes.c_int, [_vp, ctypes.c_int64, _vp, _vp, _vp, _vp,
                                             ctypes.c_int32, ctypes.POINTER(Params), _vp, _vp]),
    "smol_preprocess_batch_noalloc": (ctypes.c_int, [_vp, ctypes.c_int64, _vp, _vp, _vp, _vp,
                                                     ctypes.c_int32, ctypes.POINTER(Params), _vp,
                                                     _vp]),
    "smol_yuv420_preprocess_batch": (ctypes.c_int, [_vp, ctypes.c_int64, _vp, _vp, _vp, _vp, _vp,
                                                    ctypes.c_int32, ctypes.POINTER(Params), _vp,
                                                    _vp]),
    "smol_image_geometry": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.POINTER(Params), ctypes.POINTER(Geometry)]),
    "smol_preprocess_batch_ex": (ctypes.c_int, [_vp, ctypes.c_int64, _vp, _vp, _vp, _vp, _vp,
                                                ctypes.c_int32, ctypes.POINTER(Params),
                                                ctypes.POINTER(Options), _vp, _vp]),
    "smol_yuv420_preprocess_batch_ex": (ctypes.c_int, [_vp, ctypes.c_int64, _vp, _vp, _vp, _vp,
                                                       _vp, _vp, ctypes.c_int32,
                                                       ctypes.POINTER(Params),
                                                       ctypes.POINTER(Options), _vp, _vp]),
    "smol_image_geometry_ex": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp,
                                              ctypes.POINTER(Params), ctypes.POINTER(Options),
                                              ctypes.POINTER(Geometry)]),
    "smol_lowres_workspace_bytes": (ctypes.c_int64, [ctypes.c_int32, ctypes.c_int32]),
    "smol_lowres_preprocess_batch": (ctypes.c_int, [_vp, ctypes.c_int64, _vp, _vp, _vp, _vp,
                                                    ctypes.c_int32, ctypes.c_int32,
                                                    ctypes.POINTER(Params), _vp, ctypes.c_int64,
                                                    _vp, _vp]),
    "smol_yuv420_lowres_preprocess_batch": (ctypes.c_int, [_vp, ctypes.c_int64, _vp, _vp, _vp,
                                                           _vp, _vp, ctypes.c_int32,
                                                           ctypes.c_int32, ctypes.POINTER(Params),
                                                           _vp, ctypes.c_int64, _vp, _vp]),
    "smol_pipeline_create": (ctypes.c_int, [ctypes.POINTER(PipelineConfig),
                                            ctypes.POINTER(ctypes.c_void_p)]),
    "smol_pipeline_destroy": (ctypes.c_int, [_vp]),
    "smol_pipeline_acquire": (ctypes.c_int, [_vp, ctypes.POINTER(ctypes.c_int32),
                                             ctypes.POINTER(ctypes.c_void_p),
                                             ctypes.POINTER(ctypes.c_void_p)]),
    "smol_pipeline_release": (ctypes.c_int, [_vp, ctypes.c_int32]),
    "smol_pipeline_submit": (ctypes.c_int, [_vp, ctypes.c_int32, ctypes.c_int64, _vp, _vp, _vp,
                                            _vp, _vp, ctypes.c_int32, ctypes.POINTER(Params),
                                            ctypes.POINTER(Options), CONSUMER, _vp]),
    "smol_pipeline_submit_yuv420": (ctypes.c_int, [_vp, ctypes.c_int32, ctypes.c_int64, _vp, _vp,
                                                   _vp, _vp, _vp, _vp, ctypes.c_int32,
                                                   ctypes.POINTER(Params),
                                                   ctypes.POINTER(Options), CONSUMER, _vp]),
    "smol_pipeline_submit_jpeg": (ctypes.c_int, [_vp, ctypes.c_int32, ctypes.c_int64, _vp, _vp,
                                                 ctypes.c_int32, _vp, _vp, ctypes.c_int32,
                                                 ctypes.c_int32, ctypes.POINTER(Params),
                                                 ctypes.POINTER(Options), CONSUMER, _vp]),
    "smol_pipeline_drain": (ctypes.c_int, [_vp]),
    "smol_pipeline_get_stats": (ctypes.c_int, [_vp, ctypes.POINTER(PipelineStats)]),
    "smol_jpeg_coef_count": (ctypes.c_int64, [ctypes.c_int32, ctypes.c_int32]),
    "smol_jpeg_mcu_rect": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(Params),
                                          ctypes.POINTER(Options), _vp]),
    "smol_jpeg_decode_i420": (ctypes.c_int, [_vp, ctypes.c_int64, _vp, _vp, ctypes.c_int32,
                                             _vp, _vp, _vp, ctypes.c_int32, ctypes.c_int32, _vp,
                                             ctypes.c_int64, _vp, _vp, _vp, _vp]),
    "smol_jpeg_window_coef_count": (ctypes.c_int64, [ctypes.c_int32, ctypes.c_int32, _vp]),
    "smol_jpeg_workspace_bytes": (ctypes.c_int64, [ctypes.c_int32, _vp, _vp]),
    "smol_jpeg_roi_preprocess_batch": (ctypes.c_int, [_vp, ctypes.c_int64, _vp, _vp,
                                                      ctypes.c_int32, _vp, _vp, ctypes.c_int32,
                                                      ctypes.c_int32, ctypes.POINTER(Params),
                                                      ctypes.POINTER(Options), _vp,
                                                      ctypes.c_int64, _vp, _vp]),
    "smol_jpeg_read_info": (ctypes.c_int, [_vp, ctypes.c_int64, ctypes.POINTER(JpegInfo)]),
    "smol_jpeg_entropy_decode_batch": (ctypes.c_int, [_vp, ctypes.c_int64, _vp, _vp,
                                                      ctypes.c_int32, _vp, _vp, ctypes.c_int64,
                                                      _vp, ctypes.c_int32, _vp, ctypes.c_int32]),
    "smol_stream_probe": (ctypes.c_int, [_vp, ctypes.c_uint64, _vp, ctypes.c_uint64,
                                         ctypes.c_int32, ctypes.c_int32, _vp]),
    "smol_valu_probe": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp, _vp]),
    "smol_set_tuning": (ctypes.c_int, [ctypes.POINTER(Tuning)]),
    "smol_last_plan": (ctypes.c_int, [ctypes.POINTER(Plan)]),
    "smol_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "smol_last_error": (ctypes.c_char_p, []),
    "smol_version": (ctypes.c_int, []),
}

_lib = None


class SmolError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        super().__init__(f"smol status {status}: {detail}")


def lib() -> ctypes.CDLL:
    """Load libsmol.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2007_13005_amd.build` (needs hipcc)")
    # torch ships its own HIP runtime with the same soname (libamdhip64.so.7).
    # Loading torch first makes libsmol bind to that runtime, so that torch's
    # device pointers and streams and libsmol's launches share one runtime.
    import torch  # noqa: F401
    handle = ctypes.CDLL(LIB_PATH)
    runtimes = _mapped_hip_runtimes()
    if len(runtimes) > 1:
        raise RuntimeError(f"two HIP runtimes are loaded in this process: {runtimes}")
    bind_signatures(handle)
    _lib = handle
    return handle


def bind_signatures(handle: ctypes.CDLL, required: bool = True) -> ctypes.CDLL:
    """Type every declared symbol of a loaded build of the library (a build
    of only some of its files may skip the missing ones)."""
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(handle, name, None)
        if fn is None:
            if required:
                raise RuntimeError(f"{name} is missing from the library")
            continue
        fn.restype = res
        fn.argtypes = args
    return handle


def _mapped_hip_runtimes() -> list[str]:
    try:
        with open("/proc/self/maps") as f:
            paths = {line.split()[-1] for line in f if "libamdhip64" in line}
    except OSError:
        return []
    return sorted({os.path.realpath(p) for p in paths})


_hip = None


def hip_runtime() -> ctypes.CDLL:
    """The HIP runtime this library is bound to (the one torch loaded), with
    ``hipMemcpyAsync`` typed: for consumers that enqueue their own copies."""
    global _hip
    if _hip is None:
        lib()
        rt = _mapped_hip_runtimes()
        if not rt:
            raise RuntimeError("no HIP runtime is loaded")
        h = ctypes.CDLL(rt[0])
        h.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                     ctypes.c_int, ctypes.c_void_p]
        h.hipMemcpyAsync.restype = ctypes.c_int
        _hip = h
    return _hip


HIP_MEMCPY_DEVICE_TO_DEVICE = 3


def _check(status: int) -> None:
    if status != OK:
        detail = lib().smol_last_error().decode() or lib().smol_status_string(status).decode()
        raise SmolError(status, detail)


def make_params(resize_short: int, crop_h: int, crop_w: int, mean, std, out_dtype: int) -> Params:
    p = Params()
    p.resize_short, p.crop_h, p.crop_w, p.out_dtype = resize_short, crop_h, crop_w, out_dtype
    m = np.asarray(mean, np.float32).reshape(3)
    s = np.asarray(std, np.float32).reshape(3)
    for c in range(3):
        p.mean[c] = float(m[c])
        p.std[c] = float(s[c])
    return p


def make_options(resize_mode: int = RESIZE_SHORT_CROP, layout: int = LAYOUT_NCHW,
                 chroma_siting: int = CHROMA_CENTER) -> Options:
    o = Options()
    o.resize_mode, o.layout, o.chroma_siting = resize_mode, layout, chroma_siting
    return o


def image_geometry_ex(width: int, height: int, params: Params, yuv420: bool = False,
                      roi=None, options: Options | None = None) -> dict:
    """Geometry of an ROI (x, y, w, h) of a width x height image under options."""
    g = Geometry()
    r = None if roi is None else _table(roi, np.int32).reshape(4)
    _check(lib().smol_image_geometry_ex(width, height, int(bool(yuv420)),
                                        None if r is None else r.ctypes.data, ctypes.byref(params),
                                        None if options is None else ctypes.byref(options),
                                        ctypes.byref(g)))
    return g.as_dict()


def image_geometry(width: int, height: int, params: Params, yuv420: bool = False) -> dict:
    g = Geometry()
    _check(lib().smol_image_geometry(width, height, int(bool(yuv420)), ctypes.byref(params),
                                     ctypes.byref(g)))
    return g.as_dict()


def set_tuning(path: int = 0, band_rows: int = 0, lds_budget: int = 0,
               workgroups_per_cu: int = 0, exact: int = 0, row_order: int = 0,
               upload: int = 0) -> None:
    t = Tuning(path, band_rows, lds_budget, workgroups_per_cu, exact, row_order, upload)
    _check(lib().smol_set_tuning(ctypes.byref(t)))


def reset_tuning() -> None:
    _check(lib().smol_set_tuning(None))


def last_plan() -> dict:
    p = Plan()
    _check(lib().smol_last_plan(ctypes.byref(p)))
    return p.as_dict()


def version() -> int:
    return int(lib().smol_version())


STREAM_NT_LOADS = 1
STREAM_NT_STORES = 2
STREAM_DEEP = 4


def stream_probe(src: int, read_bytes: int, dst: int, write_bytes: int, waves: int,
                 flags: int = STREAM_NT_LOADS | STREAM_NT_STORES, stream: int = 0) -> None:
    """One launch of the streaming probe (raw device addresses, a raw stream
    handle): reads read_bytes at src, writes write_bytes at dst."""
    _check(lib().smol_stream_probe(src or None, read_bytes, dst or None, write_bytes, waves,
                                   flags, stream or None))


VALU_KINDS = ("mul_f32", "add_f32", "fma_f32", "perm", "alignbyte", "dot4", "med3_f32",
              "cvt_f32_i32", "mul_u24", "mul_lo_u32", "max_f32", "add_u32", "cndmask",
              "cvt_f32_ubyte0", "and_b32", "add_f32_salu")


def valu_probe(kind: int, waves: int, iters: int, ticks: int, stream: int = 0) -> None:
    """One launch of the VALU issue-rate probe (``include/smol_stream.h``):
    each of ``waves`` waves writes its elapsed 100 MHz ticks to the device
    buffer at ``ticks``."""
    _check(lib().smol_valu_probe(kind, waves, iters, ticks or None, stream or None))


def _table(v, dtype) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(v), dtype=dtype)


def _launch_stream(stream, *tensors) -> int:
    """The handle of the stream a call launches on. For a stream other than
    torch's current one (a torch stream or a raw handle), the stream first
    waits for the current stream's work (which made or filled the tensors),
    and the device tensors are recorded on it so that torch's allocator does
    not hand their memory out again before the call's work has finished."""
    import torch
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    st = torch.cuda.ExternalStream(stream) if isinstance(stream, int) else stream
    cur = torch.cuda.current_stream()
    if st.cuda_stream != cur.cuda_stream:
        st.wait_stream(cur)
        for t in tensors:
            if t is not None and getattr(t, "is_cuda", False):
                t.record_stream(st)
    return st.cuda_stream


def _out_tensor(out, n: int, params: Params, device, layout: int = LAYOUT_NCHW):
    import torch
    dtype = {OUT_F16: torch.float16, OUT_U8: torch.uint8}.get(params.out_dtype, torch.float32)
    shape = ((n, params.crop_h, params.crop_w, 3) if layout == LAYOUT_NHWC
             else (n, 3, params.crop_h, params.crop_w))
    if out is None:
        return torch.empty(shape, dtype=dtype, device=device)
    if tuple(out.shape) != shape or out.dtype != dtype or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous {dtype} tensor of shape {shape}")
    return out


def _rois(rois, n: int):
    if rois is None:
        return None
    r = _table(rois, np.int32)
    if r.shape != (n, 4):
        raise ValueError("rois must be an (n, 4) table of x, y, w, h")
    return r


def preprocess_batch(src, offsets, widths, heights, params: Params, pitches=None, out=None,
                     stream=None, rois=None, options: Options | None = None):
    """Packed HWC RGB uint8 images in the device tensor ``src`` -> NCHW (or,
    with options, NHWC) tensor. With ``rois`` ((n, 4): x, y, w, h) or
    ``options`` the call goes through ``smol_preprocess_batch_ex``.

    ``offsets`` / ``widths`` / ``heights`` / ``pitches`` / ``rois`` are host
    sequences.
    """
    if src.dtype.itemsize != 1 or not src.is_cuda or not src.is_contiguous():
        raise ValueError("src must be a contiguous uint8 device tensor")
    off = _table(offsets, np.int64)
    w = _table(widths, np.int32)
    h = _table(heights, np.int32)
    pt = None if pitches is None else _table(pitches, np.int32)
    n = len(off)
    if not (len(w) == len(h) == n and (pt is None or len(pt) == n)):
        raise ValueError("table lengths differ")
    r = _rois(rois, n)
    out = _out_tensor(out, n, params, src.device, options.layout if options else LAYOUT_NCHW)
    if r is None and options is None:
        _check(lib().smol_preprocess_batch(src.data_ptr(), src.numel(), off.ctypes.data,
                                           w.ctypes.data, h.ctypes.data,
                                           None if pt is None else pt.ctypes.data, n,
                                           ctypes.byref(params), out.data_ptr(),
                                           _launch_stream(stream, src, out)))
    else:
        _check(lib().smol_preprocess_batch_ex(
            src.data_ptr(), src.numel(), off.ctypes.data, w.ctypes.data, h.ctypes.data,
            None if pt is None else pt.ctypes.data, None if r is None else r.ctypes.data, n,
            ctypes.byref(params), None if options is None else ctypes.byref(options),
            out.data_ptr(), _launch_stream(stream, src, out)))
    return out


def yuv420_preprocess_batch(src, y_offsets, cb_offsets, cr_offsets, widths, heights,
                            params: Params, out=None, stream=None, rois=None,
                            options: Options | None = None):
    """Planar I420 uint8 frames in the device tensor ``src`` -> NCHW (or NHWC)
    RGB tensor; ``rois`` / ``options`` as for ``preprocess_batch``."""
    if src.dtype.itemsize != 1 or not src.is_cuda or not src.is_contiguous():
        raise ValueError("src must be a contiguous uint8 device tensor")
    yo = _table(y_offsets, np.int64)
    bo = _table(cb_offsets, np.int64)
    ro = _table(cr_offsets, np.int64)
    w = _table(widths, np.int32)
    h = _table(heights, np.int32)
    n = len(yo)
    if not (len(bo) == len(ro) == len(w) == len(h) == n):
        raise ValueError("table lengths differ")
    r = _rois(rois, n)
    out = _out_tensor(out, n, params, src.device, options.layout if options else LAYOUT_NCHW)
    if r is None and options is None:
        _check(lib().smol_yuv420_preprocess_batch(src.data_ptr(), src.numel(), yo.ctypes.data,
                                                  bo.ctypes.data, ro.ctypes.data, w.ctypes.data,
                                                  h.ctypes.data, n, ctypes.byref(params),
                                                  out.data_ptr(),
                                                  _launch_stream(stream, src, out)))
    else:
        _check(lib().smol_yuv420_preprocess_batch_ex(
            src.data_ptr(), src.numel(), yo.ctypes.data, bo.ctypes.data, ro.ctypes.data,
            w.ctypes.data, h.ctypes.data, None if r is None else r.ctypes.data, n,
            ctypes.byref(params), None if options is None else ctypes.byref(options),
            out.data_ptr(), _launch_stream(stream, src, out)))
    return out


def lowres_workspace_bytes(n: int, low_res: int) -> int:
    return int(lib().smol_lowres_workspace_bytes(n, low_res))


def _workspace(workspace, n: int, low_res: int, device):
    import torch
    need = lowres_workspace_bytes(n, low_res)
    if workspace is None:
        return torch.empty(max(need, 16), dtype=torch.uint8, device=device)
    if workspace.dtype != torch.uint8 or not workspace.is_contiguous() or workspace.numel() < need:
        raise ValueError(f"workspace must be a contiguous uint8 tensor of >= {need} bytes")
    return workspace


def lowres_preprocess_batch(src, offsets, widths, heights, params: Params, low_res: int,
                            pitches=None, out=None, workspace=None, stream=None):
    """Low-resolution augmentation of packed HWC RGB uint8 images: each image
    reduced to low_res x low_res uint8, then preprocessed with ``params``
    (``smol_lowres_preprocess_batch``). ``workspace`` (uint8 device tensor of
    ``lowres_workspace_bytes(n, low_res)`` bytes) is allocated if omitted."""
    if src.dtype.itemsize != 1 or not src.is_cuda or not src.is_contiguous():
        raise ValueError("src must be a contiguous uint8 device tensor")
    off = _table(offsets, np.int64)
    w = _table(widths, np.int32)
    h = _table(heights, np.int32)
    pt = None if pitches is None else _table(pitches, np.int32)
    n = len(off)
    if not (len(w) == len(h) == n and (pt is None or len(pt) == n)):
        raise ValueError("table lengths differ")
    out = _out_tensor(out, n, params, src.device)
    ws = _workspace(workspace, n, low_res, src.device)
    _check(lib().smol_lowres_preprocess_batch(
        src.data_ptr(), src.numel(), off.ctypes.data, w.ctypes.data, h.ctypes.data,
        None if pt is None else pt.ctypes.data, n, low_res, ctypes.byref(params), ws.data_ptr(),
        ws.numel(), out.data_ptr(), _launch_stream(stream, src, out, ws)))
    return out


def yuv420_lowres_preprocess_batch(src, y_offsets, cb_offsets, cr_offsets, widths, heights,
                                   params: Params, low_res: int, out=None, workspace=None,
                                   stream=None):
    """As ``lowres_preprocess_batch`` for planar I420 frames."""
    if src.dtype.itemsize != 1 or not src.is_cuda or not src.is_contiguous():
        raise ValueError("src must be a contiguous uint8 device tensor")
    yo = _table(y_offsets, np.int64)
    bo = _table(cb_offsets, np.int64)
    ro = _table(cr_offsets, np.int64)
    w = _table(widths, np.int32)
    h = _table(heights, np.int32)
    n = len(yo)
    if not (len(bo) == len(ro) == len(w) == len(h) == n):
        raise ValueError("table lengths differ")
    out = _out_tensor(out, n, params, src.device)
    ws = _workspace(workspace, n, low_res, src.device)
    _check(lib().smol_yuv420_lowres_preprocess_batch(
        src.data_ptr(), src.numel(), yo.ctypes.data, bo.ctypes.data, ro.ctypes.data,
        w.ctypes.data, h.ctypes.data, n, low_res, ctypes.byref(params), ws.data_ptr(),
        ws.numel(), out.data_ptr(), _launch_stream(stream, src, out, ws)))
    return out


def jpeg_coef_count(width: int, height: int) -> int:
    return int(lib().smol_jpeg_coef_count(width, height))


def jpeg_mcu_rect(width: int, height: int, params: Params,
                  options: Options | None = None) -> tuple[int, int, int, int]:
    """Algorithm 1's MCU-aligned rectangle (x, y, w, h) for one frame."""
    r = np.zeros(4, np.int32)
    _check(lib().smol_jpeg_mcu_rect(width, height, ctypes.byref(params),
                                    None if options is None else ctypes.byref(options),
                                    r.ctypes.data))
    return tuple(int(v) for v in r)


def _qtables(qtables, n: int) -> tuple[np.ndarray, int]:
    """(flat uint16 tables, n_qtables): one (luma, chroma) pair for every
    frame, shape (2, 64) or (128,), or one per frame, shape (n, 2, 64) or
    (n, 128)."""
    q = _table(qtables, np.uint16).reshape(-1)
    if q.size == 128:
        return q, 1
    if q.size == 128 * n:
        return q, n
    raise ValueError("qtables must hold 2 x 64 entries (luma, chroma), once or per frame")


def jpeg_window_coef_count(width: int, height: int, rect=None) -> int:
    r = None if rect is None else np.ascontiguousarray(rect, np.int32)
    return int(lib().smol_jpeg_window_coef_count(width, height,
                                                 None if r is None else r.ctypes.data))


def jpeg_decode_i420(coef, coef_offsets, qtables, widths, heights, out, y_offsets, cb_offsets,
                     cr_offsets, rects=None, stream=None, coef_layout: int = JPEG_COEF_FRAME):
    """Decode the blocks of each frame meeting its rectangle (``rects`` (n, 4)
    or None for whole frames) from the int16 device tensor ``coef`` into the
    uint8 device tensor ``out`` at the given plane offsets."""
    if coef.dtype.itemsize != 2 or not coef.is_cuda or not coef.is_contiguous():
        raise ValueError("coef must be a contiguous int16 device tensor")
    if out.dtype.itemsize != 1 or not out.is_cuda or not out.is_contiguous():
        raise ValueError("out must be a contiguous uint8 device tensor")
    co = _table(coef_offsets, np.int64)
    w, h = _table(widths, np.int32), _table(heights, np.int32)
    yo, bo, ro = (_table(v, np.int64) for v in (y_offsets, cb_offsets, cr_offsets))
    n = len(co)
    r = None if rects is None else _rois(rects, n)
    q, nq = _qtables(qtables, n)
    _check(lib().smol_jpeg_decode_i420(
        coef.data_ptr(), coef.numel(), co.ctypes.data, q.ctypes.data, nq, w.ctypes.data,
        h.ctypes.data, None if r is None else r.ctypes.data, n, coef_layout, out.data_ptr(),
        out.numel(), yo.ctypes.data, bo.ctypes.data, ro.ctypes.data,
        _launch_stream(stream, coef, out)))


def jpeg_workspace_bytes(widths, heights) -> int:
    w, h = _table(widths, np.int32), _table(heights, np.int32)
    return int(lib().smol_jpeg_workspace_bytes(len(w), w.ctypes.data, h.ctypes.data))


def jpeg_roi_preprocess_batch(coef, coef_offsets, qtables, widths, heights, params: Params,
                              options: Options | None = None, workspace=None, out=None,
                              stream=None, coef_layout: int = JPEG_COEF_FRAME):
    """Algorithm 1 end to end: only each frame's MCU rectangle decoded (into
    ``workspace``, allocated if omitted), then the I420 preprocessing."""
    import torch
    if coef.dtype.itemsize != 2 or not coef.is_cuda or not coef.is_contiguous():
        raise ValueError("coef must be a contiguous int16 device tensor")
    co = _table(coef_offsets, np.int64)
    w, h = _table(widths, np.int32), _table(heights, np.int32)
    n = len(co)
    q, nq = _qtables(qtables, n)
    need = jpeg_workspace_bytes(w, h)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=coef.device)
    out = _out_tensor(out, n, params, coef.device, options.layout if options else LAYOUT_NCHW)
    _check(lib().smol_jpeg_roi_preprocess_batch(
        coef.data_ptr(), coef.numel(), co.ctypes.data, q.ctypes.data, nq, w.ctypes.data,
        h.ctypes.data, n, coef_layout, ctypes.byref(params),
        None if options is None else ctypes.byref(options), workspace.data_ptr(),
        workspace.numel(), out.data_ptr(), _launch_stream(stream, coef, out, workspace)))
    return out


def jpeg_read_info(data: bytes) -> JpegInfo:
    """The headers of one JPEG stream: size, restart interval, tables."""
    buf = np.frombuffer(data, np.uint8)
    info = JpegInfo()
    _check(lib().smol_jpeg_read_info(buf.ctypes.data, buf.size, ctypes.byref(info)))
    return info


class JpegBatch:
    """Entropy-decoded JPEG streams: ``coef`` (int16, host; a pinned torch
    tensor when asked for), ``coef_offsets``, ``qtables`` (n, 2, 64),
    ``widths``, ``heights`` and the ``rects`` they were decoded for."""

    def __init__(self, coef, coef_offsets, qtables, widths, heights, rects, coef_layout):
        self.coef, self.coef_offsets, self.qtables = coef, coef_offsets, qtables
        self.widths, self.heights, self.rects = widths, heights, rects
        self.coef_layout = coef_layout

    @property
    def n(self) -> int:
        return len(self.widths)


def jpeg_entropy_decode_batch(streams, rects=None, threads: int = 0, pinned: bool = False,
                              coef_layout: int = JPEG_COEF_FRAME) -> JpegBatch:
    """Entropy-decode JPEG streams (a list of bytes) on host threads into the
    coefficient layout of the GPU calls. ``rects`` (n, 4) limits each stream
    to the MCUs its rectangle needs (other blocks stay zero); with
    ``JPEG_COEF_WINDOW`` only those MCUs are stored."""
    n = len(streams)
    sizes = np.asarray([len(b) for b in streams], np.int64)
    offs = np.concatenate([[0], np.cumsum(sizes)[:-1]]).astype(np.int64) if n else sizes
    data = np.frombuffer(b"".join(streams), np.uint8) if n else np.zeros(1, np.uint8)
    infos = [jpeg_read_info(b) for b in streams]
    w = np.asarray([i.width for i in infos], np.int32)
    h = np.asarray([i.height for i in infos], np.int32)
    r = None if rects is None else _rois(rects, n)
    if coef_layout == JPEG_COEF_WINDOW:
        if r is None:
            raise ValueError("the window layout needs rects")
        counts = np.asarray([jpeg_window_coef_count(int(a), int(b), r[i])
                             for i, (a, b) in enumerate(zip(w, h))], np.int64)
    else:
        counts = np.asarray([jpeg_coef_count(int(a), int(b)) for a, b in zip(w, h)], np.int64)
    co = np.concatenate([[0], np.cumsum(counts)[:-1]]).astype(np.int64) if n else counts
    total = max(int(counts.sum()), 8)
    if pinned:
        import torch
        coef = torch.zeros(total, dtype=torch.int16, pin_memory=True)
        ptr = coef.data_ptr()
    else:
        coef = np.zeros(total, np.int16)
        ptr = coef.ctypes.data
    q = np.zeros((max(n, 1), 2, 64), np.uint16)
    _check(lib().smol_jpeg_entropy_decode_batch(
        data.ctypes.data, data.size, offs.ctypes.data, sizes.ctypes.data, n,
        None if r is None else r.ctypes.data, ptr, total, co.ctypes.data, coef_layout,
        q.ctypes.data, threads))
    return JpegBatch(coef, co, q[:n], w, h, r, coef_layout)


def jpeg_files_preprocess(streams, params: Params, options: Options | None = None,
                          threads: int = 0, out=None, stream=None):
    """Algorithm 1 from JPEG files: per stream the MCU rectangle of the
    preprocessing, entropy decoding of only the MCUs it needs (host threads,
    pinned memory, only the rectangle's MCU window stored), the copy to the
    device, then the partial block decoding and the fused preprocessing on
    the GPU."""
    infos = [jpeg_read_info(b) for b in streams]
    rects = [jpeg_mcu_rect(i.width, i.height, params, options) for i in infos]
    b = jpeg_entropy_decode_batch(streams, rects, threads, pinned=True,
                                  coef_layout=JPEG_COEF_WINDOW)
    import torch
    st = (torch.cuda.current_stream() if stream is None else
          torch.cuda.ExternalStream(stream) if isinstance(stream, int) else stream)
    cur = torch.cuda.current_stream()
    if st.cuda_stream != cur.cuda_stream:
        # as for every call on another stream: wait for the current stream's
        # work (which may still be making or using `out`), and keep `out` from
        # being handed out again before the side stream is done with it
        st.wait_stream(cur)
        if out is not None and getattr(out, "is_cuda", False):
            out.record_stream(st)
    with torch.cuda.stream(st):
        # the copy, the workspace and the output all belong to `st`
        dev = b.coef.to("cuda", non_blocking=True)
        return jpeg_roi_preprocess_batch(dev, b.coef_offsets, b.qtables, b.widths, b.heights,
                                         params, options, None, out, None, JPEG_COEF_WINDOW)


def torch_int16():
    import torch
    return torch.int16


def _workload_options(wl) -> Options | None:
    if not wl.variant:
        return None
    return make_options(wl.resize_mode, wl.layout, wl.siting)


def run_workload(wl, src_dev, out=None, stream=None):
    """Run a ``synthetic.Workload`` whose ``src`` already sits on the device."""
    p = make_params(wl.resize_short, wl.crop_h, wl.crop_w, wl.mean, wl.std, wl.out_dtype)
    if wl.kind == "jpeg":
        return jpeg_roi_preprocess_batch(src_dev.view(torch_int16()), wl.coef_offsets, wl.qtables, wl.widths,
                                         wl.heights, p, _workload_options(wl), None, out, stream)
    if wl.low_res:
        if wl.variant:
            raise ValueError("the low-resolution augmentation takes no ROI or options")
        if wl.kind == "rgb":
            return lowres_preprocess_batch(src_dev, wl.offsets, wl.widths, wl.heights, p,
                                           wl.low_res, wl.pitches, out, None, stream)
        return yuv420_lowres_preprocess_batch(src_dev, wl.y_offsets, wl.cb_offsets,
                                              wl.cr_offsets, wl.widths, wl.heights, p,
                                              wl.low_res, out, None, stream)
    o = _workload_options(wl)
    if wl.kind == "rgb":
        return preprocess_batch(src_dev, wl.offsets, wl.widths, wl.heights, p, wl.pitches, out,
                                stream, wl.rois, o)
    return yuv420_preprocess_batch(src_dev, wl.y_offsets, wl.cb_offsets, wl.cr_offsets,
                                   wl.widths, wl.heights, p, out, stream, wl.rois, o)


class PreparedCall:
    """A batch call with every host-side argument marshalled once, for tight
    launch loops: ``call(src_ptr, src_bytes, out_ptr, stream_handle)``."""

    def __init__(self, wl):
        self.params = make_params(wl.resize_short, wl.crop_h, wl.crop_w, wl.mean, wl.std,
                                  wl.out_dtype)
        self.kind = wl.kind
        self.n = wl.n
        self._keep = []
        self.options = _workload_options(wl)
        ex = self.options is not None
        self._low = None
        self._jpeg = None
        if wl.kind == "jpeg":
            import torch
            q, nq = _qtables(wl.qtables, wl.n)
            tabs = [_table(wl.coef_offsets, np.int64), q, _table(wl.widths, np.int32),
                    _table(wl.heights, np.int32)]
            ws = torch.empty(max(jpeg_workspace_bytes(wl.widths, wl.heights), 16),
                             dtype=torch.uint8, device="cuda")
            self._keep = tabs
            ptrs = [t.ctypes.data for t in tabs]
            self._jpeg = (ptrs[:2] + [nq] + ptrs[2:], ws, ws.data_ptr(), ws.numel())
            self._fn = lib().smol_jpeg_roi_preprocess_batch
            self._pref = ctypes.byref(self.params)
            self._tail = [ctypes.byref(self.options)] if ex else [None]
            return
        if wl.low_res:
            if ex:
                raise ValueError("the low-resolution augmentation takes no ROI or options")
            import torch
            ws = torch.empty(max(lowres_workspace_bytes(wl.n, wl.low_res), 16),
                             dtype=torch.uint8, device="cuda")
            self._low = (ctypes.c_int32(wl.low_res), ws, ctypes.c_void_p(ws.data_ptr()),
                         ctypes.c_int64(ws.numel()))
        r = None if wl.rois is None else _rois(wl.rois, wl.n)
        if wl.kind == "rgb":
            tabs = [_table(wl.offsets, np.int64), _table(wl.widths, np.int32),
                    _table(wl.heights, np.int32)]
            pt = None if wl.pitches is None else _table(wl.pitches, np.int32)
            self._keep = tabs + [pt, r]
            self._args = [t.ctypes.data for t in tabs] + [None if pt is None else pt.ctypes.data]
            self._fn = (lib().smol_lowres_preprocess_batch if self._low else
                        lib().smol_preprocess_batch_ex if ex else lib().smol_preprocess_batch)
        else:
            tabs = [_table(wl.y_offsets, np.int64), _table(wl.cb_offsets, np.int64),
                    _table(wl.cr_offsets, np.int64), _table(wl.widths, np.int32),
                    _table(wl.heights, np.int32)]
            self._keep = tabs + [r]
            self._args = [t.ctypes.data for t in tabs]
            self._fn = (lib().smol_yuv420_lowres_preprocess_batch if self._low else
                        lib().smol_yuv420_preprocess_batch_ex if ex
                        else lib().smol_yuv420_preprocess_batch)
        if ex:
            self._args.append(None if r is None else r.ctypes.data)
        self._pref = ctypes.byref(self.params)
        self._tail = [ctypes.byref(self.options)] if ex else []

    def __call__(self, src_ptr: int, src_bytes: int, out_ptr: int, stream_handle) -> None:
        if self._jpeg:
            args, _, ws, ws_bytes = self._jpeg
            _check(self._fn(src_ptr, src_bytes // 2, *args, self.n, JPEG_COEF_FRAME, self._pref,
                            *self._tail, ws, ws_bytes, out_ptr, stream_handle))
            return
        if self._low:
            low, _, ws, ws_bytes = self._low
            _check(self._fn(src_ptr, src_bytes, *self._args, self.n, low, self._pref, ws,
                            ws_bytes, out_ptr, stream_handle))
            return
        _check(self._fn(src_ptr, src_bytes, *self._args, self.n, self._pref, *self._tail,
                        out_ptr, stream_handle))


_consumer_state = threading.local()


class Pipeline:
    """Pipelined ingest (``include/smol_pipeline.h``): ``slots`` reused buffer
    sets (pinned host input, device input, device output), ``streams`` compute
    streams and ``copy_streams`` copy streams. Producer threads ``acquire`` a
    slot, fill ``host_view(slot)`` with a batch and ``submit`` it; the copy,
    the preprocessing and the optional consumer run in stream order while
    other slots are filled.

    A consumer is a Python callable ``f(output, n, stream)`` (raw device
    pointer of the slot's output, image count, raw stream handle) or a
    ``CONSUMER`` callback ``f(user, output, n, stream)``. It runs on the
    submitting thread during ``submit``, which still holds the slot. For a
    Python callable, torch's current stream is the batch's stream while it
    runs (when torch has a device), so torch work it starts is ordered behind
    the preprocessing and covered by the slot's completion. From inside any
    consumer, this pipeline's ``acquire``, ``submit``, ``drain`` and
    ``close`` raise instead of waiting: the consumer's thread holds a slot,
    and waiting there for a slot or for completions can wait forever (every
    slot held by producers inside their consumers)."""

    def __init__(self, slots: int, streams: int, input_bytes: int, output_bytes: int,
                 copy_streams: int = 1, workspace_bytes: int = 0, library=None):
        self._lib = lib() if library is None else library
        cfg = PipelineConfig()
        cfg.slots, cfg.streams, cfg.copy_streams = slots, streams, copy_streams
        cfg.input_bytes, cfg.output_bytes = input_bytes, output_bytes
        cfg.workspace_bytes = workspace_bytes
        h = ctypes.c_void_p()
        self._check(self._lib.smol_pipeline_create(ctypes.byref(cfg), ctypes.byref(h)))
        self._h = h
        self.input_bytes = input_bytes
        self.output_bytes = output_bytes
        self._host = {}

    def _check(self, status: int) -> None:
        if status != OK:
            detail = (self._lib.smol_last_error().decode() or
                      self._lib.smol_status_string(status).decode())
            raise SmolError(status, detail)

    def _not_in_consumer(self, what: str) -> None:
        if getattr(_consumer_state, "pipeline", None) is self:
            raise RuntimeError(f"{what} called from inside a consumer of the same pipeline: the "
                               "consumer's thread holds a slot, and waiting there for slots or "
                               "completions can deadlock")

    def _consumer_fn(self, consumer):
        """The CONSUMER the library calls: the caller's consumer inside the
        re-entrancy guard (and, for a Python callable, on the batch's torch
        stream); an exception becomes a failed consumer (nonzero)."""
        if consumer is None:
            return CONSUMER()
        raw = isinstance(consumer, CONSUMER)

        def call(user, output, n, stream):
            prev = getattr(_consumer_state, "pipeline", None)
            _consumer_state.pipeline = self
            try:
                if raw:
                    return int(consumer(user, output, n, stream))
                torch = sys.modules.get("torch")
                if torch is not None and torch.cuda.is_available():
                    with torch.cuda.stream(torch.cuda.ExternalStream(stream)):
                        consumer(output, n, stream)
                else:
                    consumer(output, n, stream)
                return 0
            except Exception as e:  # noqa: BLE001 -- reported as a failed consumer
                _consumer_state.error = e
                return 1
            finally:
                _consumer_state.pipeline = prev

        return CONSUMER(call)

    def _submitted(self, status: int) -> None:
        """Check a submission; a consumer's exception becomes the cause."""
        err = getattr(_consumer_state, "error", None)
        _consumer_state.error = None
        try:
            self._check(status)
        except SmolError as e:
            if err is not None:
                raise e from err
            raise

    def acquire(self) -> tuple[int, int, int]:
        """(slot, host pointer, device output pointer)."""
        self._not_in_consumer("acquire")
        slot, host, out = ctypes.c_int32(), ctypes.c_void_p(), ctypes.c_void_p()
        self._check(self._lib.smol_pipeline_acquire(self._h, ctypes.byref(slot), ctypes.byref(host),
                                           ctypes.byref(out)))
        self._host[slot.value] = host.value
        return slot.value, host.value, out.value

    def host_view(self, slot: int) -> np.ndarray:
        """The acquired slot's pinned input buffer as a uint8 array."""
        buf = (ctypes.c_uint8 * self.input_bytes).from_address(self._host[slot])
        return np.ctypeslib.as_array(buf)

    def release(self, slot: int) -> None:
        self._check(self._lib.smol_pipeline_release(self._h, slot))

    def submit(self, slot: int, nbytes: int, offsets, widths, heights, params: Params,
               pitches=None, rois=None, options: Options | None = None, consumer=None,
               user: int | None = None) -> None:
        off = _table(offsets, np.int64)
        w = _table(widths, np.int32)
        h = _table(heights, np.int32)
        pt = None if pitches is None else _table(pitches, np.int32)
        n = len(off)
        r = _rois(rois, n)
        self._not_in_consumer("submit")
        _consumer_state.error = None
        self._submitted(self._lib.smol_pipeline_submit(
            self._h, slot, nbytes, off.ctypes.data, w.ctypes.data, h.ctypes.data,
            None if pt is None else pt.ctypes.data, None if r is None else r.ctypes.data, n,
            ctypes.byref(params), None if options is None else ctypes.byref(options),
            self._consumer_fn(consumer), user))

    def submit_yuv420(self, slot: int, nbytes: int, y_offsets, cb_offsets, cr_offsets, widths,
                      heights, params: Params, rois=None, options: Options | None = None,
                      consumer=None, user: int | None = None) -> None:
        yo = _table(y_offsets, np.int64)
        bo = _table(cb_offsets, np.int64)
        ro = _table(cr_offsets, np.int64)
        w = _table(widths, np.int32)
        h = _table(heights, np.int32)
        n = len(yo)
        r = _rois(rois, n)
        self._not_in_consumer("submit")
        _consumer_state.error = None
        self._submitted(self._lib.smol_pipeline_submit_yuv420(
            self._h, slot, nbytes, yo.ctypes.data, bo.ctypes.data, ro.ctypes.data, w.ctypes.data,
            h.ctypes.data, None if r is None else r.ctypes.data, n, ctypes.byref(params),
            None if options is None else ctypes.byref(options),
            self._consumer_fn(consumer), user))

    def submit_jpeg(self, slot: int, nbytes: int, coef_offsets, qtables, widths, heights,
                    params: Params, coef_layout: int = JPEG_COEF_WINDOW,
                    options: Options | None = None, consumer=None,
                    user: int | None = None) -> None:
        """Submit entropy-decoded JPEG coefficients in the slot's host buffer
        (``decode_jpeg_into``) for partial block decoding and preprocessing."""
        co = _table(coef_offsets, np.int64)
        w = _table(widths, np.int32)
        h = _table(heights, np.int32)
        n = len(co)
        q, nq = _qtables(qtables, n)
        self._not_in_consumer("submit")
        _consumer_state.error = None
        self._submitted(self._lib.smol_pipeline_submit_jpeg(
            self._h, slot, nbytes, co.ctypes.data, q.ctypes.data, nq, w.ctypes.data,
            h.ctypes.data, n, coef_layout, ctypes.byref(params),
            None if options is None else ctypes.byref(options),
            self._consumer_fn(consumer), user))

    def decode_jpeg_into(self, slot: int, streams, params: Params,
                         options: Options | None = None, threads: int = 0):
        """Entropy-decode JPEG streams into the acquired slot's pinned buffer,
        only the MCU windows of Algorithm 1's rectangles: (bytes,
        coef_offsets, qtables, widths, heights) for ``submit_jpeg``."""
        n = len(streams)
        infos = [jpeg_read_info(b) for b in streams]
        w = np.asarray([i.width for i in infos], np.int32)
        h = np.asarray([i.height for i in infos], np.int32)
        rects = _rois([jpeg_mcu_rect(i.width, i.height, params, options) for i in infos], n)
        counts = np.asarray([jpeg_window_coef_count(int(w[i]), int(h[i]), rects[i])
                             for i in range(n)], np.int64)
        co = np.concatenate([[0], np.cumsum(counts)[:-1]]).astype(np.int64)
        total = int(counts.sum())
        if 2 * total > self.input_bytes:
            raise ValueError(f"{2 * total} coefficient bytes exceed the slot's {self.input_bytes}")
        sizes = np.asarray([len(b) for b in streams], np.int64)
        offs = np.concatenate([[0], np.cumsum(sizes)[:-1]]).astype(np.int64)
        data = np.frombuffer(b"".join(streams), np.uint8)
        q = np.zeros((n, 2, 64), np.uint16)
        self._check(self._lib.smol_jpeg_entropy_decode_batch(
            data.ctypes.data, data.size, offs.ctypes.data, sizes.ctypes.data, n,
            rects.ctypes.data, self._host[slot], total, co.ctypes.data, JPEG_COEF_WINDOW,
            q.ctypes.data, threads))
        return 2 * total, co, q, w, h

    def drain(self) -> None:
        self._not_in_consumer("drain")
        self._check(self._lib.smol_pipeline_drain(self._h))

    def stats(self) -> dict:
        st = PipelineStats()
        self._check(self._lib.smol_pipeline_get_stats(self._h, ctypes.byref(st)))
        return st.as_dict()

    def close(self) -> None:
        if self._h is not None and self._h.value:
            self._not_in_consumer("close")
            h, self._h = self._h, None
            self._check(self._lib.smol_pipeline_destroy(h))

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
