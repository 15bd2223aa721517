"""C-ABI checks that need no GPU: symbols, argument validation, geometry.

Validation runs before the library makes any HIP call, so every call here is
rejected on the host; no call reaches a device.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2007_13005_amd import smol, synthetic

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
HEADERS = sorted(os.path.join(INCLUDE, f) for f in os.listdir(INCLUDE) if f.endswith(".h"))
MEAN, STD = synthetic.IMAGENET_MEAN_255, synthetic.IMAGENET_STD_255


def _declared_functions() -> list[str]:
    text = "\n".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(smol_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = smol.lib()
    declared = _declared_functions()
    assert declared, "no declarations found"
    assert set(declared) == set(smol.SIGNATURES), "binding and header disagree"
    for name in declared:
        assert hasattr(lib, name), name


def test_status_strings_and_version():
    lib = smol.lib()
    for code in (smol.OK, smol.ERR_INVALID_ARG, smol.ERR_UNSUPPORTED, smol.ERR_HIP):
        assert lib.smol_status_string(code)
    assert lib.smol_status_string(12345) == b"unknown status"
    assert smol.version() >= 100


def _params(**kw):
    base = dict(resize_short=256, crop_h=224, crop_w=224, mean=MEAN, std=STD,
                out_dtype=smol.OUT_F16)
    base.update(kw)
    return smol.make_params(base["resize_short"], base["crop_h"], base["crop_w"], base["mean"],
                            base["std"], base["out_dtype"])


FAKE_SRC = 0x10000   # never dereferenced: every call below fails validation
FAKE_OUT = 0x20000


def _rgb_call(n=1, src=FAKE_SRC, src_bytes=10**9, offsets=(0,), widths=(320,), heights=(240,),
              pitches=None, params=None, out=FAKE_OUT):
    p = params or _params()
    off = np.asarray(offsets, np.int64)
    w = np.asarray(widths, np.int32)
    h = np.asarray(heights, np.int32)
    pt = None if pitches is None else np.asarray(pitches, np.int32)
    rc = smol.lib().smol_preprocess_batch(src, src_bytes, off.ctypes.data, w.ctypes.data,
                                          h.ctypes.data, None if pt is None else pt.ctypes.data,
                                          n, ctypes.byref(p), out, None)
    return rc, smol.lib().smol_last_error().decode()


@pytest.mark.parametrize("kw,needle", [
    (dict(n=-1), "n = -1"),
    (dict(src=0), "NULL"),
    (dict(out=0), "NULL"),
    (dict(out=FAKE_OUT + 4), "aligned"),
    (dict(widths=(0,)), "size"),
    (dict(heights=(70000,)), "size"),
    (dict(src_bytes=320 * 240 * 3 - 1), "outside src"),
    (dict(offsets=(-1,)), "outside src"),
    (dict(offsets=(5,), src_bytes=320 * 240 * 3 + 4), "outside src"),
    (dict(pitches=(959,)), "pitch"),
])
def test_rgb_validation_rejects(kw, needle):
    rc, msg = _rgb_call(**kw)
    assert rc == smol.ERR_INVALID_ARG, (rc, msg)
    assert needle in msg


@pytest.mark.parametrize("kw,needle", [
    (dict(out_dtype=7), "out_dtype"),
    (dict(resize_short=0), "resize_short"),
    (dict(crop_h=0), "crop"),
    (dict(crop_w=342), "larger than resized"),
    (dict(std=(1.0, 0.0, 1.0)), "std"),
    (dict(mean=(np.inf, 0, 0)), "mean"),
    (dict(std=(1e-45, 1, 1)), "overflow"),
])
def test_param_validation_rejects(kw, needle):
    rc, msg = _rgb_call(params=_params(**kw))
    assert rc == smol.ERR_INVALID_ARG, (rc, msg)
    assert needle in msg


def test_unsupported_resized_size():
    # 65535 x 1 with S = 256: the long side would become 256 * 65535
    rc, msg = _rgb_call(widths=(65535,), heights=(1,), params=_params(crop_h=1, crop_w=1))
    assert rc == smol.ERR_UNSUPPORTED, msg


def test_ragged_table_checked_entry_by_entry():
    # second image runs past the end of src
    rc, msg = _rgb_call(n=2, offsets=(0, 1000), widths=(300, 300), heights=(300, 300),
                        src_bytes=300 * 300 * 3 + 999)
    assert rc == smol.ERR_INVALID_ARG and "image 1" in msg


def test_empty_batch_is_a_no_op():
    rc, _ = _rgb_call(n=0, src=0, out=0)
    assert rc == smol.OK


def test_yuv_validation_rejects():
    p = _params()
    z = np.zeros(1, np.int64)
    w = np.asarray([64], np.int32)
    h = np.asarray([64], np.int32)
    cb = np.asarray([64 * 64], np.int64)
    cr = np.asarray([64 * 64 + 32 * 32], np.int64)
    lib = smol.lib()
    # src too small for the Cr plane
    rc = lib.smol_yuv420_preprocess_batch(FAKE_SRC, 64 * 64 + 2 * 32 * 32 - 1, z.ctypes.data,
                                          cb.ctypes.data, cr.ctypes.data, w.ctypes.data,
                                          h.ctypes.data, 1, ctypes.byref(_params(resize_short=64,
                                                                                 crop_h=64,
                                                                                 crop_w=64)),
                                          FAKE_OUT, None)
    assert rc == smol.ERR_INVALID_ARG and "plane 2" in lib.smol_last_error().decode()
    rc = lib.smol_yuv420_preprocess_batch(FAKE_SRC, 10**6, None, cb.ctypes.data, cr.ctypes.data,
                                          w.ctypes.data, h.ctypes.data, 1, ctypes.byref(p),
                                          FAKE_OUT, None)
    assert rc == smol.ERR_INVALID_ARG


def test_tuning_validation():
    with pytest.raises(smol.SmolError):
        smol.set_tuning(path=5)
    with pytest.raises(smol.SmolError):
        smol.set_tuning(band_rows=65)
    with pytest.raises(smol.SmolError):
        smol.set_tuning(lds_budget=100)
    with pytest.raises(smol.SmolError):
        smol.set_tuning(workgroups_per_cu=17)
    with pytest.raises(smol.SmolError):
        smol.set_tuning(exact=2)
    with pytest.raises(smol.SmolError):
        smol.set_tuning(row_order=3)
    with pytest.raises(smol.SmolError):
        smol.set_tuning(upload=4)
    smol.set_tuning(path=1, band_rows=8, lds_budget=32768)
    smol.set_tuning(upload=3)
    smol.set_tuning(upload=2)
    smol.set_tuning(path=4, exact=1)
    smol.reset_tuning()


# ---------------------------------------------------------------------------
# geometry: the library's per-image geometry against the oracle, bit for bit
# ---------------------------------------------------------------------------


def test_geometry_matches_oracle():
    rng = np.random.default_rng(21)
    cases = [(320, 240, 256, 224, 224), (1920, 1080, 224, 224, 224), (128, 128, 224, 224, 224),
             (1280, 720, 256, 224, 224), (1, 1, 1, 1, 1), (2000, 260, 256, 224, 224)]
    for _ in range(500):
        W, H = (int(v) for v in rng.integers(1, 4000, size=2))
        S = int(rng.integers(1, 700))
        Ch, Cw = (int(v) for v in rng.integers(1, S + 1, size=2))
        cases.append((W, H, S, Ch, Cw))
    for W, H, S, Ch, Cw in cases:
        g = smol.image_geometry(W, H, _params(resize_short=S, crop_h=Ch, crop_w=Cw))
        Wr, Hr = oracle.resized_dims(W, H, S)
        left, top = oracle.crop_offsets(Wr, Hr, Ch, Cw)
        assert (g["resized_w"], g["resized_h"], g["crop_left"], g["crop_top"]) == (Wr, Hr, left,
                                                                                   top)
        # footprint: first/last source column and distinct rows, from the oracle's taps
        assert g["src_x_first"] == oracle.axis_tap(left, W, Wr)[0]
        assert g["src_x_last"] == oracle.axis_tap(left + Cw - 1, W, Wr)[1]
        if Ch <= 64:
            rows = set()
            for r in range(Ch):
                y0, y1, _ = oracle.axis_tap(top + r, H, Hr)
                rows.update((y0, y1))
            assert g["src_rows"] == len(rows)


@pytest.mark.parametrize("cfg,rows,span", [
    # per-config footprints worked out from the half-pixel map (source rows
    # touched by the 224 output rows; source columns spanned by the crop)
    ("c1", 212, 211), ("c3", 128, 128), ("c4", 448, 1078)])
def test_config_footprints(cfg, rows, span):
    W, H, S = {"c1": (320, 240, 256), "c3": (128, 128, 224), "c4": (1920, 1080, 224)}[cfg]
    g = smol.image_geometry(W, H, _params(resize_short=S))
    assert g["src_rows"] == rows
    assert g["src_x_last"] - g["src_x_first"] + 1 == span


def test_yuv_footprint_c5():
    g = smol.image_geometry(1280, 720, _params(resize_short=256), yuv420=True)
    assert (g["resized_w"], g["resized_h"], g["crop_left"], g["crop_top"]) == (455, 256, 115, 16)
    assert g["src_rows"] == 448 and g["src_x_last"] - g["src_x_first"] + 1 == 629
    assert g["chroma_rows"] == 316 and g["chroma_x_last"] - g["chroma_x_first"] + 1 == 316


# ---------------------------------------------------------------------------
# variants: ROI, options (validation on the host, geometry against the oracle)
# ---------------------------------------------------------------------------


def _rgb_ex_call(rois=None, opts=None, widths=(320,), heights=(240,), params=None):
    p = params or _params()
    off = np.zeros(1, np.int64)
    w = np.asarray(widths, np.int32)
    h = np.asarray(heights, np.int32)
    r = None if rois is None else np.asarray(rois, np.int32).reshape(-1, 4)
    rc = smol.lib().smol_preprocess_batch_ex(
        FAKE_SRC, 10**9, off.ctypes.data, w.ctypes.data, h.ctypes.data, None,
        None if r is None else r.ctypes.data, 1, ctypes.byref(p),
        None if opts is None else ctypes.byref(opts), FAKE_OUT, None)
    return rc, smol.lib().smol_last_error().decode()


def _opts(**kw):
    o = smol.make_options()
    for k, v in kw.items():
        if k == "reserved":
            o.reserved[0] = v
        else:
            setattr(o, k, v)
    return o


@pytest.mark.parametrize("kw,needle", [
    (dict(opts=_opts(resize_mode=2)), "resize_mode"),
    (dict(opts=_opts(layout=5)), "layout"),
    (dict(opts=_opts(chroma_siting=-1)), "chroma_siting"),
    (dict(opts=_opts(reserved=1)), "reserved"),
    (dict(rois=(-1, 0, 10, 10)), "ROI"),
    (dict(rois=(0, 0, 0, 10)), "ROI"),
    (dict(rois=(300, 0, 21, 10)), "ROI"),
    (dict(rois=(0, 200, 10, 41)), "ROI"),
    # a 100 x 100 ROI cannot hold a 224 crop after a short-side resize to 160
    (dict(rois=(0, 0, 100, 100), params=_params(resize_short=160)), "larger than resized"),
])
def test_variant_validation_rejects(kw, needle):
    rc, msg = _rgb_ex_call(**kw)
    assert rc == smol.ERR_INVALID_ARG, (rc, msg)
    assert needle in msg


def test_nhwc_refuses_forced_lds_and_gather_paths():
    for path in (smol.PATH_LDS, smol.PATH_GATHER):
        smol.set_tuning(path=path)
        try:
            rc, msg = _rgb_ex_call(opts=_opts(layout=smol.LAYOUT_NHWC))
        finally:
            smol.reset_tuning()
        assert rc == smol.ERR_UNSUPPORTED and "NHWC" in msg


def test_geometry_ex_matches_oracle():
    """ROI geometry: resized size and crop offsets of the ROI (oracle), columns
    in image coordinates; direct resize: the output size, no crop."""
    rng = np.random.default_rng(22)
    for _ in range(300):
        W, H = (int(v) for v in rng.integers(8, 3000, size=2))
        rw, rh = int(rng.integers(1, W + 1)), int(rng.integers(1, H + 1))
        rx, ry = int(rng.integers(0, W - rw + 1)), int(rng.integers(0, H - rh + 1))
        Ch, Cw = (int(v) for v in rng.integers(1, 300, size=2))
        mode = int(rng.integers(0, 2))
        S = max(Ch, Cw) + int(rng.integers(0, 50))
        p = _params(resize_short=S, crop_h=Ch, crop_w=Cw)
        Wr, Hr, left, top = oracle.output_geometry(rw, rh, S, Ch, Cw, mode)
        if Cw > Wr or Ch > Hr:
            continue
        g = smol.image_geometry_ex(W, H, p, roi=(rx, ry, rw, rh),
                                   options=smol.make_options(resize_mode=mode))
        assert (g["resized_w"], g["resized_h"], g["crop_left"], g["crop_top"]) == (Wr, Hr, left,
                                                                                   top)
        assert g["src_x_first"] == rx + oracle.axis_tap(left, rw, Wr)[0]
        assert g["src_x_last"] == rx + oracle.axis_tap(left + Cw - 1, rw, Wr)[1]


def test_left_siting_chroma_footprint():
    """Co-sited chroma: luma columns x0 .. x1 read chroma columns x0 // 2 ..
    min(x1 // 2 + 1, Wc - 1) (the centred map reads one column further left)."""
    p = _params(resize_short=112, crop_h=112, crop_w=112)
    roi = (101, 37, 300, 300)
    gc = smol.image_geometry_ex(640, 480, p, yuv420=True, roi=roi,
                                options=smol.make_options(resize_mode=1))
    gl = smol.image_geometry_ex(640, 480, p, yuv420=True, roi=roi,
                                options=smol.make_options(resize_mode=1,
                                                          chroma_siting=smol.CHROMA_LEFT))
    x0, x1 = gl["src_x_first"], gl["src_x_last"]
    assert (gl["chroma_x_first"], gl["chroma_x_last"]) == (x0 // 2, min(x1 // 2 + 1, 319))
    assert gc["chroma_x_first"] == (2 * x0 - 1) // 4


def test_u8_output_refuses_forced_tiled_paths():
    for path in (smol.PATH_LDS, smol.PATH_GATHER):
        smol.set_tuning(path=path)
        try:
            rc, msg = _rgb_call(params=_params(out_dtype=smol.OUT_U8))
        finally:
            smol.reset_tuning()
        assert rc == smol.ERR_UNSUPPORTED and "uint8" in msg, (path, rc, msg)


def test_lowres_workspace_bytes():
    f = smol.lib().smol_lowres_workspace_bytes
    assert f(256, 161) == 256 * 3 * 161 * 161 + 16
    assert f(1, 3) == 32 + 16
    assert f(0, 161) == 0 and f(-1, 4) == 0 and f(4, 0) == 0


def _lowres_call(n=1, low_res=64, params=None, ws=FAKE_OUT + 4096, ws_bytes=None):
    p = params or _params()
    off = np.zeros(1, np.int64)
    w = np.asarray([320], np.int32)
    h = np.asarray([240], np.int32)
    need = smol.lib().smol_lowres_workspace_bytes(n, low_res)
    rc = smol.lib().smol_lowres_preprocess_batch(
        FAKE_SRC, 10**9, off.ctypes.data, w.ctypes.data, h.ctypes.data, None, n, low_res,
        ctypes.byref(p), ws, need if ws_bytes is None else ws_bytes, FAKE_OUT, None)
    return rc, smol.lib().smol_last_error().decode()


@pytest.mark.parametrize("kw,needle", [
    (dict(low_res=0), "low_res"),
    (dict(low_res=70000), "low_res"),
    (dict(ws_bytes=64 * 64 * 3 + 15), "workspace"),
    (dict(ws=0), "workspace"),
    (dict(ws=FAKE_OUT + 8), "aligned"),
    (dict(params=_params(out_dtype=smol.OUT_U8)), "normalised"),
    # the 64 x 64 image resized to 256 cannot hold a 300 x 300 crop
    (dict(params=_params(crop_h=300, crop_w=300)), "larger than resized"),
    (dict(n=-1), "n = -1"),
])
def test_lowres_validation_rejects(kw, needle):
    rc, msg = _lowres_call(**kw)
    assert rc == smol.ERR_INVALID_ARG, (rc, msg)
    assert needle in msg


def test_lowres_empty_batch_is_a_no_op():
    rc, _ = _lowres_call(n=0, ws=0)
    assert rc == smol.OK


@pytest.mark.parametrize("kw,needle", [
    (dict(slots=0), "slots"), (dict(slots=65), "slots"), (dict(streams=0), "streams"),
    (dict(streams=17), "streams"), (dict(input_bytes=0), "input_bytes"),
    (dict(output_bytes=8), "output_bytes"), (dict(reserved=1), "reserved"),
    (dict(copy_streams=5), "copy_streams"), (dict(copy_streams=-1), "copy_streams"),
    (dict(workspace_bytes=-1), "workspace_bytes"),
])
def test_pipeline_config_validation(kw, needle):
    cfg = smol.PipelineConfig()
    cfg.slots, cfg.streams, cfg.input_bytes, cfg.output_bytes = 2, 1, 1024, 1024
    for k, v in kw.items():
        setattr(cfg, k, v)
    h = ctypes.c_void_p(1)
    rc = smol.lib().smol_pipeline_create(ctypes.byref(cfg), ctypes.byref(h))
    assert rc == smol.ERR_INVALID_ARG and h.value is None
    assert needle in smol.lib().smol_last_error().decode()


def test_pipeline_null_handles_are_rejected():
    lib = smol.lib()
    slot, host, out = ctypes.c_int32(), ctypes.c_void_p(), ctypes.c_void_p()
    assert lib.smol_pipeline_acquire(None, ctypes.byref(slot), ctypes.byref(host),
                                     ctypes.byref(out)) == smol.ERR_INVALID_ARG
    assert lib.smol_pipeline_release(None, 0) == smol.ERR_INVALID_ARG
    assert lib.smol_pipeline_drain(None) == smol.ERR_INVALID_ARG
    assert lib.smol_pipeline_destroy(None) == smol.OK
    p = smol.make_params(256, 224, 224, MEAN, STD, smol.OUT_F16)
    assert lib.smol_pipeline_submit(None, 0, 1, None, None, None, None, None, 0, ctypes.byref(p),
                                    None, smol.CONSUMER(), None) == smol.ERR_INVALID_ARG


@pytest.mark.parametrize("W,H,S,C,mode", [(1920, 1080, 224, 224, 0), (1280, 720, 256, 224, 0),
                                          (641, 359, 128, 112, 0), (17, 33, 16, 8, 0),
                                          (640, 480, 1, 96, 1), (1000, 200, 300, 150, 0)])
def test_jpeg_mcu_rect_matches_oracle(W, H, S, C, mode):
    p = smol.make_params(S, C, C, MEAN, STD, smol.OUT_F16)
    o = smol.make_options(resize_mode=mode)
    assert smol.jpeg_mcu_rect(W, H, p, o) == oracle.jpeg_mcu_rect(W, H, S, C, C, mode)


def test_jpeg_sizes_match_oracle():
    for W, H in [(1, 1), (16, 16), (17, 33), (1920, 1080)]:
        assert smol.jpeg_coef_count(W, H) == oracle.jpeg_coef_count(W, H)
    w, h = [3, 16], [5, 16]
    assert smol.jpeg_workspace_bytes(w, h) == ((15 + 2 * 2 * 3 + 256 + 2 * 64 + 15) // 16) * 16 + 16


def _jpeg_decode_call(qt=None, rect=(0, 0, 16, 16), out_bytes=16 * 16 + 2 * 64, n=1, nq=1,
                      layout=0, coef_elems=10**6):
    q = np.ones(128, np.uint16) if qt is None else np.asarray(qt, np.uint16)
    w = np.asarray([16], np.int32)
    z = np.zeros(1, np.int64)
    r = None if rect is None else np.asarray(rect, np.int32)
    rc = smol.lib().smol_jpeg_decode_i420(FAKE_SRC, coef_elems, z.ctypes.data, q.ctypes.data, nq,
                                          w.ctypes.data, w.ctypes.data,
                                          None if r is None else r.ctypes.data, n, layout,
                                          FAKE_OUT, out_bytes, z.ctypes.data,
                                          np.asarray([256], np.int64).ctypes.data,
                                          np.asarray([320], np.int64).ctypes.data, None)
    return rc, smol.lib().smol_last_error().decode()


@pytest.mark.parametrize("kw,needle", [
    (dict(qt=[0] + [1] * 127), "entry 0 = 0"), (dict(qt=[1] * 127 + [256]), "entry 127"),
    (dict(nq=2), "n_qtables = 2"), (dict(nq=0), "n_qtables = 0"),
    (dict(layout=2), "coef_layout 2"), (dict(layout=1, rect=None), "needs rects"),
    (dict(coef_elems=6 * 64 - 1), "outside coef"),
    (dict(layout=1, rect=(0, 0, 8, 8), coef_elems=6 * 64 - 1), "outside coef"),
    (dict(rect=(1, 0, 8, 8)), "odd origin"), (dict(rect=(0, 0, 17, 16)), "rectangle"),
    (dict(out_bytes=383), "outside out"), (dict(n=-1), "n = -1"),
])
def test_jpeg_decode_validation(kw, needle):
    rc, msg = _jpeg_decode_call(**kw)
    assert rc == smol.ERR_INVALID_ARG and needle in msg, (rc, msg)


def _jpeg_roi_call(opts=None, ws=FAKE_OUT + 4096, ws_bytes=None, params=None):
    p = params or smol.make_params(32, 24, 24, MEAN, STD, smol.OUT_F16)
    w = np.asarray([64], np.int32)
    h = np.asarray([48], np.int32)
    q = np.ones(128, np.uint16)
    z = np.zeros(1, np.int64)
    need = smol.lib().smol_jpeg_workspace_bytes(1, w.ctypes.data, h.ctypes.data)
    rc = smol.lib().smol_jpeg_roi_preprocess_batch(
        FAKE_SRC, 10**6, z.ctypes.data, q.ctypes.data, 1, w.ctypes.data, h.ctypes.data, 1, 0,
        ctypes.byref(p), None if opts is None else ctypes.byref(opts), ws,
        need if ws_bytes is None else ws_bytes, FAKE_OUT, None)
    return rc, smol.lib().smol_last_error().decode()


@pytest.mark.parametrize("kw,needle", [
    (dict(opts=smol.make_options(chroma_siting=smol.CHROMA_LEFT)), "centred"),
    (dict(opts=smol.make_options(layout=3)), "layout"),
    (dict(ws_bytes=100), "workspace"),
    (dict(ws=FAKE_OUT + 4), "aligned"),
    (dict(params=smol.make_params(32, 40, 40, MEAN, STD, smol.OUT_F16)), "larger than resized"),
])
def test_jpeg_roi_preprocess_validation(kw, needle):
    rc, msg = _jpeg_roi_call(**kw)
    assert rc == smol.ERR_INVALID_ARG and needle in msg, (rc, msg)


@pytest.mark.parametrize("kw, needle", [
    (dict(read_bytes=24), "multiples of 16"),
    (dict(write_bytes=8), "multiples of 16"),
    (dict(read_bytes=0, write_bytes=0), "nothing"),
    (dict(src=0), "non-null"),
    (dict(src=FAKE_SRC + 8), "aligned"),
    (dict(dst=0, write_bytes=64), "non-null"),
    (dict(waves=0), "waves"),
    (dict(waves=(1 << 20) + 1), "waves"),
    (dict(flags=8), "flags"),
])
def test_stream_probe_validation(kw, needle):
    a = dict(src=FAKE_SRC, read_bytes=1024, dst=FAKE_OUT, write_bytes=0, waves=64, flags=3)
    a.update(kw)
    rc = smol.lib().smol_stream_probe(a["src"] or None, a["read_bytes"], a["dst"] or None,
                                      a["write_bytes"], a["waves"], a["flags"], None)
    assert rc == smol.ERR_INVALID_ARG
    assert needle in smol.lib().smol_last_error().decode()


@pytest.mark.parametrize("kind, waves, iters, ticks, needle", [
    (-1, 64, 16, FAKE_OUT, "kind"), (16, 64, 16, FAKE_OUT, "kind"),
    (0, 0, 16, FAKE_OUT, "waves"), (0, (1 << 20) + 1, 16, FAKE_OUT, "waves"),
    (0, 64, 0, FAKE_OUT, "iters"), (0, 64, 16, 0, "NULL"),
])
def test_valu_probe_validation(kind, waves, iters, ticks, needle):
    rc = smol.lib().smol_valu_probe(kind, waves, iters, ticks or None, None)
    assert rc == smol.ERR_INVALID_ARG
    assert needle in smol.lib().smol_last_error().decode()


def test_valu_probe_kinds_match_the_header():
    """The binding's kind names follow the header's SMOL_VALU_* numbering."""
    hdr = open(os.path.join(os.path.dirname(__file__), "..", "include", "smol_stream.h")).read()
    kinds = {int(v): n for n, v in re.findall(r"#define SMOL_VALU_(\w+) (\d+)", hdr)}
    count = kinds.pop(len(smol.VALU_KINDS), None)
    assert count == "KINDS"
    assert sorted(kinds) == list(range(len(smol.VALU_KINDS)))
    for k, name in kinds.items():
        assert name.lower().replace("_", "") == smol.VALU_KINDS[k].replace("_", ""), (k, name)


def test_noalloc_refuses_batches_over_its_table():
    n = 4097
    p = _params()
    offs = np.zeros(n, np.int64)
    w = np.full(n, 320, np.int32)
    h = np.full(n, 240, np.int32)
    rc = smol.lib().smol_preprocess_batch_noalloc(FAKE_SRC, 10**9, offs.ctypes.data, w.ctypes.data,
                                                  h.ctypes.data, None, n, ctypes.byref(p),
                                                  FAKE_OUT, None)
    assert rc == smol.ERR_UNSUPPORTED
    assert "4096" in smol.lib().smol_last_error().decode()


@pytest.mark.parametrize("kw", [dict(crop_h=0), dict(crop_w=0), dict(resize_short=0),
                                dict(std=(0.0, 1.0, 1.0))])
@pytest.mark.parametrize("mode", [smol.RESIZE_SHORT_CROP, smol.RESIZE_DIRECT])
def test_mcu_rect_checks_params_like_the_batch_calls(kw, mode):
    # a zero crop under a direct resize once reached a division by zero
    p = _params(**kw)
    rect = np.zeros(4, np.int32)
    rc = smol.lib().smol_jpeg_mcu_rect(640, 480, ctypes.byref(p),
                                       ctypes.byref(smol.make_options(mode)), rect.ctypes.data)
    assert rc == smol.ERR_INVALID_ARG
