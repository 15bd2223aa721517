"""Seeded synthetic workloads shaped like the paper's inputs.

This module only *generates inputs*: pixel buffers, per-image offset and size
tables, and the preprocessing parameters of each workload. It contains none of
the preprocessing arithmetic, so both the HIP path and the CPU oracle can be fed
from it without sharing any of the method.

The paper's datasets (ImageNet-style full-resolution photos, 161 px thumbnails,
1080p / 480p traffic-camera video; section 8, "Datasets") are not available, so
seeded stand-ins reproduce their shapes, size mix and value ranges:

  c1  32 x 320x240 RGB, uniform 0..255; short side 256, crop 224, fp32 out
  c2  256 ragged RGB, W and H each uniform in [300, 600], packed back to back
      with no alignment; short side 256, crop 224, fp16 out
  c3  1024 x 128x128 RGB smooth gradients + noise +-16 (natively low-res
      thumbnails); upscale to 224x224, fp16 out
  c4  64 x 1920x1080 RGB video frames: windows of one random base image at
      small per-frame shifts; short side 224, crop 224, fp16 out
  c5  128 x 1280x720 planar YCbCr 4:2:0 frames, Y in 16..235, Cb/Cr in 16..240;
      short side 256, crop 224, fp16 out
  c6  256 regions of interest (64..512 px boxes) in 16 1080p RGB frames,
      resized directly to 112x112, channels-last fp16 (detection / face crops,
      the ROI use of section 6.4)
  c8  128 JPEG-coded 1280x720 4:2:0 frames as entropy-decoded coefficient
      blocks (smooth DC field, Laplacian AC falling with frequency, synthetic
      quantisation tables); only Algorithm 1's MCU rectangle is decoded,
      then short side 256, crop 224, fp16 out (section 6.4, ROI decoding)
  c7  256 ragged RGB as c2, low-resolution augmentation: reduced to 161x161
      (the thumbnail size of section 5.2) then upsampled to 224x224 (short
      side 224, crop 224), fp16 out (the training augmentation of section 5.3)

Config k draws from ``numpy.random.default_rng(13005 + k)`` (PCG64).
The normalisation constants are the ImageNet per-channel statistics the
standard ResNet pipeline uses (section 2, step 3), scaled to 0..255 units and
rounded once to fp32.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

OUT_F32 = 0
OUT_F16 = 1
OUT_U8 = 2

# (0.485, 0.456, 0.406) * 255 and (0.229, 0.224, 0.225) * 255, formed in double
# and rounded once to fp32.
IMAGENET_MEAN_255 = (np.array([0.485, 0.456, 0.406], np.float64) * 255.0).astype(np.float32)
IMAGENET_STD_255 = (np.array([0.229, 0.224, 0.225], np.float64) * 255.0).astype(np.float32)

SEED_BASE = 13005


@dataclass
class Workload:
    """One batch of inputs plus the preprocessing parameters to apply."""

    name: str
    kind: str  # "rgb" (packed HWC uint8) or "yuv420" (planar I420 uint8)
    src: np.ndarray  # flat uint8 buffer holding every image / plane
    widths: np.ndarray  # int32 [n]
    heights: np.ndarray  # int32 [n]
    resize_short: int
    crop_h: int
    crop_w: int
    out_dtype: int
    offsets: np.ndarray | None = None  # int64 [n], rgb: first byte of image i
    pitches: np.ndarray | None = None  # int32 [n], rgb: row pitch in bytes (None: 3W)
    y_offsets: np.ndarray | None = None  # int64 [n], yuv420
    cb_offsets: np.ndarray | None = None
    cr_offsets: np.ndarray | None = None
    mean: np.ndarray = field(default_factory=lambda: IMAGENET_MEAN_255.copy())
    std: np.ndarray = field(default_factory=lambda: IMAGENET_STD_255.copy())
    description: str = ""
    # variants: an ROI per image (int32 [n, 4]: x, y, w, h), the resize mode
    # (0 short side + centre crop, 1 direct), the layout (0 NCHW, 1 NHWC) and
    # the I420 chroma siting (0 centred, 1 co-sited)
    rois: np.ndarray | None = None
    resize_mode: int = 0
    layout: int = 0
    siting: int = 0
    # low-resolution augmentation: each image first reduced to low_res x
    # low_res (0: off)
    low_res: int = 0
    # kind "jpeg": src holds the int16 coefficients' bytes; frame i's start at
    # element coef_offsets[i]; qtables (2, 64) uint16, luma then chroma, for
    # every frame, or (n, 2, 64), one pair per frame
    coef_offsets: np.ndarray | None = None
    qtables: np.ndarray | None = None

    def frame_qtables(self, i: int) -> tuple[np.ndarray, np.ndarray]:
        """Frame i's (luma, chroma) dequantisation tables."""
        q = np.asarray(self.qtables).reshape(-1, 2, 64)
        q = q[0] if len(q) == 1 else q[i]
        return q[0], q[1]

    @property
    def variant(self) -> bool:
        return (self.rois is not None or self.resize_mode != 0 or self.layout != 0 or
                self.siting != 0)

    @property
    def n(self) -> int:
        return int(len(self.widths))

    @property
    def out_elem_bytes(self) -> int:
        return {OUT_F32: 4, OUT_F16: 2, OUT_U8: 1}[self.out_dtype]

    def out_shape(self) -> tuple[int, int, int, int]:
        if self.layout == 1:
            return (self.n, self.crop_h, self.crop_w, 3)
        return (self.n, 3, self.crop_h, self.crop_w)


def _pack_rgb(images: list[np.ndarray], align: int = 1):
    """Pack HxWx3 uint8 images back to back (offset of each rounded up to align)."""
    offsets, cur = [], 0
    for im in images:
        cur = (cur + align - 1) // align * align
        offsets.append(cur)
        cur += im.size
    src = np.zeros(cur, np.uint8)
    for off, im in zip(offsets, images):
        src[off:off + im.size] = im.reshape(-1)
    return src, np.asarray(offsets, np.int64)


def rgb_workload(name: str, images: list[np.ndarray], S: int, C: int | tuple[int, int],
                 out_dtype: int, align: int = 1, description: str = "") -> Workload:
    """Wrap a list of HxWx3 uint8 images as a packed ragged batch."""
    ch, cw = (C, C) if isinstance(C, int) else C
    src, offsets = _pack_rgb(images, align)
    return Workload(name=name, kind="rgb", src=src,
                    widths=np.asarray([im.shape[1] for im in images], np.int32),
                    heights=np.asarray([im.shape[0] for im in images], np.int32),
                    resize_short=S, crop_h=ch, crop_w=cw, out_dtype=out_dtype,
                    offsets=offsets, description=description)


def uniform_rgb_workload(name: str, batch: np.ndarray, S: int, C: int | tuple[int, int],
                         out_dtype: int, description: str = "") -> Workload:
    """A dense N x H x W x 3 uint8 batch (image i at offset i*H*W*3)."""
    n, h, w, _ = batch.shape
    ch, cw = (C, C) if isinstance(C, int) else C
    stride = h * w * 3
    return Workload(name=name, kind="rgb", src=np.ascontiguousarray(batch).reshape(-1),
                    widths=np.full(n, w, np.int32), heights=np.full(n, h, np.int32),
                    resize_short=S, crop_h=ch, crop_w=cw, out_dtype=out_dtype,
                    offsets=np.arange(n, dtype=np.int64) * stride, description=description)


def yuv420_workload(name: str, planes: list[tuple[np.ndarray, np.ndarray, np.ndarray]], S: int,
                    C: int | tuple[int, int], out_dtype: int, description: str = "") -> Workload:
    """Pack (Y, Cb, Cr) planes per frame as [Y | Cb | Cr], frames back to back."""
    ch, cw = (C, C) if isinstance(C, int) else C
    yo, bo, ro, cur = [], [], [], 0
    for y, cb, cr in planes:
        yo.append(cur)
        cur += y.size
        bo.append(cur)
        cur += cb.size
        ro.append(cur)
        cur += cr.size
    src = np.empty(cur, np.uint8)
    for (y, cb, cr), a, b, c in zip(planes, yo, bo, ro):
        src[a:a + y.size] = y.reshape(-1)
        src[b:b + cb.size] = cb.reshape(-1)
        src[c:c + cr.size] = cr.reshape(-1)
    return Workload(name=name, kind="yuv420", src=src,
                    widths=np.asarray([p[0].shape[1] for p in planes], np.int32),
                    heights=np.asarray([p[0].shape[0] for p in planes], np.int32),
                    resize_short=S, crop_h=ch, crop_w=cw, out_dtype=out_dtype,
                    y_offsets=np.asarray(yo, np.int64), cb_offsets=np.asarray(bo, np.int64),
                    cr_offsets=np.asarray(ro, np.int64), description=description)


# ---------------------------------------------------------------------------
# the five workloads
# ---------------------------------------------------------------------------


def c1(n: int = 32) -> Workload:
    rng = np.random.default_rng(SEED_BASE + 1)
    batch = rng.integers(0, 256, size=(n, 240, 320, 3), dtype=np.uint8)
    return uniform_rgb_workload("c1", batch, 256, 224, OUT_F32,
                                f"{n} x 320x240 RGB uint8 HWC, uniform 0-255; short side 256, "
                                "center crop 224x224, NCHW fp32")


def c2_sizes(n: int = 256) -> np.ndarray:
    """(n, 2) int array of (W, H), each uniform in [300, 600]."""
    rng = np.random.default_rng(SEED_BASE + 2)
    return rng.integers(300, 601, size=(n, 2))


def c2(n: int = 256, align: int = 1) -> Workload:
    rng = np.random.default_rng(SEED_BASE + 2)
    sizes = rng.integers(300, 601, size=(n, 2))
    total = int(sum(int(w) * int(h) * 3 for w, h in sizes))
    pix = rng.integers(0, 256, size=total, dtype=np.uint8)
    images, cur = [], 0
    for w, h in sizes:
        k = int(w) * int(h) * 3
        images.append(pix[cur:cur + k].reshape(int(h), int(w), 3))
        cur += k
    return rgb_workload("c2", images, 256, 224, OUT_F16, align,
                        f"ragged {n} RGB uint8 HWC, W,H ~ U[300,600], packed with "
                        f"{'no' if align == 1 else str(align) + ' B'} alignment; short side "
                        "256, center crop 224x224, NCHW fp16")


def c3(n: int = 1024) -> Workload:
    rng = np.random.default_rng(SEED_BASE + 3)
    size = 128
    yy, xx = np.mgrid[0:size, 0:size].astype(np.float64)
    alpha = rng.uniform(0.0, 255.0, size=(n, 1, 1, 3))
    beta = rng.uniform(-1.0, 1.0, size=(n, 1, 1, 3))
    gamma = rng.uniform(-1.0, 1.0, size=(n, 1, 1, 3))
    noise = rng.integers(-16, 17, size=(n, size, size, 3))
    img = alpha + beta * xx[None, :, :, None] + gamma * yy[None, :, :, None] + noise
    batch = np.clip(np.rint(img), 0, 255).astype(np.uint8)
    return uniform_rgb_workload("c3", batch, 224, 224, OUT_F16,
                                f"{n} x 128x128 RGB uint8 HWC, smooth gradients + noise +-16; "
                                "bilinear upscale to 224x224, NCHW fp16")


def c4(n: int = 64, height: int = 1080, width: int = 1920) -> Workload:
    rng = np.random.default_rng(SEED_BASE + 4)
    margin = 8
    base = rng.integers(0, 256, size=(height + 2 * margin, width + 2 * margin, 3), dtype=np.uint8)
    shifts = rng.integers(-margin, margin + 1, size=(n, 2))
    batch = np.empty((n, height, width, 3), np.uint8)
    for f, (dy, dx) in enumerate(shifts):
        y0, x0 = margin + int(dy), margin + int(dx)
        batch[f] = base[y0:y0 + height, x0:x0 + width]
    return uniform_rgb_workload("c4", batch, 224, 224, OUT_F16,
                                f"{n} x {width}x{height} RGB uint8 HWC video frames (one seeded "
                                "base image, per-frame shifts of up to 8 px); short side 224, "
                                "center crop 224x224, NCHW fp16")


def c5(n: int = 128, height: int = 720, width: int = 1280) -> Workload:
    rng = np.random.default_rng(SEED_BASE + 5)
    hc, wc = (height + 1) // 2, (width + 1) // 2
    ys = rng.integers(16, 236, size=(n, height, width), dtype=np.uint8)
    cbs = rng.integers(16, 241, size=(n, hc, wc), dtype=np.uint8)
    crs = rng.integers(16, 241, size=(n, hc, wc), dtype=np.uint8)
    return yuv420_workload("c5", [(ys[i], cbs[i], crs[i]) for i in range(n)], 256, 224, OUT_F16,
                           f"{n} x {width}x{height} planar YCbCr 4:2:0 uint8 (Y 16-235, Cb/Cr "
                           "16-240); BT.601 full range, short side 256, center crop 224x224, "
                           "NCHW fp16")


def c6(n: int = 256, height: int = 1080, width: int = 1920) -> Workload:
    """Detection / face crops: one ROI per 1080p frame (square-ish boxes of
    64..512 px at random positions), each resized directly to 112x112, fp16,
    channels last -- the shape of a second-stage recogniser's input."""
    rng = np.random.default_rng(SEED_BASE + 6)
    frames = 16  # the ROIs index a smaller set of frames, several per frame
    base = rng.integers(0, 256, size=(frames, height, width, 3), dtype=np.uint8)
    side = rng.integers(64, 513, size=n)
    aspect = rng.uniform(0.75, 1.33, size=n)
    w = np.clip(np.rint(side * np.sqrt(aspect)), 16, width).astype(np.int64)
    h = np.clip(np.rint(side / np.sqrt(aspect)), 16, height).astype(np.int64)
    x = (rng.random(n) * (width - w + 1)).astype(np.int64)
    y = (rng.random(n) * (height - h + 1)).astype(np.int64)
    fi = rng.integers(0, frames, size=n)
    stride = height * width * 3
    wl = Workload(name="c6", kind="rgb", src=base.reshape(-1),
                  widths=np.full(n, width, np.int32), heights=np.full(n, height, np.int32),
                  resize_short=112, crop_h=112, crop_w=112, out_dtype=OUT_F16,
                  offsets=fi.astype(np.int64) * stride,
                  description=f"{n} ROIs (64..512 px boxes) in {frames} x {width}x{height} RGB "
                              "uint8 frames; direct resize to 112x112, NHWC fp16")
    wl.rois = np.stack([x, y, w, h], axis=1).astype(np.int32)
    wl.resize_mode = 1
    wl.layout = 1
    return wl


def c7(n: int = 256, low_res: int = 161) -> Workload:
    """Low-resolution-aware training augmentation over ImageNet-sized photos:
    every image reduced to low_res x low_res, then upsampled to the network's
    224 x 224 input."""
    rng = np.random.default_rng(SEED_BASE + 7)
    sizes = rng.integers(300, 601, size=(n, 2))
    images = [rng.integers(0, 256, size=(int(h), int(w), 3), dtype=np.uint8) for w, h in sizes]
    wl = rgb_workload("c7", images, 224, 224, OUT_F16, 1,
                      f"ragged {n} RGB uint8 HWC, W,H ~ U[300,600]; reduced to "
                      f"{low_res}x{low_res} uint8, then short side 224, center crop 224x224, "
                      "NCHW fp16")
    wl.low_res = low_res
    return wl


def jpeg_qtables() -> np.ndarray:
    """Synthetic dequantisation tables (luma, chroma): coarser with frequency."""
    u = np.arange(8)
    f = u[None, :] + u[:, None]
    return np.stack([2 + 2 * f, 3 + 3 * f]).reshape(2, 64).astype(np.uint16)


def jpeg_coefficients(rng, W: int, H: int, q: np.ndarray) -> np.ndarray:
    """Entropy-decoded coefficients of one W x H 4:2:0 frame (MCU-padded block
    grid, luma then Cb then Cr, 64 per block in natural order): a smooth DC
    field plus Laplacian AC terms whose scale falls with frequency, quantised
    by the tables."""
    bw, bh = 2 * ((W + 15) // 16), 2 * ((H + 15) // 16)
    u = np.arange(8)
    f = (u[None, :] + u[:, None]).reshape(64)
    out = []
    for comp, (gw, gh) in enumerate([(bw, bh), (bw // 2, bh // 2), (bw // 2, bh // 2)]):
        qt = q[0 if comp == 0 else 1].astype(np.float64)
        yy, xx = np.mgrid[0:gh, 0:gw].astype(np.float64)
        a, b, ph = rng.uniform(0.02, 0.2, 2), rng.uniform(0.02, 0.2, 2), rng.uniform(0, 6.3, 2)
        level = 128 + 70 * np.sin(a[0] * xx + b[0] * yy + ph[0]) * np.cos(a[1] * xx - b[1] * yy + ph[1])
        blocks = rng.laplace(0.0, 1.0, size=(gh * gw, 64)) * (40.0 / (1.0 + f))[None, :]
        blocks[:, 0] = (level.reshape(-1) - 128) * 8
        out.append(np.rint(blocks / qt[None, :]).astype(np.int16).reshape(-1))
    return np.concatenate(out)


def jpeg_workload(name: str, sizes, S: int, C: int | tuple[int, int], out_dtype: int, seed: int,
                  description: str = "") -> Workload:
    """Frames of the given (W, H) sizes as coefficient blocks, packed."""
    rng = np.random.default_rng(seed)
    ch, cw = (C, C) if isinstance(C, int) else C
    q = jpeg_qtables()
    coefs = [jpeg_coefficients(rng, int(w), int(h), q) for w, h in sizes]
    offs = np.cumsum([0] + [c.size for c in coefs[:-1]]).astype(np.int64)
    coef = np.concatenate(coefs)
    return Workload(name=name, kind="jpeg", src=coef.view(np.uint8),
                    widths=np.asarray([w for w, _ in sizes], np.int32),
                    heights=np.asarray([h for _, h in sizes], np.int32), resize_short=S,
                    crop_h=ch, crop_w=cw, out_dtype=out_dtype, coef_offsets=offs, qtables=q,
                    description=description)


def photo_ycbcr(rng, W: int, H: int) -> np.ndarray:
    """A W x H x 3 YCbCr uint8 image with photo-like structure: smooth
    luminance and colour fields, a few hard-edged rectangles and fine
    Gaussian grain."""
    yy, xx = np.mgrid[0:H, 0:W].astype(np.float32)
    img = np.empty((H, W, 3), np.float32)
    for c, amp in enumerate((70.0, 35.0, 35.0)):
        a, b, ph = rng.uniform(0.005, 0.08, 2), rng.uniform(0.005, 0.08, 2), rng.uniform(0, 6.3, 2)
        img[..., c] = 128 + amp * np.sin(a[0] * xx + b[0] * yy + ph[0]) * np.cos(
            a[1] * xx - b[1] * yy + ph[1])
    for _ in range(int(rng.integers(2, 6))):
        x0, y0 = int(rng.integers(0, W)), int(rng.integers(0, H))
        x1, y1 = x0 + int(rng.integers(1, max(2, W // 3))), y0 + int(rng.integers(1, max(2, H // 3)))
        img[y0:y1, x0:x1] += rng.uniform(-50, 50, 3).astype(np.float32)
    img += rng.standard_normal(img.shape, dtype=np.float32) * 4.0
    return np.clip(np.rint(img), 0, 255).astype(np.uint8)


def jpeg_files(sizes, seed: int, quality=75, restart_blocks: int = 0,
               distinct: int = 0) -> list[bytes]:
    """Baseline 4:2:0 JPEG streams of seeded photo-like images, encoded by
    libjpeg through PIL, standing in for a JPEG dataset. ``quality`` is one
    libjpeg quality for all or one per image; ``restart_blocks`` > 0 puts a
    restart marker every that many MCUs; ``distinct`` > 0 encodes only the
    first that many streams and repeats them in turn (same sizes needed)."""
    import io

    from PIL import Image
    rng = np.random.default_rng(seed)
    qs = [quality] * len(sizes) if np.isscalar(quality) else list(quality)
    out = []
    for i, ((W, H), q) in enumerate(zip(sizes, qs)):
        if distinct and i >= distinct:
            assert tuple(sizes[i % distinct]) == (W, H)
            out.append(out[i % distinct])
            continue
        b = io.BytesIO()
        kw = {"restart_marker_blocks": int(restart_blocks)} if restart_blocks else {}
        Image.fromarray(photo_ycbcr(rng, int(W), int(H)), "YCbCr").save(
            b, "JPEG", quality=int(q), subsampling=2, **kw)
        out.append(b.getvalue())
    return out


def jpeg_file_batch(n: int = 128, width: int = 1280, height: int = 720, quality: int = 75,
                    restart_blocks: int = 80, distinct: int = 32) -> list[bytes]:
    """The file benchmark's batch: n photo-like width x height streams at one
    libjpeg quality, a restart marker every MCU row of a 1280-wide frame,
    ``distinct`` different images repeated."""
    return jpeg_files([(width, height)] * n, SEED_BASE + 9, quality, restart_blocks, distinct)


def c8(n: int = 128, height: int = 720, width: int = 1280) -> Workload:
    return jpeg_workload("c8", [(width, height)] * n, 256, 224, OUT_F16, SEED_BASE + 8,
                         f"{n} JPEG-coded {width}x{height} 4:2:0 frames as entropy-decoded "
                         "coefficient blocks; only the MCU rectangle of the crop decoded "
                         "(dequantisation, 8x8 inverse DCT), then short side 256, center crop "
                         "224x224, NCHW fp16")


CONFIGS = {"c1": c1, "c2": c2, "c3": c3, "c4": c4, "c5": c5, "c6": c6, "c7": c7, "c8": c8}


def make(name: str, **kw) -> Workload:
    return CONFIGS[name](**kw)
