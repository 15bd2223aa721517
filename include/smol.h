/*
 * smol.h -- C ABI of the MI355X (gfx950) fused image-preprocessing library.
 *
 * The library performs, in one pass of hand-written HIP kernels, the
 * preprocessing that the Smol paper (Kang et al., PVLDB 14) identifies as the
 * bottleneck of end-to-end DNN inference on images and video frames: the
 * standard ResNet pipeline of section 2 ("Breakdown of end-to-end DNN
 * inference"), steps 2-4, on already-decoded pixels --
 *
 *   step 2  aspect-preserving resize so the short edge becomes S, then a
 *           central crop of C_h x C_w;
 *   step 3  conversion to float and per-channel normalisation;
 *   step 4  rearrangement to channels-first;
 *
 * fused into a single kernel as section 6.2 allows (normalisation, type
 * conversion and channel reordering fuse; resize and crop may be swapped, so
 * the resize is evaluated only at the cropped output pixels). For planar
 * YCbCr 4:2:0 frames (the decoder output of JPEG and H.264 inputs, App. A
 * "Components": colorspace conversion) the chroma upsample and BT.601
 * conversion run in the same kernel, at every luma pixel the resize reads.
 *
 * Exact semantics (shared by nothing in this library but written down here):
 *   - resized size: the short side becomes S, the long side is
 *     floor(S * long / short); a square image becomes S x S;
 *   - crop offsets: left = floor((W' - C_w) / 2), top = floor((H' - C_h) / 2)
 *     (Algorithm 1's l and t);
 *   - bilinear, half-pixel centres (align_corners = false), edge clamp, no
 *     antialiasing: output index x maps to the source coordinate
 *     ((2x + 1) * in - out) / (2 * out); its integer part is exact, its
 *     fractional weight is rounded once to fp32;
 *   - arithmetic in fp32; output (v - mean_c) / std_c, NCHW, RGB order;
 *   - fp16 output is rounded to nearest even;
 *   - YCbCr: BT.601 full range (Kr = 0.299, Kb = 0.114), centred 4:2:0 siting
 *     (the chroma coordinate of luma index x is x/2 - 1/4, clamped), each
 *     channel clamped to [0, 255] in fp32 before the resize.
 *
 * Threading and streams: every call enqueues work on the caller's HIP stream
 * and returns without synchronising. Calls are thread-safe; calls from
 * different threads on different streams may overlap. Validation is complete
 * before anything is enqueued: a call that returns an error has enqueued
 * nothing. Device faults (only possible if the caller's buffers are smaller
 * than declared) surface at the caller's next synchronisation.
 */
#ifndef SMOL_H
#define SMOL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define SMOL_OK 0
#define SMOL_ERR_INVALID_ARG (-1) /* a null pointer, a size out of range, a   */
                                  /* buffer too small for its table entries  */
#define SMOL_ERR_UNSUPPORTED (-2) /* valid in principle, beyond the library's */
                                  /* limits (see the per-call notes)          */
#define SMOL_ERR_HIP (-3)         /* the HIP runtime reported an error        */

/* Output element types. SMOL_OUT_U8 holds the resized value itself, rounded
 * to the nearest integer with ties to even (no normalisation; mean and std
 * are then not used). It runs on the row-streaming kernels (contiguous row
 * order; the row_order knob is ignored) and the direct kernels, and for I420
 * input on the direct kernel only: with it, a forced LDS-staged or
 * register-gather path, or a forced row-streaming path for I420 input, fails
 * with SMOL_ERR_UNSUPPORTED. */
#define SMOL_OUT_F32 0
#define SMOL_OUT_F16 1
#define SMOL_OUT_U8 2

/* Limits. */
#define SMOL_MAX_DIM 65535          /* max source width / height, luma pixels */
#define SMOL_MAX_RESIZED 4194303    /* max resized width / height (< 2^22)    */
#define SMOL_MAX_BATCH 1048576      /* max images per call                    */

/* Preprocessing parameters, read during the call only.
 *   resize_short  S, the short side after the aspect-preserving resize (>= 1)
 *   crop_h/crop_w output height / width; the crop must fit inside the resized
 *                 image of every image in the batch
 *   out_dtype     SMOL_OUT_F32, SMOL_OUT_F16 or SMOL_OUT_U8
 *   mean, std     per channel R, G, B in 0..255 pixel units; finite, std != 0
 *                 (not used, and not checked, with SMOL_OUT_U8)
 *                 (the ImageNet statistics are (0.485, 0.456, 0.406) * 255 and
 *                 (0.229, 0.224, 0.225) * 255) */
typedef struct smol_params {
    int32_t resize_short;
    int32_t crop_h;
    int32_t crop_w;
    int32_t out_dtype;
    float mean[3];
    float std[3];
} smol_params;

/* Per-image geometry as the kernels use it (host-side query).
 *   resized_w/h     W', H'
 *   crop_left/top   Algorithm 1's l, t
 *   src_x_first/last  first and last source column any output pixel reads
 *                     (inclusive; luma columns for YUV input)
 *   src_rows        number of distinct source rows the vertical taps read
 *                   (luma rows for YUV input)
 *   chroma_x_first/last, chroma_rows  the same for each chroma plane of a
 *                   YUV 4:2:0 frame (0 for RGB queries) */
typedef struct smol_geometry {
    int32_t resized_w;
    int32_t resized_h;
    int32_t crop_left;
    int32_t crop_top;
    int32_t src_x_first;
    int32_t src_x_last;
    int32_t src_rows;
    int32_t chroma_x_first;
    int32_t chroma_x_last;
    int32_t chroma_rows;
} smol_geometry;

/* smol_preprocess_batch -- packed HWC RGB uint8 images -> NCHW.
 *
 * Section 2, steps 2-4, fused per section 6.2.
 *
 *   src        DEVICE pointer, caller-owned: every image's bytes. No alignment
 *              requirement.
 *   src_bytes  size of the src buffer in bytes; every image must lie inside.
 *   offsets    HOST [n]: byte offset in src of image i's first pixel (>= 0).
 *   widths, heights  HOST [n]: image i is widths[i] x heights[i] pixels,
 *              1 .. SMOL_MAX_DIM each.
 *   row_pitch  HOST [n]: bytes between rows of image i (>= 3 * widths[i]),
 *              or NULL for tightly packed rows (3 * widths[i]).
 *   n          number of images, 0 .. SMOL_MAX_BATCH (0 enqueues nothing).
 *   p          parameters (HOST).
 *   out        DEVICE pointer, caller-owned, 16-byte aligned:
 *              n x 3 x crop_h x crop_w elements of p->out_dtype, dense.
 *   stream     hipStream_t of the current device, or NULL for the default
 *              stream.
 *
 * Host tables and p are read before the call returns. When the images do not
 * share one size and a constant offset stride, the call writes a per-image
 * descriptor table (80 bytes per image) to a pinned staging buffer that the
 * library keeps per device and reuses in stream order; the kernel reads it
 * from there (see smol_tuning.upload).
 *
 * Returns SMOL_OK, SMOL_ERR_INVALID_ARG (nothing enqueued),
 * SMOL_ERR_UNSUPPORTED (resized side beyond SMOL_MAX_RESIZED) or SMOL_ERR_HIP.
 */
int smol_preprocess_batch(const uint8_t *src, int64_t src_bytes, const int64_t *offsets,
                          const int32_t *widths, const int32_t *heights,
                          const int32_t *row_pitch, int32_t n, const smol_params *p, void *out,
                          void *stream);

/* smol_preprocess_batch_noalloc -- smol_preprocess_batch for callers that
 * cannot allocate memory during the call (tight serving loops, harnesses
 * that forbid allocation).
 *
 * Same arguments, validation, kernels and results as smol_preprocess_batch.
 * The call allocates nothing: no device memory, no pinned host memory (the
 * library's other calls allocate the descriptor table and its staging buffer
 * on first use). A batch that needs a descriptor table (images of different
 * sizes or offset strides) keeps it in a fixed device array of
 * SMOL_NOALLOC_MAX_IMAGES descriptors that the library holds on every device
 * it runs on until the process ends; the table is copied there from host
 * memory with an ordinary asynchronous host-to-device copy on `stream`.
 *
 * Limit: n <= SMOL_NOALLOC_MAX_IMAGES (else SMOL_ERR_UNSUPPORTED, nothing
 * enqueued).
 *
 * Every call on a device shares that device's array. Calls on one stream are
 * ordered by the stream; calls that overlap on one device (different streams
 * with no ordering between them, or different host threads) race for the
 * array and must not be issued.
 *
 * Returns as smol_preprocess_batch.
 */
#define SMOL_NOALLOC_MAX_IMAGES 4096
int smol_preprocess_batch_noalloc(const uint8_t *src, int64_t src_bytes, const int64_t *offsets,
                                  const int32_t *widths, const int32_t *heights,
                                  const int32_t *row_pitch, int32_t n, const smol_params *p,
                                  void *out, void *stream);

/* smol_yuv420_preprocess_batch -- planar YCbCr 4:2:0 (I420) uint8 frames ->
 * NCHW RGB.
 *
 * App. A "Components" (colorspace conversion) followed by section 2,
 * steps 2-4, all in one kernel.
 *
 *   src         DEVICE pointer, caller-owned, no alignment requirement.
 *   src_bytes   size of src in bytes; every plane must lie inside.
 *   y_offsets, cb_offsets, cr_offsets  HOST [n]: byte offsets in src of frame
 *               i's Y plane (widths[i] x heights[i]) and Cb and Cr planes
 *               (ceil(W/2) x ceil(H/2) each); all planes tightly pitched.
 *   widths, heights  HOST [n]: luma size, 1 .. SMOL_MAX_DIM.
 *   n, p, out, stream  as for smol_preprocess_batch.
 *
 * Returns as smol_preprocess_batch.
 */
int smol_yuv420_preprocess_batch(const uint8_t *src, int64_t src_bytes, const int64_t *y_offsets,
                                 const int64_t *cb_offsets, const int64_t *cr_offsets,
                                 const int32_t *widths, const int32_t *heights, int32_t n,
                                 const smol_params *p, void *out, void *stream);

/* smol_image_geometry -- the geometry the kernels use for one image of
 * width x height (luma size for yuv420 != 0) under p. Host only; touches no
 * device. Returns SMOL_OK or SMOL_ERR_INVALID_ARG / SMOL_ERR_UNSUPPORTED. */
int smol_image_geometry(int32_t width, int32_t height, int32_t yuv420, const smol_params *p,
                        smol_geometry *g);

/* ------------------------------------------------------------------------
 * Variants: region of interest, direct resize, channels-last, chroma siting.
 *
 * Section 6.4 ("Leveraging partial decoding") lets a caller give an ROI per
 * image (a face, a detection box, the central crop) so that only the ROI is
 * processed, and notes that networks take fixed input sizes (224 x 224 for
 * ResNet-50). Semantics:
 *   - ROI (x, y, w, h), luma pixels for I420: 0 <= x, 0 <= y, w, h >= 1,
 *     x + w <= width, y + h <= height. The ROI is cut out of the decoded image
 *     and processed as a w x h image: the resize taps clamp at the ROI's
 *     edges. For I420 the frame is converted first: chroma taps use frame
 *     coordinates and clamp at the frame's chroma planes.
 *   - resize_mode SMOL_RESIZE_SHORT_CROP: step 2 as above (short side to S,
 *     central crop); SMOL_RESIZE_DIRECT: the image (or ROI) is resized to
 *     crop_w x crop_h, aspect ratio not kept, nothing cropped (resize_short
 *     is then not used, but must still be valid).
 *   - layout SMOL_LAYOUT_NCHW (step 4) or SMOL_LAYOUT_NHWC: n x crop_h x
 *     crop_w x 3, channels last.
 *   - chroma_siting (I420 only) SMOL_CHROMA_CENTER: chroma of luma column x
 *     at x/2 - 1/4 (JPEG); SMOL_CHROMA_LEFT: at x/2 (co-sited, as MPEG-2 and
 *     H.264 decoders emit). Rows are centred (y/2 - 1/4) in both.
 * NHWC output runs on the row-streaming and direct kernels only: with it,
 * a forced LDS-staged or register-gather path fails with
 * SMOL_ERR_UNSUPPORTED. */
#define SMOL_RESIZE_SHORT_CROP 0
#define SMOL_RESIZE_DIRECT 1
#define SMOL_LAYOUT_NCHW 0
#define SMOL_LAYOUT_NHWC 1
#define SMOL_CHROMA_CENTER 0
#define SMOL_CHROMA_LEFT 1

/* Options of the _ex calls (NULL: all zero, the calls above). reserved must
 * be zero. */
typedef struct smol_options {
    int32_t resize_mode;
    int32_t layout;
    int32_t chroma_siting;
    int32_t reserved[5];
} smol_options;

/* smol_preprocess_batch_ex -- smol_preprocess_batch with an ROI per image
 * and options.
 *
 * Section 2 steps 2-4 on the ROI (section 6.4), fused per section 6.2.
 *
 *   rois   HOST [n][4] int32: x, y, w, h of image i's ROI, or NULL for whole
 *          images.
 *   opts   HOST, or NULL.
 *   out    n x 3 x crop_h x crop_w (NCHW) or n x crop_h x crop_w x 3 (NHWC)
 *          elements of p->out_dtype, 16-byte aligned.
 *   Every other argument as for smol_preprocess_batch; the whole image i
 *   must lie inside src, as there. Returns as smol_preprocess_batch. */
int smol_preprocess_batch_ex(const uint8_t *src, int64_t src_bytes, const int64_t *offsets,
                             const int32_t *widths, const int32_t *heights,
                             const int32_t *row_pitch, const int32_t *rois, int32_t n,
                             const smol_params *p, const smol_options *opts, void *out,
                             void *stream);

/* smol_yuv420_preprocess_batch_ex -- smol_yuv420_preprocess_batch with an
 * ROI per frame (luma pixels) and options.
 *
 * App. A "Components" (colorspace conversion, chroma sited per
 * opts->chroma_siting), then section 2 steps 2-4 on the ROI (section 6.4).
 * Arguments as for smol_yuv420_preprocess_batch, plus rois and opts as for
 * smol_preprocess_batch_ex. Returns as smol_preprocess_batch. */
int smol_yuv420_preprocess_batch_ex(const uint8_t *src, int64_t src_bytes,
                                    const int64_t *y_offsets, const int64_t *cb_offsets,
                                    const int64_t *cr_offsets, const int32_t *widths,
                                    const int32_t *heights, const int32_t *rois, int32_t n,
                                    const smol_params *p, const smol_options *opts, void *out,
                                    void *stream);

/* ------------------------------------------------------------------------
 * Low-resolution-aware augmentation (section 5.3, "Training DNNs for
 * Low-resolution Visual Data"): at training time an input is downsampled to
 * the target resolution and upsampled back to the network's input size, so
 * that the network learns the artifacts of stored low-resolution data (the
 * section's example: 161 x 161 thumbnails upscaled to 224 x 224).
 *
 * Two launches of the resize kernels on `stream`:
 *   1. each image (or I420 frame, centred chroma) is reduced to an r x r
 *      uint8 RGB image -- short side resized to r, central r x r crop, values
 *      rounded to nearest, ties to even (SMOL_OUT_U8, NHWC) -- packed in the
 *      workspace, image i at byte i * 3 * r * r;
 *   2. those n r x r images go through smol_preprocess_batch with p.
 * ------------------------------------------------------------------------ */

/* Bytes of workspace the augmentation needs: n * 3 * low_res^2 rounded up to
 * a multiple of 16, plus 16 (0 for n < 1 or low_res < 1). */
int64_t smol_lowres_workspace_bytes(int32_t n, int32_t low_res);

/* smol_lowres_preprocess_batch -- RGB images reduced to low_res x low_res,
 * then preprocessed.
 *
 *   low_res    r, 1 .. SMOL_MAX_DIM.
 *   workspace  DEVICE pointer, caller-owned, 16-byte aligned, at least
 *              smol_lowres_workspace_bytes(n, low_res) bytes; overlaps
 *              neither src nor out. Holds the r x r images when the stream
 *              reaches the second launch; the caller may reuse it once the
 *              call's work on the stream is done.
 *   p          parameters of the second step; p->out_dtype SMOL_OUT_F32 or
 *              SMOL_OUT_F16 (SMOL_OUT_U8: SMOL_ERR_INVALID_ARG).
 *   out        n x 3 x crop_h x crop_w elements, as for
 *              smol_preprocess_batch.
 *   Every other argument as for smol_preprocess_batch. Both steps are
 *   validated before the first launch (the crop must fit the r x r image
 *   resized to p->resize_short). Returns as smol_preprocess_batch. */
int smol_lowres_preprocess_batch(const uint8_t *src, int64_t src_bytes, const int64_t *offsets,
                                 const int32_t *widths, const int32_t *heights,
                                 const int32_t *row_pitch, int32_t n, int32_t low_res,
                                 const smol_params *p, void *workspace, int64_t workspace_bytes,
                                 void *out, void *stream);

/* smol_yuv420_lowres_preprocess_batch -- the same for I420 frames (tables as
 * for smol_yuv420_preprocess_batch). */
int smol_yuv420_lowres_preprocess_batch(const uint8_t *src, int64_t src_bytes,
                                        const int64_t *y_offsets, const int64_t *cb_offsets,
                                        const int64_t *cr_offsets, const int32_t *widths,
                                        const int32_t *heights, int32_t n, int32_t low_res,
                                        const smol_params *p, void *workspace,
                                        int64_t workspace_bytes, void *out, void *stream);

/* smol_image_geometry_ex -- smol_image_geometry of an ROI (HOST int32[4], or
 * NULL for the whole image) under opts (NULL: defaults). resized_w/h and
 * crop_left/top are those of the ROI; src_x_first/last, chroma_x_first/last
 * are in image (frame) coordinates. */
int smol_image_geometry_ex(int32_t width, int32_t height, int32_t yuv420, const int32_t *roi,
                           const smol_params *p, const smol_options *opts, smol_geometry *g);

/* Tuning and testing knobs, process-wide, applied to later calls. Zero in any
 * field means "automatic".
 *   path        1: always the direct-gather kernels (one thread per output
 *               pixel, taps read from global memory); 2: always the
 *               LDS-staged kernels (a call whose source span cannot be staged
 *               then fails with SMOL_ERR_UNSUPPORTED); 3: the persistent
 *               register-gather RGB kernel, with per-image tap tables in LDS
 *               (images whose last 8-byte source window reaches the end of
 *               src use the direct kernel; a crop too wide for the tap
 *               tables fails with SMOL_ERR_UNSUPPORTED); 4: the
 *               row-streaming RGB kernel (crops up to 512 columns whose
 *               source span plus 32 bytes is at most 4 KiB and fits the LDS
 *               budget twice, else SMOL_ERR_UNSUPPORTED; images whose 16-byte
 *               source chunks cross an end of src use the direct kernel);
 *               0: automatic (RGB: row-streaming when it fits, else
 *               register-gather when its tables fit, else LDS-staged when
 *               the span fits, else direct; I420: row-streaming when the
 *               crop is at most 512 columns, the luma span at most 2016
 *               bytes and the chroma span at most 992, else direct). For I420 only 0, 1 and 4 are
 *               valid; 4 fails with SMOL_ERR_UNSUPPORTED past those limits
 *   band_rows   output rows per band in the LDS-staged kernels (1..64); for
 *               the row-streaming kernel, 1 or 2 sets how many output rows
 *               ahead of the interpolated one each wave loads
 *   lds_budget  bytes of LDS one workgroup may use (4096..163840, and at most
 *               the device's per-workgroup limit)
 *   workgroups_per_cu  cap on the resident workgroups per compute unit
 *               the persistent kernels (paths 2-4) are sized for (1..16);
 *               for the row-streaming kernels, whose workgroups hold 1, 2
 *               or 4 independent waves, the cap counts waves; by default as
 *               many as can be resident (row streaming with 4 KiB staged
 *               rows: 8 waves); for block decoding (smol_jpeg.h) the
 *               launch's one-wave workgroups per compute unit (default 128)
 *   exact       1: the row-streaming kernels form the normalisation as the
 *               correctly rounded quotient (v - mean) / std and round to
 *               fp16 from that fp32 value, bit-identical to a scalar fp32
 *               evaluation of the definition (the other kernels always do);
 *               0 (default): they multiply v - mean by RN(1/std), at most
 *               one fp32 ulp from the quotient, and may round that product
 *               to fp16 directly (within one fp16 ulp). Every interpolation
 *               and colour-conversion step is exact in both modes.
 *   row_order   row-streaming kernels: 1 each wave takes a contiguous range
 *               of output rows; 2 wave q of G takes rows q, q + G, ...
 *               (concurrently running waves stream neighbouring rows);
 *               0 (default): 2 for uniform RGB batches whose staged rows
 *               exceed 2 KiB, else 1
 *   upload      how a ragged batch's descriptor table reaches the device:
 *               0 (default) or 3: no copy, the preprocessing kernel reads the
 *               pinned staging slot itself (one launch per call); 1 a DMA
 *               copy on the library's copy stream, which the caller's stream
 *               waits for (overlaps earlier kernels; costs more host time per
 *               call); 2: a small copy kernel on the caller's stream that
 *               moves the pinned staging slot to device memory first */
typedef struct smol_tuning {
    int32_t path;
    int32_t band_rows;
    int32_t lds_budget;
    int32_t workgroups_per_cu;
    int32_t exact;
    int32_t row_order;
    int32_t upload;
    int32_t reserved[1];
} smol_tuning;

/* Set the knobs (NULL resets to automatic). SMOL_ERR_INVALID_ARG if a field
 * is out of range. */
int smol_set_tuning(const smol_tuning *t);

/* How the calling thread's last successful batch call ran.
 *   path        1 direct-gather, 2 LDS-staged, 3 register-gather, 4 row
 *               streaming (the most specialised kernel the call launched)
 *   band_rows   output rows per band (LDS-staged) or 0
 *   lds_bytes   dynamic LDS per workgroup of that kernel
 *   launches    kernel launches the call made (all kernels)
 *   uploaded_descriptors  1 if a per-image descriptor table was uploaded
 *               (ragged batch), 0 if the batch was uniform
 *   grid        workgroups of that kernel's first launch (0 for direct)
 *   work_items  of that launch: bands (LDS-staged), passes of 2048 output
 *               pixels (register-gather), output rows (row streaming) or
 *               output pixels (direct) */
typedef struct smol_plan {
    int32_t path;
    int32_t band_rows;
    int32_t lds_bytes;
    int32_t launches;
    int32_t uploaded_descriptors;
    int32_t grid;
    int64_t work_items;
} smol_plan;

int smol_last_plan(smol_plan *plan);

/* Static description of a status code. */
const char *smol_status_string(int status);

/* Detail of the last error returned on the calling thread ("" if none). */
const char *smol_last_error(void);

/* Library ABI version (major * 10000 + minor * 100 + patch). */
int smol_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SMOL_H */
