/*
 * smol_jpeg.h -- partial JPEG decoding on the GPU ahead of the fused
 * preprocessing (section 6.4, "ROI decoding", and Algorithm 1): only the
 * 8 x 8 blocks of the smallest MCU-aligned rectangle holding what the
 * preprocessing reads are dequantised and inverse-transformed.
 *
 * Scope: baseline JPEG with 4:2:0 subsampling (16 x 16 luma MCUs holding
 * four luma blocks and one Cb and one Cr block). The entropy decoding
 * (Huffman codes, zig-zag order) is bit-serial and runs on the CPU, as in
 * the paper's system (smol_jpeg_entropy_decode_batch, host threads); the GPU
 * calls take its output, int16 coefficients per block in natural order (row
 * = vertical frequency v, column = horizontal frequency u), blocks in raster
 * order over the MCU-padded frame -- 2 ceil(W/16) x 2 ceil(H/16) luma
 * blocks, then ceil(W/16) x ceil(H/16) Cb blocks, then as many Cr blocks.
 *
 * Arithmetic (one definition, also the tests' reference): dequantised value
 * = coefficient x table entry (exact in fp32); the ITU-T T.81 A.3.3 inverse
 * DCT as two 1-D passes in fp32, horizontal frequencies first, each sum in
 * increasing frequency order with every product and sum rounded on its own,
 * cosine table c[k][n] = C(k)/2 cos((2n+1) k pi / 16) (C(0) = 1/sqrt 2)
 * formed in double and rounded once; then + 128, rounded to nearest (ties to
 * even), clamped to 0..255. Chroma is centred (JPEG).
 */
#ifndef SMOL_JPEG_H
#define SMOL_JPEG_H

#include <stdint.h>

#include "smol.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Coefficient layouts of a frame:
 *   SMOL_JPEG_COEF_FRAME   the whole MCU-padded frame, as above;
 *   SMOL_JPEG_COEF_WINDOW  only the MCU window of the frame's rectangle (MCU
 *                          columns x/16 .. (x+w-1)/16 and rows likewise, for
 *                          a rectangle x, y, w, h): its luma blocks in raster
 *                          order (2 columns and 2 rows per MCU), then its Cb
 *                          blocks, then its Cr blocks. Partial decoding needs
 *                          nothing else, so this is what crosses to the GPU. */
#define SMOL_JPEG_COEF_FRAME 0
#define SMOL_JPEG_COEF_WINDOW 1

/* int16 coefficients of one width x height frame (0 if a size is < 1). */
int64_t smol_jpeg_coef_count(int32_t width, int32_t height);

/* int16 coefficients of the MCU window of rect (HOST int32[4]; NULL: the
 * whole frame) in a width x height frame; 0 if a size is < 1 or the
 * rectangle leaves the frame. */
int64_t smol_jpeg_window_coef_count(int32_t width, int32_t height, const int32_t *rect);

/* smol_jpeg_mcu_rect -- Algorithm 1: the smallest rectangle aligned to the
 * 16 x 16 MCU grid (clipped to the frame) that holds every luma and chroma
 * sample the preprocessing of a width x height frame under p reads
 * (opts->resize_mode; opts may be NULL). The algorithm's own scale factor is
 * replaced by the exact footprint of the resize taps. rect: HOST int32[4],
 * x, y, w, h in luma pixels. Host only; returns SMOL_OK or the status the
 * batch calls would return for these parameters. */
int smol_jpeg_mcu_rect(int32_t width, int32_t height, const smol_params *p,
                       const smol_options *opts, int32_t *rect);

/* smol_jpeg_decode_i420 -- decode the blocks of each frame that meet its
 * rectangle into I420 planes.
 *
 *   coef          DEVICE int16 coefficients, 16-byte aligned; frame i's at
 *                 element coef_offsets[i] (HOST [n], multiples of 8), in
 *                 coef_layout: SMOL_JPEG_COEF_FRAME (smol_jpeg_coef_count
 *                 elements) or SMOL_JPEG_COEF_WINDOW (the MCU window of its
 *                 rectangle, smol_jpeg_window_coef_count elements; rects
 *                 needed), all inside coef_elems elements.
 *   qtables       HOST uint16[n_qtables][2][64]: luma and chroma dequantisation
 *                 tables, natural order, entries 1..255; n_qtables = 1 (one
 *                 pair for every frame) or n (frame i's pair at 128 i).
 *   widths, heights  HOST [n], 1 .. SMOL_MAX_DIM.
 *   rects         HOST [n][4] (x, y, w, h, luma pixels, inside the frame;
 *                 x and y even) or NULL for whole frames. A block is decoded
 *                 when it holds a pixel of the rectangle (chroma: a sample
 *                 of its columns x/2 .. (x+w-1)/2 and rows likewise).
 *   out           DEVICE, out_bytes bytes: frame i's Y plane (W x H) at
 *                 y_offsets[i], its Cb and Cr planes (ceil(W/2) x ceil(H/2))
 *                 at cb_offsets[i] and cr_offsets[i] (HOST [n]), tightly
 *                 pitched. Pixels of blocks that are not decoded are not
 *                 written.
 *   stream        as for smol_preprocess_batch.
 * Returns SMOL_OK, SMOL_ERR_INVALID_ARG (nothing enqueued) or SMOL_ERR_HIP. */
int smol_jpeg_decode_i420(const int16_t *coef, int64_t coef_elems, const int64_t *coef_offsets,
                          const uint16_t *qtables, int32_t n_qtables, const int32_t *widths,
                          const int32_t *heights, const int32_t *rects, int32_t n,
                          int32_t coef_layout, uint8_t *out, int64_t out_bytes,
                          const int64_t *y_offsets, const int64_t *cb_offsets,
                          const int64_t *cr_offsets, void *stream);

/* Bytes of workspace smol_jpeg_roi_preprocess_batch needs: the n I420
 * frames packed back to back (frame i's Y, Cb, Cr planes at the running
 * offset), rounded up to 16, plus 16. */
int64_t smol_jpeg_workspace_bytes(int32_t n, const int32_t *widths, const int32_t *heights);

/* smol_jpeg_roi_preprocess_batch -- Algorithm 1 end to end: for each frame
 * the MCU rectangle of the preprocessing under p and opts (smol_jpeg_mcu_rect),
 * only its blocks decoded into the workspace, then
 * smol_yuv420_preprocess_batch_ex over the workspace (no ROI; centred chroma
 * only). The output equals that of decoding whole frames.
 *
 *   coef_layout SMOL_JPEG_COEF_FRAME, or SMOL_JPEG_COEF_WINDOW for
 *               coefficients of each frame's MCU window, the rectangle being
 *               smol_jpeg_mcu_rect under the same p and opts (as
 *               smol_jpeg_entropy_decode_batch writes them given those
 *               rectangles).
 *   workspace   DEVICE, 16-byte aligned, at least smol_jpeg_workspace_bytes;
 *               overlaps neither coef nor out.
 *   opts        resize_mode and layout as for the _ex calls; chroma_siting
 *               must be SMOL_CHROMA_CENTER; may be NULL.
 *   out, stream as for smol_preprocess_batch_ex.
 * Both steps are validated before the first launch. Returns as
 * smol_jpeg_decode_i420. */
int smol_jpeg_roi_preprocess_batch(const int16_t *coef, int64_t coef_elems,
                                   const int64_t *coef_offsets, const uint16_t *qtables,
                                   int32_t n_qtables, const int32_t *widths,
                                   const int32_t *heights, int32_t n, int32_t coef_layout,
                                   const smol_params *p, const smol_options *opts,
                                   void *workspace, int64_t workspace_bytes, void *out,
                                   void *stream);

/* ------------------------------------------------------------------------
 * Entropy decoding on the host (ITU-T T.81: Annex B stream syntax, Annex C
 * Huffman tables, Annex F sequential decoding). Accepted streams: baseline
 * (SOF0) or extended sequential (SOF1) Huffman coding, 8-bit samples, three
 * components sampled 2x2, 1x1, 1x1 (4:2:0) in one interleaved scan, Cb and
 * Cr on one quantisation table, 8-bit table entries, optional restart
 * intervals. Other JPEGs (progressive, arithmetic, other subsampling,
 * grayscale) fail with SMOL_ERR_UNSUPPORTED; malformed streams with
 * SMOL_ERR_INVALID_ARG.
 * ---------------------------------------------------------------------- */

/* What the headers of one stream say. */
typedef struct smol_jpeg_info {
    int32_t width, height;      /* luma pixels                             */
    int32_t restart_interval;   /* MCUs per restart interval, 0: none      */
    int32_t reserved;
    int64_t scan_offset;        /* first byte of the entropy-coded data    */
    uint16_t qtables[2][64];    /* luma, chroma tables, natural order      */
} smol_jpeg_info;

/* smol_jpeg_read_info -- parse the markers of one stream (HOST, `bytes`
 * bytes) up to the start of its scan. Host only. */
int smol_jpeg_read_info(const uint8_t *data, int64_t bytes, smol_jpeg_info *info);

/* smol_jpeg_entropy_decode_batch -- entropy-decode n streams into the
 * coefficient layout above, one stream per host thread at a time.
 *
 *   data          HOST: stream i is bytes offsets[i] .. offsets[i] + sizes[i]
 *                 - 1 (HOST [n] tables), all inside data_bytes.
 *   rects         HOST [n][4] (x, y, w, h in luma pixels, inside the frame)
 *                 or NULL. With a rectangle only the MCUs from the first to
 *                 the last that hold one of its pixels are decoded (restart
 *                 intervals wholly before the first are skipped unread), and
 *                 only blocks of the MCU rows and columns it spans are
 *                 written: every block smol_jpeg_decode_i420 reads for the
 *                 same rectangle (or for any rectangle inside those MCUs).
 *                 Other blocks are left as they were.
 *   coef          HOST int16: stream i's coefficients at element
 *                 coef_offsets[i] (HOST [n]) in coef_layout (the window
 *                 layout needs rects), inside coef_elems. Pinned memory lets
 *                 the copy to the device run asynchronously.
 *   qtables       HOST uint16 [n][2][64] receiving each stream's luma and
 *                 chroma tables (natural order), or NULL.
 *   threads       worker threads (<= 0: one per CPU in the process's
 *                 affinity mask); at most n and 256 run.
 * Every stream is decoded; the call then returns SMOL_OK or the status of
 * the lowest-numbered failing stream (its coefficients are incomplete), with
 * "image i: ..." in smol_last_error(). */
int smol_jpeg_entropy_decode_batch(const uint8_t *data, int64_t data_bytes,
                                   const int64_t *offsets, const int64_t *sizes, int32_t n,
                                   const int32_t *rects, int16_t *coef, int64_t coef_elems,
                                   const int64_t *coef_offsets, int32_t coef_layout,
                                   uint16_t *qtables, int32_t threads);

#ifdef __cplusplus
}
#endif

#endif /* SMOL_JPEG_H */
