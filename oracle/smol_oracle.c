/*
 * smol_oracle.c -- plain, slow, scalar CPU oracle for fused image preprocessing
 * (Kang et al., "Jointly Optimizing Preprocessing and Inference for DNN-based
 * Visual Analytics", PVLDB 14).
 *
 * TEST INFRASTRUCTURE. Only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark load this library. The product path (the HIP library)
 * shares no code, header, table or constant with it.
 *
 * What it computes is the standard ResNet preprocessing of the paper's
 * measurement study (section 2, "Breakdown of end-to-end DNN inference",
 * steps 2-4), applied to already-decoded pixels:
 *   step 2  aspect-preserving resize so the short edge is S, then a central
 *           C_h x C_w crop;
 *   step 3  convert to float32 and normalise per channel;
 *   step 4  rearrange to channels-first (NCHW).
 * plus, for planar YCbCr 4:2:0 input, the colorspace conversion that the
 * implementation appendix lists among its preprocessing methods (App. A,
 * "Components"), done before the resize.
 *
 * The crop is taken in output space: resizing and cropping may be swapped
 * (section 6.2, reordering rule 3), so the oracle evaluates the resize only at
 * the output pixels that survive the crop. The crop offsets are Algorithm 1's
 * l = (w' - 224)/2, t = (h' - 224)/2, generalised to C_w, C_h and floored.
 *
 * Readings where the paper is silent (interpolation convention, rounding of the
 * long side, colour matrix, fp16 rounding) are fixed as follows:
 *   - resized long side: floor(S * long / short), exact integer arithmetic;
 *   - crop offsets: floor((W' - C_w)/2), floor((H' - C_h)/2);
 *   - bilinear with half-pixel centres (align_corners = false), clamped at the
 *     edges, no antialiasing; the source coordinate of output index x is the
 *     exact rational ((2x+1)*in - out) / (2*out); its integer part is taken
 *     exactly and only the fractional weight is rounded, once, to fp32;
 *   - interpolation in fp32 in the lerp form a + w*(b - a), horizontal first,
 *     every operation rounded on its own (build with -ffp-contract=off);
 *   - normalisation (v - mean_c) / std_c in fp32 with mean and std in 0..255
 *     units;
 *   - fp16 output rounds to nearest, ties to even, written out below from the
 *     IEEE-754 binary16 format;
 *   - YCbCr: BT.601 full range (JFIF) with centred 4:2:0 chroma siting; the
 *     chroma sample that serves luma pixel x sits at x/2 - 1/4; each channel is
 *     clamped to [0, 255] in fp32 (no integer rounding) at every luma pixel,
 *     before the resize.
 *
 * Variants (the "_ex" calls), each a reading of a passage the paper leaves
 * open:
 *   - region of interest: the paper's partial-decoding discussion (section
 *     6.4, "Leveraging partial decoding") lets a caller pass an ROI per image,
 *     e.g. a face or detection crop, and only the ROI is processed. The ROI
 *     (x, y, w, h) is cut out of the decoded image first and then treated as
 *     a w x h image: the resize taps clamp at the ROI's edges. For I420 the
 *     frame is converted to RGB first (chroma taps in frame coordinates,
 *     clamped at the frame's chroma planes), then the ROI is cut;
 *   - direct resize: the network's fixed input size (the section cites
 *     224 x 224) reached without keeping the aspect ratio: the image (or ROI)
 *     is resized to C_w x C_h and nothing is cropped;
 *   - channels-last (NHWC) output instead of step 4's channels-first;
 *   - left (co-sited) 4:2:0 chroma, as MPEG-2 / H.264 decoders emit: the
 *     chroma sample of luma column x sits at x/2 (rows stay centred).
 *
 * Low-resolution-aware augmentation (section 5.3, "Training DNNs for
 * Low-resolution Visual Data"): at training time the full-resolution input is
 * downsampled to the target resolution r and upsampled back to the network's
 * input size. Readings: the low-resolution image is what a stored
 * low-resolution copy would hold -- the standard step 2 geometry with S = r
 * and an r x r central crop, each resized value rounded to the nearest
 * integer (ties to even) as uint8 ("uint8 output", no normalisation) -- and
 * that r x r image then goes through steps 2-4 like any other image.
 *
 * Partial JPEG decoding (section 6.4, "ROI decoding", Algorithm 1) and, ahead
 * of it, baseline JPEG entropy decoding written from ITU-T T.81: their
 * readings sit with the functions at the end of this file.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORACLE_OUT_F32 = 0, ORACLE_OUT_F16 = 1, ORACLE_OUT_U8 = 2 };
enum { ORACLE_RESIZE_SHORT_CROP = 0, ORACLE_RESIZE_DIRECT = 1 };
enum { ORACLE_NCHW = 0, ORACLE_NHWC = 1 };
enum { ORACLE_CHROMA_CENTER = 0, ORACLE_CHROMA_LEFT = 1 };
enum { ORACLE_OK = 0, ORACLE_ERR = -1 };

/* ------------------------------------------------------------------------- */
/* Geometry                                                                   */
/* ------------------------------------------------------------------------- */

/* Section 2, step 2: aspect-preserving resize whose short edge becomes S. The
 * long side is floored. A square image becomes S x S. */
void oracle_resized_dims(int64_t W, int64_t H, int64_t S, int64_t *Wr, int64_t *Hr)
{
    if (W <= H) {
        *Wr = S;
        *Hr = (S * H) / W;
    } else {
        *Hr = S;
        *Wr = (S * W) / H;
    }
}

/* Algorithm 1: l, t = (w' - C_w)/2, (h' - C_h)/2, floored. */
void oracle_crop_offsets(int64_t Wr, int64_t Hr, int64_t Ch, int64_t Cw, int64_t *left,
                         int64_t *top)
{
    *left = (Wr - Cw) / 2;
    *top = (Hr - Ch) / 2;
}

/* One axis of the half-pixel bilinear map from an output index x (in the
 * resized image of length `out`) to the source (length `in`):
 *     u = (x + 1/2) * in / out - 1/2 = ((2x + 1) * in - out) / (2 * out).
 * u below 0 clamps to 0; u at or beyond in - 1 clamps to in - 1. The two taps
 * are floor(u) and floor(u) + 1 with weight u - floor(u) on the second. */
void oracle_axis_tap(int64_t x, int64_t in, int64_t out, int64_t *x0, int64_t *x1, float *w)
{
    int64_t num = (2 * x + 1) * in - out; /* 2*out times u */
    int64_t den = 2 * out;
    if (num <= 0) {
        *x0 = 0;
        *x1 = 0;
        *w = 0.0f;
        return;
    }
    int64_t q = num / den;
    int64_t rem = num - q * den;
    if (q >= in - 1) {
        *x0 = in - 1;
        *x1 = in - 1;
        *w = 0.0f;
        return;
    }
    *x0 = q;
    *x1 = q + 1;
    *w = (float)rem / (float)den; /* both operands exact in fp32 (< 2^24) */
}

/* ------------------------------------------------------------------------- */
/* Colour                                                                     */
/* ------------------------------------------------------------------------- */

/* BT.601 full-range (JFIF) YCbCr -> RGB with Kr = 0.299, Kb = 0.114:
 *   R = Y + 2(1-Kr) (Cr-128)
 *   G = Y - [2Kb(1-Kb)/Kg] (Cb-128) - [2Kr(1-Kr)/Kg] (Cr-128)
 *   B = Y + 2(1-Kb) (Cb-128)
 * Coefficients are derived in double and rounded once to fp32; the expressions
 * are evaluated left to right in fp32; each channel is clamped to [0, 255]. */
void oracle_ycbcr_to_rgb(float Y, float Cb, float Cr, float *rgb)
{
    const double kr = 0.299, kb = 0.114, kg = 1.0 - kr - kb;
    const float r_cr = (float)(2.0 * (1.0 - kr));
    const float g_cb = (float)(2.0 * kb * (1.0 - kb) / kg);
    const float g_cr = (float)(2.0 * kr * (1.0 - kr) / kg);
    const float b_cb = (float)(2.0 * (1.0 - kb));
    float cb = Cb - 128.0f;
    float cr = Cr - 128.0f;
    float r = Y + r_cr * cr;
    float g = Y - g_cb * cb;
    g = g - g_cr * cr;
    float b = Y + b_cb * cb;
    rgb[0] = r < 0.0f ? 0.0f : (r > 255.0f ? 255.0f : r);
    rgb[1] = g < 0.0f ? 0.0f : (g > 255.0f ? 255.0f : g);
    rgb[2] = b < 0.0f ? 0.0f : (b > 255.0f ? 255.0f : b);
}

/* Centred 4:2:0 siting: the chroma coordinate of luma index x is u = x/2 - 1/4
 * (exact in fp32 for the sizes allowed here). Same clamping as the luma map. */
static void chroma_tap(int64_t x, int64_t n, int64_t *c0, int64_t *c1, float *w)
{
    float u = (float)x * 0.5f - 0.25f;
    if (u <= 0.0f) {
        *c0 = 0;
        *c1 = 0;
        *w = 0.0f;
        return;
    }
    int64_t f = (int64_t)floorf(u);
    if (f >= n - 1) {
        *c0 = n - 1;
        *c1 = n - 1;
        *w = 0.0f;
        return;
    }
    *c0 = f;
    *c1 = f + 1;
    *w = u - (float)f;
}

/* Left (co-sited) siting, horizontal axis: the chroma coordinate of luma
 * column x is u = x/2. */
static void chroma_tap_left(int64_t x, int64_t n, int64_t *c0, int64_t *c1, float *w)
{
    float u = (float)x * 0.5f;
    int64_t f = (int64_t)floorf(u);
    if (f >= n - 1) {
        *c0 = n - 1;
        *c1 = n - 1;
        *w = 0.0f;
        return;
    }
    *c0 = f;
    *c1 = f + 1;
    *w = u - (float)f;
}

/* Planar I420 (Y: W x H, Cb and Cr: ceil(W/2) x ceil(H/2), tightly pitched)
 * to an fp32 RGB image, W x H x 3 interleaved: chroma is bilinearly upsampled
 * to every luma pixel, then converted and clamped there. */
void oracle_yuv420_to_rgb_sited(const uint8_t *yp, const uint8_t *cbp, const uint8_t *crp,
                                int64_t W, int64_t H, int32_t siting, float *rgb)
{
    int64_t Wc = (W + 1) / 2, Hc = (H + 1) / 2;
    for (int64_t y = 0; y < H; ++y) {
        int64_t r0, r1;
        float wy;
        chroma_tap(y, Hc, &r0, &r1, &wy);
        for (int64_t x = 0; x < W; ++x) {
            int64_t k0, k1;
            float wx;
            if (siting == ORACLE_CHROMA_LEFT)
                chroma_tap_left(x, Wc, &k0, &k1, &wx);
            else
                chroma_tap(x, Wc, &k0, &k1, &wx);
            float c[2];
            const uint8_t *planes[2] = {cbp, crp};
            for (int p = 0; p < 2; ++p) {
                const uint8_t *pl = planes[p];
                float a = (float)pl[r0 * Wc + k0], b = (float)pl[r0 * Wc + k1];
                float t = a + wx * (b - a);
                a = (float)pl[r1 * Wc + k0];
                b = (float)pl[r1 * Wc + k1];
                float bo = a + wx * (b - a);
                c[p] = t + wy * (bo - t);
            }
            oracle_ycbcr_to_rgb((float)yp[y * W + x], c[0], c[1], &rgb[(y * W + x) * 3]);
        }
    }
}

void oracle_yuv420_to_rgb(const uint8_t *yp, const uint8_t *cbp, const uint8_t *crp, int64_t W,
                          int64_t H, float *rgb)
{
    oracle_yuv420_to_rgb_sited(yp, cbp, crp, W, H, ORACLE_CHROMA_CENTER, rgb);
}

/* ------------------------------------------------------------------------- */
/* fp16 rounding                                                              */
/* ------------------------------------------------------------------------- */

/* IEEE-754 binary32 -> binary16, round to nearest, ties to even. */
uint16_t oracle_f32_to_f16(float f)
{
    uint32_t x;
    memcpy(&x, &f, 4);
    uint32_t sign = (x >> 16) & 0x8000u;
    uint32_t e = (x >> 23) & 0xffu;
    uint32_t m = x & 0x7fffffu;
    if (e == 0xffu) /* inf or nan (nan keeps a set quiet bit) */
        return (uint16_t)(sign | 0x7c00u | (m ? 0x200u | (m >> 13) : 0u));
    int32_t he = (int32_t)e - 127 + 15; /* biased binary16 exponent */
    if (he >= 31)                       /* too large even before rounding */
        return (uint16_t)(sign | 0x7c00u);
    if (he <= 0) {
        /* binary16 subnormal (or zero): value = sig * 2^(e-150), sig = 1.m
         * as a 24-bit integer; the result is sig * 2^(e-150) / 2^-24 =
         * sig >> (126 - e), rounded to nearest even. */
        if (he < -10) /* below half the smallest subnormal: rounds to zero */
            return (uint16_t)sign;
        uint32_t sig = m | 0x800000u;
        uint32_t shift = (uint32_t)(126 - (int32_t)e); /* 14 .. 24 */
        uint32_t q = sig >> shift;
        uint32_t rest = sig & ((1u << shift) - 1u);
        uint32_t half = 1u << (shift - 1);
        if (rest > half || (rest == half && (q & 1u)))
            q += 1u; /* may carry into the smallest normal: still correct */
        return (uint16_t)(sign | q);
    }
    uint32_t q = ((uint32_t)he << 10) | (m >> 13);
    uint32_t rest = m & 0x1fffu;
    if (rest > 0x1000u || (rest == 0x1000u && (q & 1u)))
        q += 1u; /* a carry into the exponent field is the correct result */
    return (uint16_t)(sign | q);
}

/* ------------------------------------------------------------------------- */
/* Resize + crop + normalise + NCHW store                                     */
/* ------------------------------------------------------------------------- */

/* Resized size and crop offsets of a W x H image: step 2's short-side resize
 * and central crop, or the direct resize to C_w x C_h (no crop). */
void oracle_output_geometry(int64_t W, int64_t H, int64_t S, int64_t Ch, int64_t Cw,
                            int32_t resize_mode, int64_t *Wr, int64_t *Hr, int64_t *left,
                            int64_t *top)
{
    if (resize_mode == ORACLE_RESIZE_DIRECT) {
        *Wr = Cw;
        *Hr = Ch;
        *left = 0;
        *top = 0;
        return;
    }
    oracle_resized_dims(W, H, S, Wr, Hr);
    oracle_crop_offsets(*Wr, *Hr, Ch, Cw, left, top);
}

/* A resized value v (in [0, 255]) as uint8: the nearest integer, ties to
 * even. v - floor(v) is exact in fp32, so the comparison with 1/2 decides. */
static uint8_t round_u8(float v)
{
    float f = floorf(v);
    float d = v - f;
    int64_t k = (int64_t)f;
    if (d > 0.5f || (d == 0.5f && (k & 1)))
        ++k;
    return (uint8_t)(k < 0 ? 0 : k > 255 ? 255 : k);
}

/* rgb: fp32 image, W x H x 3 interleaved (rows `rstride` floats apart).
 * out: 3 x Ch x Cw (NCHW) or Ch x Cw x 3 (NHWC) of the out dtype; uint8
 * output holds the resized values rounded, not normalised. */
static void resample_crop_normalize(const float *rgb, int64_t rstride, int64_t W, int64_t H,
                                    int64_t S, int64_t Ch, int64_t Cw, const float *mean,
                                    const float *stdv, int out_dtype, int32_t resize_mode,
                                    int32_t layout, void *out)
{
    int64_t Wr, Hr, left, top;
    oracle_output_geometry(W, H, S, Ch, Cw, resize_mode, &Wr, &Hr, &left, &top);
    for (int64_t yc = 0; yc < Ch; ++yc) {
        int64_t y0, y1;
        float wy;
        oracle_axis_tap(yc + top, H, Hr, &y0, &y1, &wy);
        for (int64_t xc = 0; xc < Cw; ++xc) {
            int64_t x0, x1;
            float wx;
            oracle_axis_tap(xc + left, W, Wr, &x0, &x1, &wx);
            for (int c = 0; c < 3; ++c) {
                float p00 = rgb[y0 * rstride + x0 * 3 + c];
                float p01 = rgb[y0 * rstride + x1 * 3 + c];
                float p10 = rgb[y1 * rstride + x0 * 3 + c];
                float p11 = rgb[y1 * rstride + x1 * 3 + c];
                float t = p00 + wx * (p01 - p00);
                float b = p10 + wx * (p11 - p10);
                float v = t + wy * (b - t);
                int64_t idx = layout == ORACLE_NHWC ? (yc * Cw + xc) * 3 + c
                                                    : ((int64_t)c * Ch + yc) * Cw + xc;
                if (out_dtype == ORACLE_OUT_U8) {
                    ((uint8_t *)out)[idx] = round_u8(v);
                    continue;
                }
                float o = (v - mean[c]) / stdv[c];
                if (out_dtype == ORACLE_OUT_F32)
                    ((float *)out)[idx] = o;
                else
                    ((uint16_t *)out)[idx] = oracle_f32_to_f16(o);
            }
        }
    }
}

static int params_ok_ex(int64_t W, int64_t H, int32_t S, int32_t Ch, int32_t Cw,
                        int32_t out_dtype, int32_t resize_mode, int32_t layout)
{
    if (W < 1 || H < 1 || S < 1 || Ch < 1 || Cw < 1)
        return 0;
    if (out_dtype != ORACLE_OUT_F32 && out_dtype != ORACLE_OUT_F16 && out_dtype != ORACLE_OUT_U8)
        return 0;
    if ((resize_mode != ORACLE_RESIZE_SHORT_CROP && resize_mode != ORACLE_RESIZE_DIRECT) ||
        (layout != ORACLE_NCHW && layout != ORACLE_NHWC))
        return 0;
    int64_t Wr, Hr, left, top;
    oracle_output_geometry(W, H, S, Ch, Cw, resize_mode, &Wr, &Hr, &left, &top);
    if (Ch > Hr || Cw > Wr) /* the crop must lie inside the resized image */
        return 0;
    /* the fp32 weight needs 2*out < 2^24 to be formed from exact operands */
    if (2 * Wr >= (1 << 24) || 2 * Hr >= (1 << 24))
        return 0;
    return 1;
}

/* A region of interest inside a W x H image. */
static int roi_ok(int64_t W, int64_t H, int32_t rx, int32_t ry, int32_t rw, int32_t rh)
{
    return rx >= 0 && ry >= 0 && rw >= 1 && rh >= 1 && rx + (int64_t)rw <= W &&
           ry + (int64_t)rh <= H;
}

/* One packed HWC RGB uint8 image (row pitch in bytes): the ROI (rx, ry, rw,
 * rh) cut out, resized, cropped, normalised, in the given layout. */
int smol_ref_preprocess_image_ex(const uint8_t *img, int32_t W, int32_t H, int32_t pitch,
                                 int32_t rx, int32_t ry, int32_t rw, int32_t rh, int32_t S,
                                 int32_t Ch, int32_t Cw, const float *mean, const float *stdv,
                                 int32_t out_dtype, int32_t resize_mode, int32_t layout,
                                 void *out)
{
    if (W < 1 || H < 1 || pitch < 3 * W || !roi_ok(W, H, rx, ry, rw, rh) ||
        !params_ok_ex(rw, rh, S, Ch, Cw, out_dtype, resize_mode, layout))
        return ORACLE_ERR;
    float *rgb = (float *)malloc((size_t)rw * (size_t)rh * 3 * sizeof(float));
    if (!rgb)
        return ORACLE_ERR;
    for (int64_t y = 0; y < rh; ++y)
        for (int64_t x = 0; x < 3 * (int64_t)rw; ++x)
            rgb[y * 3 * rw + x] = (float)img[(ry + y) * (int64_t)pitch + 3 * (int64_t)rx + x];
    resample_crop_normalize(rgb, 3 * (int64_t)rw, rw, rh, S, Ch, Cw, mean, stdv, out_dtype,
                            resize_mode, layout, out);
    free(rgb);
    return ORACLE_OK;
}

/* One packed HWC RGB uint8 image (row pitch in bytes) -> 3 x Ch x Cw. */
int smol_ref_preprocess_image(const uint8_t *img, int32_t W, int32_t H, int32_t pitch, int32_t S,
                              int32_t Ch, int32_t Cw, const float *mean, const float *stdv,
                              int32_t out_dtype, void *out)
{
    return smol_ref_preprocess_image_ex(img, W, H, pitch, 0, 0, W, H, S, Ch, Cw, mean, stdv,
                                        out_dtype, ORACLE_RESIZE_SHORT_CROP, ORACLE_NCHW, out);
}

/* One planar I420 frame: converted to RGB at every luma pixel (chroma sited
 * as given), the ROI cut out of that, then resized, cropped, normalised. */
int smol_ref_yuv420_preprocess_image_ex(const uint8_t *yp, const uint8_t *cbp,
                                        const uint8_t *crp, int32_t W, int32_t H, int32_t rx,
                                        int32_t ry, int32_t rw, int32_t rh, int32_t S, int32_t Ch,
                                        int32_t Cw, const float *mean, const float *stdv,
                                        int32_t out_dtype, int32_t resize_mode, int32_t layout,
                                        int32_t siting, void *out)
{
    if (W < 1 || H < 1 || !roi_ok(W, H, rx, ry, rw, rh) ||
        !params_ok_ex(rw, rh, S, Ch, Cw, out_dtype, resize_mode, layout) ||
        (siting != ORACLE_CHROMA_CENTER && siting != ORACLE_CHROMA_LEFT))
        return ORACLE_ERR;
    float *rgb = (float *)malloc((size_t)W * (size_t)H * 3 * sizeof(float));
    if (!rgb)
        return ORACLE_ERR;
    oracle_yuv420_to_rgb_sited(yp, cbp, crp, W, H, siting, rgb);
    resample_crop_normalize(rgb + ((int64_t)ry * W + rx) * 3, 3 * (int64_t)W, rw, rh, S, Ch, Cw,
                            mean, stdv, out_dtype, resize_mode, layout, out);
    free(rgb);
    return ORACLE_OK;
}

/* One planar I420 frame -> 3 x Ch x Cw. */
int smol_ref_yuv420_preprocess_image(const uint8_t *yp, const uint8_t *cbp, const uint8_t *crp,
                                     int32_t W, int32_t H, int32_t S, int32_t Ch, int32_t Cw,
                                     const float *mean, const float *stdv, int32_t out_dtype,
                                     void *out)
{
    return smol_ref_yuv420_preprocess_image_ex(yp, cbp, crp, W, H, 0, 0, W, H, S, Ch, Cw, mean,
                                               stdv, out_dtype, ORACLE_RESIZE_SHORT_CROP,
                                               ORACLE_NCHW, ORACLE_CHROMA_CENTER, out);
}

static size_t out_image_bytes(int32_t Ch, int32_t Cw, int32_t out_dtype)
{
    return (size_t)3 * (size_t)Ch * (size_t)Cw *
           (out_dtype == ORACLE_OUT_F32 ? 4u : out_dtype == ORACLE_OUT_F16 ? 2u : 1u);
}

/* Batch of packed HWC RGB images with an optional ROI table (rois: n x
 * {x, y, w, h}, or NULL for whole images). */
int smol_ref_preprocess_batch_ex(const uint8_t *src, int64_t src_bytes, const int64_t *offsets,
                                 const int32_t *widths, const int32_t *heights,
                                 const int32_t *pitches, const int32_t *rois, int32_t n,
                                 int32_t S, int32_t Ch, int32_t Cw, const float *mean,
                                 const float *stdv, int32_t out_dtype, int32_t resize_mode,
                                 int32_t layout, void *out)
{
    size_t ob = out_image_bytes(Ch, Cw, out_dtype);
    for (int32_t i = 0; i < n; ++i) {
        int32_t pitch = pitches ? pitches[i] : 3 * widths[i];
        int64_t end = offsets[i] + (int64_t)(heights[i] - 1) * pitch + 3 * (int64_t)widths[i];
        if (offsets[i] < 0 || end > src_bytes)
            return ORACLE_ERR;
        const int32_t *r = rois ? rois + 4 * (size_t)i : NULL;
        int rc = smol_ref_preprocess_image_ex(src + offsets[i], widths[i], heights[i], pitch,
                                              r ? r[0] : 0, r ? r[1] : 0, r ? r[2] : widths[i],
                                              r ? r[3] : heights[i], S, Ch, Cw, mean, stdv,
                                              out_dtype, resize_mode, layout,
                                              (uint8_t *)out + ob * i);
        if (rc)
            return rc;
    }
    return ORACLE_OK;
}

/* Batch of planar I420 frames with per-frame plane offsets and an optional
 * ROI table. */
int smol_ref_yuv420_preprocess_batch_ex(const uint8_t *src, int64_t src_bytes,
                                        const int64_t *y_offsets, const int64_t *cb_offsets,
                                        const int64_t *cr_offsets, const int32_t *widths,
                                        const int32_t *heights, const int32_t *rois, int32_t n,
                                        int32_t S, int32_t Ch, int32_t Cw, const float *mean,
                                        const float *stdv, int32_t out_dtype,
                                        int32_t resize_mode, int32_t layout, int32_t siting,
                                        void *out)
{
    size_t ob = out_image_bytes(Ch, Cw, out_dtype);
    for (int32_t i = 0; i < n; ++i) {
        int64_t W = widths[i], H = heights[i];
        int64_t Wc = (W + 1) / 2, Hc = (H + 1) / 2;
        if (y_offsets[i] < 0 || y_offsets[i] + W * H > src_bytes || cb_offsets[i] < 0 ||
            cb_offsets[i] + Wc * Hc > src_bytes || cr_offsets[i] < 0 ||
            cr_offsets[i] + Wc * Hc > src_bytes)
            return ORACLE_ERR;
        const int32_t *r = rois ? rois + 4 * (size_t)i : NULL;
        int rc = smol_ref_yuv420_preprocess_image_ex(
            src + y_offsets[i], src + cb_offsets[i], src + cr_offsets[i], widths[i], heights[i],
            r ? r[0] : 0, r ? r[1] : 0, r ? r[2] : widths[i], r ? r[3] : heights[i], S, Ch, Cw,
            mean, stdv, out_dtype, resize_mode, layout, siting, (uint8_t *)out + ob * i);
        if (rc)
            return rc;
    }
    return ORACLE_OK;
}

/* Batch of packed HWC RGB images; image i starts at src + offsets[i] and has
 * widths[i] x heights[i] pixels with row pitch pitches[i] bytes (NULL: 3W).
 * out holds n x 3 x Ch x Cw elements. */
int smol_ref_preprocess_batch(const uint8_t *src, int64_t src_bytes, const int64_t *offsets,
                              const int32_t *widths, const int32_t *heights,
                              const int32_t *pitches, int32_t n, int32_t S, int32_t Ch, int32_t Cw,
                              const float *mean, const float *stdv, int32_t out_dtype, void *out)
{
    size_t ob = out_image_bytes(Ch, Cw, out_dtype);
    for (int32_t i = 0; i < n; ++i) {
        int32_t pitch = pitches ? pitches[i] : 3 * widths[i];
        int64_t end = offsets[i] + (int64_t)(heights[i] - 1) * pitch + 3 * (int64_t)widths[i];
        if (offsets[i] < 0 || end > src_bytes)
            return ORACLE_ERR;
        int rc = smol_ref_preprocess_image(src + offsets[i], widths[i], heights[i], pitch, S, Ch,
                                           Cw, mean, stdv, out_dtype, (uint8_t *)out + ob * i);
        if (rc)
            return rc;
    }
    return ORACLE_OK;
}

/* Batch of planar I420 frames with per-frame plane offsets. */
int smol_ref_yuv420_preprocess_batch(const uint8_t *src, int64_t src_bytes,
                                     const int64_t *y_offsets, const int64_t *cb_offsets,
                                     const int64_t *cr_offsets, const int32_t *widths,
                                     const int32_t *heights, int32_t n, int32_t S, int32_t Ch,
                                     int32_t Cw, const float *mean, const float *stdv,
                                     int32_t out_dtype, void *out)
{
    size_t ob = out_image_bytes(Ch, Cw, out_dtype);
    for (int32_t i = 0; i < n; ++i) {
        int64_t W = widths[i], H = heights[i];
        int64_t Wc = (W + 1) / 2, Hc = (H + 1) / 2;
        if (y_offsets[i] < 0 || y_offsets[i] + W * H > src_bytes || cb_offsets[i] < 0 ||
            cb_offsets[i] + Wc * Hc > src_bytes || cr_offsets[i] < 0 ||
            cr_offsets[i] + Wc * Hc > src_bytes)
            return ORACLE_ERR;
        int rc = smol_ref_yuv420_preprocess_image(src + y_offsets[i], src + cb_offsets[i],
                                                  src + cr_offsets[i], widths[i], heights[i], S,
                                                  Ch, Cw, mean, stdv, out_dtype,
                                                  (uint8_t *)out + ob * i);
        if (rc)
            return rc;
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------- */
/* Low-resolution-aware augmentation (section 5.3)                           */
/* ------------------------------------------------------------------------- */

/* One packed HWC RGB image: reduced to the r x r uint8 image (short side r,
 * central r x r crop, rounded), which then goes through steps 2-4. */
int smol_ref_lowres_preprocess_image(const uint8_t *img, int32_t W, int32_t H, int32_t pitch,
                                     int32_t r, int32_t S, int32_t Ch, int32_t Cw,
                                     const float *mean, const float *stdv, int32_t out_dtype,
                                     void *out)
{
    if (r < 1 || out_dtype == ORACLE_OUT_U8)
        return ORACLE_ERR;
    uint8_t *low = (uint8_t *)malloc((size_t)r * (size_t)r * 3);
    if (!low)
        return ORACLE_ERR;
    int rc = smol_ref_preprocess_image_ex(img, W, H, pitch, 0, 0, W, H, r, r, r, mean, stdv,
                                          ORACLE_OUT_U8, ORACLE_RESIZE_SHORT_CROP, ORACLE_NHWC,
                                          low);
    if (rc == ORACLE_OK)
        rc = smol_ref_preprocess_image(low, r, r, 3 * r, S, Ch, Cw, mean, stdv, out_dtype, out);
    free(low);
    return rc;
}

/* One planar I420 frame: converted (centred chroma) and reduced to the r x r
 * uint8 RGB image, which then goes through steps 2-4. */
int smol_ref_yuv420_lowres_preprocess_image(const uint8_t *yp, const uint8_t *cbp,
                                            const uint8_t *crp, int32_t W, int32_t H, int32_t r,
                                            int32_t S, int32_t Ch, int32_t Cw, const float *mean,
                                            const float *stdv, int32_t out_dtype, void *out)
{
    if (r < 1 || out_dtype == ORACLE_OUT_U8)
        return ORACLE_ERR;
    uint8_t *low = (uint8_t *)malloc((size_t)r * (size_t)r * 3);
    if (!low)
        return ORACLE_ERR;
    int rc = smol_ref_yuv420_preprocess_image_ex(yp, cbp, crp, W, H, 0, 0, W, H, r, r, r, mean,
                                                 stdv, ORACLE_OUT_U8, ORACLE_RESIZE_SHORT_CROP,
                                                 ORACLE_NHWC, ORACLE_CHROMA_CENTER, low);
    if (rc == ORACLE_OK)
        rc = smol_ref_preprocess_image(low, r, r, 3 * r, S, Ch, Cw, mean, stdv, out_dtype, out);
    free(low);
    return rc;
}

/* Batch forms (tables as in smol_ref_preprocess_batch and
 * smol_ref_yuv420_preprocess_batch). */
int smol_ref_lowres_preprocess_batch(const uint8_t *src, int64_t src_bytes,
                                     const int64_t *offsets, const int32_t *widths,
                                     const int32_t *heights, const int32_t *pitches, int32_t n,
                                     int32_t r, int32_t S, int32_t Ch, int32_t Cw,
                                     const float *mean, const float *stdv, int32_t out_dtype,
                                     void *out)
{
    size_t ob = out_image_bytes(Ch, Cw, out_dtype);
    for (int32_t i = 0; i < n; ++i) {
        int32_t pitch = pitches ? pitches[i] : 3 * widths[i];
        int64_t end = offsets[i] + (int64_t)(heights[i] - 1) * pitch + 3 * (int64_t)widths[i];
        if (offsets[i] < 0 || end > src_bytes)
            return ORACLE_ERR;
        int rc = smol_ref_lowres_preprocess_image(src + offsets[i], widths[i], heights[i], pitch,
                                                  r, S, Ch, Cw, mean, stdv, out_dtype,
                                                  (uint8_t *)out + ob * i);
        if (rc)
            return rc;
    }
    return ORACLE_OK;
}

int smol_ref_yuv420_lowres_preprocess_batch(const uint8_t *src, int64_t src_bytes,
                                            const int64_t *y_offsets, const int64_t *cb_offsets,
                                            const int64_t *cr_offsets, const int32_t *widths,
                                            const int32_t *heights, int32_t n, int32_t r,
                                            int32_t S, int32_t Ch, int32_t Cw, const float *mean,
                                            const float *stdv, int32_t out_dtype, void *out)
{
    size_t ob = out_image_bytes(Ch, Cw, out_dtype);
    for (int32_t i = 0; i < n; ++i) {
        int64_t W = widths[i], H = heights[i];
        int64_t Wc = (W + 1) / 2, Hc = (H + 1) / 2;
        if (y_offsets[i] < 0 || y_offsets[i] + W * H > src_bytes || cb_offsets[i] < 0 ||
            cb_offsets[i] + Wc * Hc > src_bytes || cr_offsets[i] < 0 ||
            cr_offsets[i] + Wc * Hc > src_bytes)
            return ORACLE_ERR;
        int rc = smol_ref_yuv420_lowres_preprocess_image(
            src + y_offsets[i], src + cb_offsets[i], src + cr_offsets[i], widths[i], heights[i],
            r, S, Ch, Cw, mean, stdv, out_dtype, (uint8_t *)out + ob * i);
        if (rc)
            return rc;
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------- */
/* Partial JPEG decoding (section 6.4, "ROI decoding", Algorithm 1)          */
/* ------------------------------------------------------------------------- */
/*
 * Readings (none of this is fixed by the paper, which relies on a decoder
 * library):
 *   - the decoder's output is baseline JPEG 4:2:0: 16 x 16 luma MCUs, each
 *     holding four luma and one Cb and one Cr 8 x 8 block; the entropy
 *     decoding (Huffman, zig-zag) happens on the CPU and is not modelled:
 *     the input is the dequantisation's input, int16 coefficients per block
 *     in natural order (row v = vertical frequency, column u), blocks in
 *     raster order over the MCU-padded frame, luma then Cb then Cr;
 *   - dequantisation multiplies by the table entry; the inverse DCT is
 *     ITU-T T.81's A.3.3 formula, evaluated in fp32 as two 1-D passes
 *     (horizontal frequencies first). T.81 fixes the real value only; each
 *     1-D sum x[n] = sum_k c[k][n] d[k] is evaluated through the parity of
 *     the cosine basis, c[k][7-n] = (-1)^k c[k][n] (an identity of the
 *     formula): for n = 0..3, E = c[0][n] d[0] + c[2][n] d[2] + c[4][n] d[4]
 *     + c[6][n] d[6] and O = c[1][n] d[1] + c[3][n] d[3] + c[5][n] d[5]
 *     + c[7][n] d[7], each summed in increasing frequency, then
 *     x[n] = E + O and x[7-n] = E - O; every product and sum is rounded on
 *     its own, and the table c[k][n] = C(k)/2 cos((2n+1) k pi / 16)
 *     (C(0) = 1/sqrt(2), else 1) for n = 0..3 is formed in double and
 *     rounded once to fp32; then + 128, rounded to nearest (ties to even)
 *     and clamped to 0..255;
 *   - Algorithm 1's rectangle: the smallest MCU-aligned rectangle holding
 *     every luma and chroma sample the resize taps read (the algorithm's
 *     scale = min(h, w) / 224 is replaced by the exact tap footprint, as for
 *     the crop itself), clipped to the frame.
 */

static void jpeg_idct_table(float c[64])
{
    const double pi = 3.14159265358979323846;
    for (int k = 0; k < 8; ++k)
        for (int n = 0; n < 8; ++n) {
            double ck = k == 0 ? 1.0 / sqrt(2.0) : 1.0;
            c[k * 8 + n] = (float)(ck / 2.0 * cos((2.0 * n + 1.0) * k * pi / 16.0));
        }
}

/* One 1-D inverse transform of the 8 values in[0], in[st], ..., in[7 st]
 * into out[0], out[st], ...: the sum over k of c[k][n] in[k] for each n,
 * through the parity identity (see the readings above). */
static void idct_1d(const float c[64], const float *in, float *out, int st)
{
    for (int n = 0; n < 4; ++n) {
        float e = c[0 * 8 + n] * in[0 * st];
        e = e + c[2 * 8 + n] * in[2 * st];
        e = e + c[4 * 8 + n] * in[4 * st];
        e = e + c[6 * 8 + n] * in[6 * st];
        float o = c[1 * 8 + n] * in[1 * st];
        o = o + c[3 * 8 + n] * in[3 * st];
        o = o + c[5 * 8 + n] * in[5 * st];
        o = o + c[7 * 8 + n] * in[7 * st];
        out[n * st] = e + o;
        out[(7 - n) * st] = e - o;
    }
}

/* One block: coef[v*8+u] times q[v*8+u], inverse DCT, level shift, round,
 * clamp; the w x h top-left pixels (w, h <= 8) are written to out (row
 * pitch `pitch` bytes). */
void oracle_idct_block(const int16_t *coef, const uint16_t *q, uint8_t *out, int64_t pitch,
                       int32_t w, int32_t h)
{
    float c[64], d[64], g[64], f[64];
    jpeg_idct_table(c);
    for (int i = 0; i < 64; ++i)
        d[i] = (float)((int32_t)coef[i] * (int32_t)q[i]); /* exact: |.| < 2^24 */
    for (int v = 0; v < 8; ++v) /* horizontal pass: row v of frequencies */
        idct_1d(c, d + v * 8, g + v * 8, 1);
    for (int x = 0; x < 8; ++x) /* vertical pass: column x */
        idct_1d(c, g + x, f + x, 8);
    for (int y = 0; y < h; ++y)
        for (int x = 0; x < w; ++x)
            out[y * pitch + x] = round_u8(f[y * 8 + x] + 128.0f);
}

/* Blocks of the MCU-padded frame: luma bw x bh, chroma bw/2 x bh/2 each. */
static void jpeg_grid(int64_t W, int64_t H, int64_t *bw, int64_t *bh)
{
    *bw = 2 * ((W + 15) / 16);
    *bh = 2 * ((H + 15) / 16);
}

/* Coefficients (int16 elements) of one frame. */
int64_t oracle_jpeg_coef_count(int32_t W, int32_t H)
{
    int64_t bw, bh;
    jpeg_grid(W, H, &bw, &bh);
    return 64 * (bw * bh + 2 * (bw / 2) * (bh / 2));
}

/* The MCU-aligned rectangle (x, y, w, h in luma pixels) holding every sample
 * the resize of a W x H I420 frame reads (centred chroma), for the short-side
 * crop or direct resize of `mode`. */
int oracle_jpeg_mcu_rect(int32_t W, int32_t H, int32_t S, int32_t Ch, int32_t Cw, int32_t mode,
                         int32_t *rect)
{
    if (!params_ok_ex(W, H, S, Ch, Cw, ORACLE_OUT_F32, mode, ORACLE_NCHW))
        return ORACLE_ERR;
    int64_t Wr, Hr, left, top, a, b, xf, xl, yf, yl, c0, c1, d0, d1;
    float w;
    oracle_output_geometry(W, H, S, Ch, Cw, mode, &Wr, &Hr, &left, &top);
    oracle_axis_tap(left, W, Wr, &xf, &a, &w);
    oracle_axis_tap(left + Cw - 1, W, Wr, &b, &xl, &w);
    oracle_axis_tap(top, H, Hr, &yf, &a, &w);
    oracle_axis_tap(top + Ch - 1, H, Hr, &b, &yl, &w);
    /* chroma samples of the first and last luma columns / rows, in luma units */
    chroma_tap(xf, (W + 1) / 2, &c0, &a, &w);
    chroma_tap(xl, (W + 1) / 2, &b, &c1, &w);
    chroma_tap(yf, (H + 1) / 2, &d0, &a, &w);
    chroma_tap(yl, (H + 1) / 2, &b, &d1, &w);
    int64_t x0 = xf < 2 * c0 ? xf : 2 * c0, x1 = xl > 2 * c1 + 1 ? xl : 2 * c1 + 1;
    int64_t y0 = yf < 2 * d0 ? yf : 2 * d0, y1 = yl > 2 * d1 + 1 ? yl : 2 * d1 + 1;
    x0 = x0 / 16 * 16;
    y0 = y0 / 16 * 16;
    x1 = (x1 / 16 + 1) * 16;
    y1 = (y1 / 16 + 1) * 16;
    rect[0] = (int32_t)x0;
    rect[1] = (int32_t)y0;
    rect[2] = (int32_t)((x1 < W ? x1 : W) - x0);
    rect[3] = (int32_t)((y1 < H ? y1 : H) - y0);
    return ORACLE_OK;
}

/* Decode the blocks of a W x H frame that meet `rect` (x, y, w, h; NULL: the
 * whole frame) into full-size I420 planes (Y W x H, Cb and Cr ceil(W/2) x
 * ceil(H/2), tightly pitched); pixels of other blocks are left untouched. */
int oracle_jpeg_decode_i420(const int16_t *coef, const uint16_t *qy, const uint16_t *qc,
                            int32_t W, int32_t H, const int32_t *rect, uint8_t *yp, uint8_t *cbp,
                            uint8_t *crp)
{
    if (W < 1 || H < 1)
        return ORACLE_ERR;
    int64_t bw, bh;
    jpeg_grid(W, H, &bw, &bh);
    int64_t rx = rect ? rect[0] : 0, ry = rect ? rect[1] : 0;
    int64_t rw = rect ? rect[2] : W, rh = rect ? rect[3] : H;
    if (rx < 0 || ry < 0 || rw < 1 || rh < 1 || rx + rw > W || ry + rh > H)
        return ORACLE_ERR;
    const int64_t Wc = (W + 1) / 2, Hc = (H + 1) / 2;
    /* luma blocks */
    for (int64_t by = ry / 8; by <= (ry + rh - 1) / 8; ++by)
        for (int64_t bx = rx / 8; bx <= (rx + rw - 1) / 8; ++bx) {
            int32_t w = (int32_t)(W - 8 * bx < 8 ? W - 8 * bx : 8);
            int32_t h = (int32_t)(H - 8 * by < 8 ? H - 8 * by : 8);
            oracle_idct_block(coef + 64 * (by * bw + bx), qy, yp + 8 * by * W + 8 * bx, W, w, h);
        }
    /* chroma blocks: the chroma samples of the rectangle's luma columns */
    const int64_t cx0 = rx / 2, cx1 = (rx + rw - 1) / 2, cy0 = ry / 2, cy1 = (ry + rh - 1) / 2;
    const int16_t *cb = coef + 64 * bw * bh, *cr = cb + 64 * (bw / 2) * (bh / 2);
    for (int64_t by = cy0 / 8; by <= cy1 / 8; ++by)
        for (int64_t bx = cx0 / 8; bx <= cx1 / 8; ++bx) {
            int32_t w = (int32_t)(Wc - 8 * bx < 8 ? Wc - 8 * bx : 8);
            int32_t h = (int32_t)(Hc - 8 * by < 8 ? Hc - 8 * by : 8);
            int64_t k = by * (bw / 2) + bx;
            oracle_idct_block(cb + 64 * k, qc, cbp + 8 * by * Wc + 8 * bx, Wc, w, h);
            oracle_idct_block(cr + 64 * k, qc, crp + 8 * by * Wc + 8 * bx, Wc, w, h);
        }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------- */
/* Baseline JPEG entropy decoding (the CPU step ahead of section 6.4's       */
/* partial decode), written from ITU-T T.81                                  */
/* ------------------------------------------------------------------------- */
/*
 * The whole scan is decoded, always: a partial decode must produce the same
 * coefficients for every block it keeps. Accepted streams: baseline (SOF0)
 * or extended (SOF1) Huffman coding, 8-bit samples, three components with
 * sampling factors 2x2, 1x1, 1x1 (4:2:0), Cb and Cr on one quantisation
 * table, 8-bit table entries, one interleaved scan with Ss = 0, Se = 63,
 * Ah = Al = 0, and optional restart intervals (DRI). The output is this
 * library's coefficient layout: per block 64 values in natural order
 * (row = vertical frequency), luma blocks in raster order over the
 * MCU-padded frame, then Cb, then Cr.
 */

/* Zig-zag order (T.81 Figure A.6): zz_pos[k] = row * 8 + column of the k-th
 * coefficient, generated by walking the anti-diagonals d = row + column in
 * turn, upwards (row falling) on even d and downwards on odd d. */
static void zigzag_positions(int zz_pos[64])
{
    int k = 0;
    for (int d = 0; d < 15; ++d)
        for (int i = 0; i < 8; ++i) {
            int row = (d % 2 == 0) ? d - i : i;
            int col = d - row;
            if (row >= 0 && row < 8 && col >= 0 && col < 8)
                zz_pos[k++] = row * 8 + col;
        }
}

/* A Huffman table in T.81's decoder form (C.1, C.2 and F.2.2.3, Figure F.15):
 * for each code length l, the largest code MAXCODE[l] (-1: none), the
 * smallest MINCODE[l] and the index VALPTR[l] of its first value in HUFFVAL. */
typedef struct {
    int present;
    int32_t maxcode[18], mincode[17], valptr[17];
    uint8_t huffval[256];
} jpeg_huff;

static int huff_build(jpeg_huff *t, const uint8_t bits[16], const uint8_t *vals, int nvals)
{
    /* C.1: HUFFSIZE lists the code lengths in order; C.2: HUFFCODE the codes */
    int huffsize[257], huffcode[257], k = 0;
    for (int l = 1; l <= 16; ++l)
        for (int i = 0; i < bits[l - 1]; ++i)
            huffsize[k++] = l;
    huffsize[k] = 0;
    if (k != nvals || k > 256)
        return 0;
    int code = 0, si = huffsize[0];
    for (int p = 0; p < k;) {
        while (p < k && huffsize[p] == si)
            huffcode[p++] = code++;
        if ((long)code > (1L << si))
            return 0; /* lengths that do not form a prefix code */
        code <<= 1;
        ++si;
    }
    /* F.15 */
    int j = 0;
    for (int l = 1; l <= 16; ++l) {
        if (bits[l - 1] == 0) {
            t->maxcode[l] = -1;
            continue;
        }
        t->valptr[l] = j;
        t->mincode[l] = huffcode[j];
        j += bits[l - 1];
        t->maxcode[l] = huffcode[j - 1];
    }
    t->maxcode[17] = 0x7fffffff;
    memcpy(t->huffval, vals, (size_t)nvals);
    t->present = 1;
    return 1;
}

/* The entropy-coded segment as a bit source: NEXTBIT of F.2.2.5 (Figure
 * F.18) with the stuffed zero byte after 0xFF removed; a marker ends the
 * bits (reading past it is an error). */
typedef struct {
    const uint8_t *d;
    int64_t n, pos;
    int cnt, b, bad;
} jpeg_bits;

static int next_bit(jpeg_bits *s)
{
    if (s->cnt == 0) {
        if (s->pos >= s->n) {
            s->bad = 1;
            return 0;
        }
        s->b = s->d[s->pos++];
        s->cnt = 8;
        if (s->b == 0xFF) {
            if (s->pos >= s->n || s->d[s->pos] != 0x00) {
                s->bad = 1; /* a marker inside the data */
                return 0;
            }
            ++s->pos;
        }
    }
    --s->cnt;
    return (s->b >> s->cnt) & 1;
}

/* DECODE (Figure F.16) */
static int huff_decode(jpeg_bits *s, const jpeg_huff *t)
{
    int32_t code = next_bit(s);
    int l = 1;
    while (code > t->maxcode[l]) {
        if (l == 16) {
            s->bad = 1;
            return 0;
        }
        code = (code << 1) | next_bit(s);
        ++l;
    }
    return t->huffval[t->valptr[l] + code - t->mincode[l]];
}

/* RECEIVE (Figure F.17) followed by EXTEND (Figure F.12) */
static int32_t receive_extend(jpeg_bits *s, int ssss)
{
    int32_t v = 0;
    for (int i = 0; i < ssss; ++i)
        v = (v << 1) | next_bit(s);
    if (ssss > 0 && v < (1 << (ssss - 1)))
        v -= (1 << ssss) - 1;
    return v;
}

static int be16(const uint8_t *p) { return (p[0] << 8) | p[1]; }

/* Decode a whole baseline 4:2:0 JPEG stream: coefficients into coef
 * (oracle_jpeg_coef_count(W, H) elements), tables in natural order into
 * qy and qc (uint16[64] each), size into *W and *H. coef_elems bounds
 * coef; pass coef = NULL to read only the headers (size and tables). */
int oracle_jpeg_entropy_decode(const uint8_t *d, int64_t n, int16_t *coef, int64_t coef_elems,
                               uint16_t *qy, uint16_t *qc, int32_t *Wout, int32_t *Hout)
{
    int zz_pos[64];
    zigzag_positions(zz_pos);
    uint16_t qt[4][64];
    int qt_present[4] = {0, 0, 0, 0};
    jpeg_huff dc[4], ac[4];
    memset(dc, 0, sizeof dc);
    memset(ac, 0, sizeof ac);
    int W = 0, H = 0, comp_id[3] = {0, 0, 0}, comp_q[3] = {0, 0, 0}, have_sof = 0;
    int64_t restart = 0;
    if (n < 4 || d[0] != 0xFF || d[1] != 0xD8)
        return ORACLE_ERR;
    int64_t p = 2;
    for (;;) {
        if (p + 4 > n || d[p] != 0xFF)
            return ORACLE_ERR;
        while (p < n && d[p] == 0xFF) /* fill bytes before a marker */
            ++p;
        if (p + 3 > n)
            return ORACLE_ERR;
        const int m = d[p++];
        if (m == 0xD9 || m == 0xD8 || (m >= 0xD0 && m <= 0xD7) || m == 0x01)
            return ORACLE_ERR; /* EOI, SOI or RST before the scan */
        const int len = be16(d + p);
        if (len < 2 || p + len > n)
            return ORACLE_ERR;
        const uint8_t *s = d + p + 2;
        const int64_t seg_end = p + len;
        if (m == 0xDB) { /* DQT */
            int64_t q = p + 2;
            while (q < seg_end) {
                const int pq = d[q] >> 4, tq = d[q] & 15;
                if (pq != 0 || tq > 3 || q + 65 > seg_end)
                    return ORACLE_ERR; /* 16-bit tables are not accepted */
                for (int k = 0; k < 64; ++k)
                    qt[tq][zz_pos[k]] = d[q + 1 + k];
                qt_present[tq] = 1;
                q += 65;
            }
        } else if (m == 0xC4) { /* DHT */
            int64_t q = p + 2;
            while (q < seg_end) {
                if (q + 17 > seg_end)
                    return ORACLE_ERR;
                const int tc = d[q] >> 4, th = d[q] & 15;
                int total = 0;
                for (int i = 0; i < 16; ++i)
                    total += d[q + 1 + i];
                if (tc > 1 || th > 3 || q + 17 + total > seg_end)
                    return ORACLE_ERR;
                if (!huff_build(tc == 0 ? &dc[th] : &ac[th], d + q + 1, d + q + 17, total))
                    return ORACLE_ERR;
                q += 17 + total;
            }
        } else if (m == 0xDD) { /* DRI */
            if (len != 4)
                return ORACLE_ERR;
            restart = be16(s);
        } else if (m == 0xC0 || m == 0xC1) { /* SOF0, SOF1 */
            if (len != 17 || s[0] != 8 || s[5] != 3)
                return ORACLE_ERR;
            H = be16(s + 1);
            W = be16(s + 3);
            const int want[3] = {0x22, 0x11, 0x11};
            for (int c = 0; c < 3; ++c) {
                comp_id[c] = s[6 + 3 * c];
                if (s[7 + 3 * c] != want[c] || s[8 + 3 * c] > 3)
                    return ORACLE_ERR;
                comp_q[c] = s[8 + 3 * c];
            }
            if (W < 1 || H < 1 || comp_q[1] != comp_q[2])
                return ORACLE_ERR;
            have_sof = 1;
        } else if (m >= 0xC2 && m <= 0xCF && m != 0xC4 && m != 0xC8 && m != 0xCC) {
            return ORACLE_ERR; /* progressive, lossless, hierarchical, arithmetic */
        } else if (m == 0xDA) { /* SOS */
            if (!have_sof || !qt_present[comp_q[0]] || !qt_present[comp_q[1]])
                return ORACLE_ERR;
            if (len != 12 || s[0] != 3 || s[7] != 0 || s[8] != 63 || s[9] != 0)
                return ORACLE_ERR;
            int td[3], ta[3];
            for (int c = 0; c < 3; ++c) {
                if (s[1 + 2 * c] != comp_id[c])
                    return ORACLE_ERR; /* components in frame order */
                td[c] = s[2 + 2 * c] >> 4;
                ta[c] = s[2 + 2 * c] & 15;
                if (td[c] > 3 || ta[c] > 3 || !dc[td[c]].present || !ac[ta[c]].present)
                    return ORACLE_ERR;
            }
            for (int k = 0; k < 64; ++k) {
                qy[k] = qt[comp_q[0]][k];
                qc[k] = qt[comp_q[1]][k];
            }
            *Wout = W;
            *Hout = H;
            if (!coef)
                return ORACLE_OK;
            if (coef_elems < oracle_jpeg_coef_count(W, H))
                return ORACLE_ERR;
            int64_t bw, bh;
            jpeg_grid(W, H, &bw, &bh);
            const int64_t mcux = bw / 2, mcuy = bh / 2, mcus = mcux * mcuy;
            int16_t *plane[3] = {coef, coef + 64 * bw * bh, coef + 64 * bw * bh + 64 * mcus};
            jpeg_bits bs = {d, n, seg_end, 0, 0, 0};
            int32_t pred[3] = {0, 0, 0};
            for (int64_t mcu = 0; mcu < mcus; ++mcu) {
                if (restart > 0 && mcu > 0 && mcu % restart == 0) {
                    /* the interval ends: skip the remaining bits of the byte,
                     * then expect RST((mcu / restart - 1) mod 8) */
                    bs.cnt = 0;
                    const int64_t want_rst = 0xD0 + (mcu / restart - 1) % 8;
                    if (bs.pos + 2 > n || d[bs.pos] != 0xFF || d[bs.pos + 1] != want_rst)
                        return ORACLE_ERR;
                    bs.pos += 2;
                    pred[0] = pred[1] = pred[2] = 0;
                }
                const int64_t my = mcu / mcux, mx = mcu % mcux;
                /* four luma blocks (left to right, top to bottom), Cb, Cr */
                for (int b = 0; b < 6; ++b) {
                    const int c = b < 4 ? 0 : b - 3;
                    int64_t blk;
                    if (c == 0)
                        blk = (2 * my + b / 2) * bw + 2 * mx + b % 2;
                    else
                        blk = mcu;
                    int16_t *z = plane[c] + 64 * blk;
                    memset(z, 0, 64 * sizeof(int16_t));
                    /* F.2.2.1: DC difference */
                    const int t = huff_decode(&bs, &dc[td[c]]);
                    if (t > 11)
                        return ORACLE_ERR;
                    pred[c] += receive_extend(&bs, t);
                    if (pred[c] < -32768 || pred[c] > 32767)
                        return ORACLE_ERR;
                    z[0] = (int16_t)pred[c];
                    /* F.2.2.2 (Figure F.13): AC coefficients */
                    for (int k = 1; k < 64;) {
                        const int rs = huff_decode(&bs, &ac[ta[c]]);
                        const int ssss = rs & 15, rrrr = rs >> 4;
                        if (ssss == 0) {
                            if (rrrr != 15)
                                break; /* end of block */
                            k += 16;
                            continue;
                        }
                        k += rrrr;
                        if (k > 63 || ssss > 10)
                            return ORACLE_ERR;
                        z[zz_pos[k]] = (int16_t)receive_extend(&bs, ssss);
                        ++k;
                    }
                    if (bs.bad)
                        return ORACLE_ERR;
                }
            }
            return ORACLE_OK;
        }
        /* APPn, COM and other segments are skipped */
        p = seg_end;
    }
}
