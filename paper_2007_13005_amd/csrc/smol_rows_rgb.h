// smol_rows_rgb.h -- the RGB row-streaming kernel (rgb_rows_kernel) and the
// choice of its instance for a plan. The smol_rows_rgb_*.hip files instantiate
// its parts.
#pragma once

#include "smol_rows.h"

namespace smol {
namespace {

// FORM: bit 0 NHWC output, bit 1 odd crop width (kFormNhwc, kFormOdd).
template <int F16, int J, int EXACT, int G, int P, int STRIDE, int FORM>
__global__ void __launch_bounds__(64 * kRowsMaxWavesPerGroup) rgb_rows_kernel(BatchArgs a)
{
    constexpr int NHWC = FORM & kFormNhwc, ODD = (FORM & kFormOdd) ? 1 : 0;
    extern __shared__ __attribute__((aligned(16))) uint8_t lds_all[];
    int lane;
    long long r0;
    int n_rows;
    const int Ch = a.Ch;
    uint8_t *const lds = rows_wave<STRIDE>(lds_all, 2048 * G, a, lane, r0, n_rows);
    // The host launches at most one wave per row, so every wave has rows (an
    // early exit here would hold the remaining argument loads behind it).
    __builtin_assume(n_rows > 0);
    const RowStep step = row_step_of<STRIDE>(a);
    constexpr int kEsz = F16 == 2 ? 1 : F16 ? 2 : 4;
    int c_img, c_rr;  // row to interpolate
    split_row<STRIDE>(r0, Ch, c_img, c_rr);
    RowCursor lc;  // next row to load
    cursor_image<STRIDE>(lc, a, c_img, c_rr, step);

    // The load cursor stops at the wave's last row: past the end the loads
    // repeat that row (fetching one chunk), so every step issues the same
    // loads and the compiler can count exactly what is outstanding when a
    // row is written to LDS.
    int lrow = 0;
    bool at_end = false;  // the cursor sits on the wave's last row, already loaded
    auto advance = [&]() {
        if (lrow + 1 < n_rows) {
            cursor_next<STRIDE>(lc, a, step);
            ++lrow;
        } else {
            at_end = true;
        }
    };
    // The first row (two with P = 2) is requested before the column taps
    // and the rest of the set-up are computed.
    StagedRows<G> A, B, C;
    load_rows<G, STRIDE>(A, lc, lane, false);
    advance();
    if (P == 2) {
        load_rows<G, STRIDE>(B, lc, lane, at_end);
        advance();
    }

    // Output row pointer of the row to interpolate: a step adds 3 Ch di + dr
    // rows, plus 2 Ch (planes 1 and 2 of the image left) when it wraps.
    // bytes between an image's output rows: Cw elements per plane (NCHW) or
    // 3 Cw (NHWC); a wrap to the next image skips the rest of the image.
    const long long rb = (long long)a.Cw * kEsz, rowb = NHWC ? 3 * rb : rb;
    const long long imgb = 3LL * Ch * rb;
    uint8_t *orow = (uint8_t *)a.out + (long long)(a.img_base + c_img) * imgb + c_rr * rowb;
    const long long ostep = step.di * imgb + step.dr * rowb, owrap = imgb - Ch * rowb;
    int cx[J][2];
    float cw[J][2];
    int cW, cWr, cleft;
    {
        const RowImg g = row_img(a, c_img);
        row_taps<J>(g, a.Cw, cx, cw, lane);
        cW = g.W;
        cWr = g.Wr;
        cleft = g.left;
    }
    const NormK nk = norm_consts(a);
    const uint32_t lds0 = lds_addr(lds);

    // P = 2: a step loads row k + 2 into FUT, interpolates row k (staged in
    // LDS), writes row k + 1 (in NXT) into the slot; the three register sets
    // rotate over three steps without copies. P = 1: one register set, loaded
    // with row k + 1 before row k is interpolated. The loop runs the n_rows - 1
    // steps that stage a next row and leaves only at its end, with nothing
    // outstanding but the prefetched row; the last row is interpolated after
    // it.
    write_rows<G>(lds, A, lane);
    int csh0 = A.sh0, csh1 = A.sh1, cy0 = A.y0, cy1 = A.y1;
    float cwy = A.wy;
    // Contiguous ranges keep the horizontal lerps of the last two source
    // rows (see rows_compute_reuse); J = 4 would need 48 more registers.
    constexpr bool kReuse = STRIDE == 0 && J <= 2;
    float h0[J][2][3], h1[J][2][3];
    int py0 = -1, py1 = -1;
    const long long plane = (long long)Ch * a.Cw * kEsz;
    RowOut<F16, J> out;
    auto compute = [&]() {
        if constexpr (kReuse)
            rows_compute_reuse<F16, J, EXACT>(nk, lds0 + (uint32_t)csh0,
                                              lds0 + (uint32_t)(1024 * G + csh1), cwy, cy0, cy1,
                                              py0, py1, h0, h1, cx, cw, out);
        else
            rows_compute<F16, J, EXACT>(nk, lds0 + (uint32_t)csh0,
                                        lds0 + (uint32_t)(1024 * G + csh1), cwy, cx, cw, out);
    };
#define SMOL_ROWS_STEP(NXT, FUT)                                                              \
    {                                                                                         \
        load_rows<G, STRIDE>(FUT, lc, lane, at_end);                                                  \
        advance();                                                                            \
        compute();                                                                            \
        write_rows<G>(lds, NXT, lane);                                                        \
        store_row<F16, J, ODD>(orow, plane, a.Cw, lane, out, NHWC);                         \
        csh0 = NXT.sh0;                                                                       \
        csh1 = NXT.sh1;                                                                       \
        cy0 = NXT.y0;                                                                         \
        cy1 = NXT.y1;                                                                         \
        cwy = NXT.wy;                                                                         \
        const int pimg = c_img;                                                               \
        c_img += step.di;                                                                     \
        c_rr += step.dr;                                                                      \
        orow += ostep;                                                                        \
        if (c_rr >= Ch) {                                                                     \
            c_rr -= Ch;                                                                       \
            ++c_img;                                                                          \
            orow += owrap;                                                                    \
        }                                                                                     \
        if (c_img != pimg) {                                                                  \
            py0 = py1 = -1; /* another image's rows */                                        \
            const RowImg g = row_img(a, c_img);                                               \
            if (g.W != cW || g.Wr != cWr || g.left != cleft) {                                \
                cW = g.W;                                                                     \
                cWr = g.Wr;                                                                   \
                cleft = g.left;                                                               \
                row_taps<J>(g, a.Cw, cx, cw, lane);                                           \
            }                                                                                 \
        }                                                                                     \
    }
    int left = n_rows - 1;
    if (P == 2) {
        for (; left >= 3; left -= 3) {
            SMOL_ROWS_STEP(B, C)
            SMOL_ROWS_STEP(C, A)
            SMOL_ROWS_STEP(A, B)
        }
        if (left >= 1)
            SMOL_ROWS_STEP(B, C)
        if (left >= 2)
            SMOL_ROWS_STEP(C, A)
    } else {
        for (; left > 0; --left)
            SMOL_ROWS_STEP(A, A)
    }
#undef SMOL_ROWS_STEP
    compute();
    store_row<F16, J, ODD>(orow, plane, a.Cw, lane, out, NHWC);
}

// pairs per lane and prefetch depth from the launch arguments.
template <int F16, int EXACT, int G, int STRIDE, int FORM>
const void *rgb_rows_g(int col_iters, int prefetch)
{
    if (prefetch == 1)
        return col_iters <= 1   ? (const void *)rgb_rows_kernel<F16, 1, EXACT, G, 1, STRIDE, FORM>
               : col_iters <= 2 ? (const void *)rgb_rows_kernel<F16, 2, EXACT, G, 1, STRIDE, FORM>
                                : (const void *)rgb_rows_kernel<F16, 4, EXACT, G, 1, STRIDE, FORM>;
    return col_iters <= 1   ? (const void *)rgb_rows_kernel<F16, 1, EXACT, G, 2, STRIDE, FORM>
           : col_iters <= 2 ? (const void *)rgb_rows_kernel<F16, 2, EXACT, G, 2, STRIDE, FORM>
                            : (const void *)rgb_rows_kernel<F16, 4, EXACT, G, 2, STRIDE, FORM>;
}

template <int F16, int EXACT, int STRIDE, int FORM>
const void *rgb_rows_e(int col_iters, int groups, int prefetch)
{
    return groups <= 1   ? rgb_rows_g<F16, EXACT, 1, STRIDE, FORM>(col_iters, prefetch)
           : groups <= 2 ? rgb_rows_g<F16, EXACT, 2, STRIDE, FORM>(col_iters, prefetch)
                         : rgb_rows_g<F16, EXACT, 4, STRIDE, FORM>(col_iters, prefetch);
}

// The crop width's parity picks the FORM of a layout.
template <int F16, int EXACT, int STRIDE, int NHWC>
const void *rgb_rows_f(const BatchArgs &a)
{
    return (a.Cw & 1) ? rgb_rows_e<F16, EXACT, STRIDE, NHWC | kFormOdd>(a.col_iters, a.row_groups,
                                                                       a.prefetch)
                      : rgb_rows_e<F16, EXACT, STRIDE, NHWC>(a.col_iters, a.row_groups, a.prefetch);
}

template <int F16, int STRIDE, int NHWC>
const void *rgb_rows_table(const BatchArgs &a)
{
    return a.exact ? rgb_rows_f<F16, 1, STRIDE, NHWC>(a) : rgb_rows_f<F16, 0, STRIDE, NHWC>(a);
}
}  // namespace
}  // namespace smol
