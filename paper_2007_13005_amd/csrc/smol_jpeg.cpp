// smol_jpeg.cpp -- C ABI of partial JPEG decoding (include/smol_jpeg.h):
// validation, Algorithm 1's rectangle per frame, grouping of frames into
// launches of the block-decoding kernel, and the decode-then-preprocess call.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "smol.h"
#include "smol_internal.h"
#include "smol_magic.h"
#include "smol_jpeg.h"

namespace smol {
// The workgroups_per_cu knob of smol_set_tuning, 0 when automatic
// (smol_host.cpp).
int tuned_workgroups_per_cu();
}  // namespace smol

namespace {

// launches of block decoding made by the calling thread's last decode
thread_local int t_decode_launches = 0;

// Block ranges of one frame's rectangle.
struct Blocks {
    int32_t W, H, bw, bh;
    int32_t lbx0, lby0, lnbx, lnby, cbx0, cby0, cnbx, cnby;
    int32_t wx0, wy0, wmx, wmy;  // MCU window the coefficients hold
    bool same_geometry(const Blocks &o) const
    {
        return W == o.W && H == o.H && lbx0 == o.lbx0 && lby0 == o.lby0 && lnbx == o.lnbx &&
               lnby == o.lnby && wx0 == o.wx0 && wy0 == o.wy0 && wmx == o.wmx && wmy == o.wmy;
    }
};

Blocks blocks_of(int64_t W, int64_t H, int64_t rx, int64_t ry, int64_t rw, int64_t rh)
{
    Blocks b;
    b.W = (int32_t)W;
    b.H = (int32_t)H;
    b.bw = (int32_t)(2 * ((W + 15) / 16));
    b.bh = (int32_t)(2 * ((H + 15) / 16));
    b.lbx0 = (int32_t)(rx / 8);
    b.lby0 = (int32_t)(ry / 8);
    b.lnbx = (int32_t)((rx + rw - 1) / 8 - rx / 8 + 1);
    b.lnby = (int32_t)((ry + rh - 1) / 8 - ry / 8 + 1);
    const int64_t cx0 = rx / 2, cx1 = (rx + rw - 1) / 2, cy0 = ry / 2, cy1 = (ry + rh - 1) / 2;
    b.cbx0 = (int32_t)(cx0 / 8);
    b.cby0 = (int32_t)(cy0 / 8);
    b.cnbx = (int32_t)(cx1 / 8 - cx0 / 8 + 1);
    b.cnby = (int32_t)(cy1 / 8 - cy0 / 8 + 1);
    return b;
}

int64_t coef_count(int64_t W, int64_t H)
{
    const int64_t bw = 2 * ((W + 15) / 16), bh = 2 * ((H + 15) / 16);
    return 64 * (bw * bh + 2 * (bw / 2) * (bh / 2));
}

// MCU window of a rectangle: first column and row, columns, rows
void mcu_window(int64_t W, int64_t H, const int32_t *rect, int64_t win[4])
{
    if (!rect) {
        win[0] = win[1] = 0;
        win[2] = (W + 15) / 16;
        win[3] = (H + 15) / 16;
        return;
    }
    win[0] = rect[0] / 16;
    win[1] = rect[1] / 16;
    win[2] = ((int64_t)rect[0] + rect[2] - 1) / 16 - win[0] + 1;
    win[3] = ((int64_t)rect[1] + rect[3] - 1) / 16 - win[1] + 1;
}

int64_t frame_bytes(int64_t W, int64_t H)
{
    return W * H + 2 * ((W + 1) / 2) * ((H + 1) / 2);
}

}  // namespace

extern "C" {

int64_t smol_jpeg_coef_count(int32_t width, int32_t height)
{
    if (width < 1 || height < 1)
        return 0;
    return coef_count(width, height);
}

int64_t smol_jpeg_window_coef_count(int32_t width, int32_t height, const int32_t *rect)
{
    if (width < 1 || height < 1)
        return 0;
    if (rect && (rect[0] < 0 || rect[1] < 0 || rect[2] < 1 || rect[3] < 1 ||
                 (int64_t)rect[0] + rect[2] > width || (int64_t)rect[1] + rect[3] > height))
        return 0;
    int64_t win[4];
    mcu_window(width, height, rect, win);
    return 64 * 6 * win[2] * win[3];
}

int smol_jpeg_mcu_rect(int32_t width, int32_t height, const smol_params *p,
                       const smol_options *opts, int32_t *rect)
{
    smol::clear_error();
    if (!p || !rect)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "params or rect is NULL");
    if (width < 1 || height < 1 || width > SMOL_MAX_DIM || height > SMOL_MAX_DIM)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "size %dx%d outside 1..%d", width, height,
                               SMOL_MAX_DIM);
    const int mode = opts ? opts->resize_mode : SMOL_RESIZE_SHORT_CROP;
    if (mode != SMOL_RESIZE_SHORT_CROP && mode != SMOL_RESIZE_DIRECT)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "resize_mode %d unknown", mode);
    return smol::mcu_rect(width, height, p, mode, rect);
}

int smol_jpeg_decode_i420(const int16_t *coef, int64_t coef_elems, const int64_t *coef_offsets,
                          const uint16_t *qtables, int32_t n_qtables, const int32_t *widths,
                          const int32_t *heights, const int32_t *rects, int32_t n,
                          int32_t coef_layout, uint8_t *out, int64_t out_bytes,
                          const int64_t *y_offsets, const int64_t *cb_offsets,
                          const int64_t *cr_offsets, void *stream)
{
    smol::clear_error();
    if (n < 0 || n > SMOL_MAX_BATCH)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "n = %d outside 0..%d", n, SMOL_MAX_BATCH);
    if (n == 0)
        return SMOL_OK;
    if (!coef || !coef_offsets || !qtables || !widths || !heights || !out || !y_offsets ||
        !cb_offsets || !cr_offsets)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "a NULL pointer or table");
    if (((uintptr_t)coef & 15) != 0)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "coef must be 16-byte aligned");
    if (n_qtables != 1 && n_qtables != n)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "n_qtables = %d: 1 or n (%d)", n_qtables,
                               n);
    for (int64_t i = 0; i < 128LL * n_qtables; ++i)
        if (qtables[i] < 1 || qtables[i] > 255)
            return smol::set_error(SMOL_ERR_INVALID_ARG, "table %lld entry %lld = %d outside "
                                   "1..255", (long long)(i / 128), (long long)(i % 128),
                                   qtables[i]);
    if (coef_layout != SMOL_JPEG_COEF_FRAME && coef_layout != SMOL_JPEG_COEF_WINDOW)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "coef_layout %d unknown", coef_layout);
    if (coef_layout == SMOL_JPEG_COEF_WINDOW && !rects)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "the window layout needs rects");
    std::vector<Blocks> blk((size_t)n);
    for (int32_t i = 0; i < n; ++i) {
        const int64_t W = widths[i], H = heights[i];
        if (W < 1 || H < 1 || W > SMOL_MAX_DIM || H > SMOL_MAX_DIM)
            return smol::set_error(SMOL_ERR_INVALID_ARG, "frame %d: size %lldx%lld outside 1..%d",
                                   i, (long long)W, (long long)H, SMOL_MAX_DIM);
        if (coef_offsets[i] % 8 != 0)
            return smol::set_error(SMOL_ERR_INVALID_ARG, "frame %d: coefficient offset not a "
                                   "multiple of 8", i);
        const int64_t Wc = (W + 1) / 2, Hc = (H + 1) / 2;
        const int64_t offs[3] = {y_offsets[i], cb_offsets[i], cr_offsets[i]};
        const int64_t sizes[3] = {W * H, Wc * Hc, Wc * Hc};
        for (int k = 0; k < 3; ++k)
            if (offs[k] < 0 || offs[k] > out_bytes || sizes[k] > out_bytes - offs[k])
                return smol::set_error(SMOL_ERR_INVALID_ARG, "frame %d: plane %d outside out",
                                       i, k);
        int64_t rx = 0, ry = 0, rw = W, rh = H;
        if (rects) {
            rx = rects[4 * i];
            ry = rects[4 * i + 1];
            rw = rects[4 * i + 2];
            rh = rects[4 * i + 3];
            if (rx < 0 || ry < 0 || rw < 1 || rh < 1 || rx + rw > W || ry + rh > H ||
                (rx & 1) || (ry & 1))
                return smol::set_error(SMOL_ERR_INVALID_ARG, "frame %d: rectangle (%lld, %lld, "
                                       "%lld, %lld) outside the frame or at an odd origin", i,
                                       (long long)rx, (long long)ry, (long long)rw,
                                       (long long)rh);
        }
        Blocks &g = blk[(size_t)i];
        g = blocks_of(W, H, rx, ry, rw, rh);
        int64_t win[4];
        mcu_window(W, H, coef_layout == SMOL_JPEG_COEF_WINDOW ? rects + 4 * (size_t)i : nullptr,
                   win);
        g.wx0 = (int32_t)win[0];
        g.wy0 = (int32_t)win[1];
        g.wmx = (int32_t)win[2];
        g.wmy = (int32_t)win[3];
        if (coef_offsets[i] < 0 || coef_offsets[i] > coef_elems ||
            64 * 6 * win[2] * win[3] > coef_elems - coef_offsets[i])
            return smol::set_error(SMOL_ERR_INVALID_ARG, "frame %d: coefficients outside coef",
                                   i);
    }

    smol::JpegArgs a;
    std::memset(&a, 0, sizeof a);
    // frame i's luma and chroma tables
    auto tables = [&](int32_t i) { return qtables + (n_qtables == 1 ? 0 : 128 * (size_t)i); };
    auto same_tables = [&](int32_t i, int32_t j) {
        return n_qtables == 1 || std::memcmp(tables(i), tables(j), 128 * sizeof(uint16_t)) == 0;
    };
    int ntables = 0;
    int32_t table_frame[smol::kJpegMaxTables];  // a frame using each of the launch's tables
    const double pi = 3.14159265358979323846;
    for (int k = 0; k < 8; ++k)
        for (int m = 0; m < 8; ++m)
            a.c[k * 8 + m] = (float)((k == 0 ? 1.0 / std::sqrt(2.0) : 1.0) / 2.0 *
                                     std::cos((2.0 * m + 1.0) * k * pi / 16.0));
    const int cus = smol::device_cus();
    a.coef = coef;
    a.out = out;
    // Runs of frames with one geometry, one pair of tables and constant
    // strides; up to kJpegMaxRuns runs and kJpegMaxTables pairs share a launch.
    long long jobs = 0;
    auto flush = [&]() -> int {
        if (a.runs == 0)
            return SMOL_OK;
        // 128 one-wave workgroups per compute unit, each looping over jobs
        // (or the workgroups_per_cu knob): measured faster than 32
        // (long-lived waves) and than one workgroup per job on 128 720p
        // frames
        const int per_cu = smol::tuned_workgroups_per_cu() > 0 ? smol::tuned_workgroups_per_cu() : 128;
        const int grid = (int)std::min<long long>(jobs, (long long)(cus > 0 ? cus : 256) * per_cu);
        const int rc = smol::launch_jpeg_idct(a, grid, stream);
        t_decode_launches += rc == (int)hipSuccess ? 1 : 0;
        a.runs = 0;
        jobs = 0;
        ntables = 0;
        if (rc != (int)hipSuccess)
            return smol::set_error(SMOL_ERR_HIP, "block decoding launch: %s",
                                   hipGetErrorString((hipError_t)rc));
        return SMOL_OK;
    };
    for (int32_t b = 0; b < n;) {
        int32_t e = b + 1;
        const int64_t cs = e < n ? coef_offsets[e] - coef_offsets[b] : 0;
        const int64_t os = e < n ? y_offsets[e] - y_offsets[b] : 0;
        while (e < n && blk[(size_t)e].same_geometry(blk[(size_t)b]) &&
               coef_offsets[e] - coef_offsets[e - 1] == cs &&
               y_offsets[e] - y_offsets[e - 1] == os &&
               cb_offsets[e] - y_offsets[e] == cb_offsets[b] - y_offsets[b] &&
               cr_offsets[e] - y_offsets[e] == cr_offsets[b] - y_offsets[b] &&
               same_tables(e, b))
            ++e;
        // the kernel's job indices stay below 2^31: split runs and launches
        const Blocks &g0 = blk[(size_t)b];
        const long long per_frame =
            (long long)(g0.lnbx + 7) / 8 * g0.lnby + 2LL * ((g0.cnbx + 7) / 8) * g0.cnby;
        const long long max_jobs = 0x7fffffffLL;
        if (jobs + per_frame > max_jobs) {
            const int rc = flush();
            if (rc != SMOL_OK)
                return rc;
        }
        e = (int32_t)std::min<long long>(e, b + (max_jobs - jobs) / per_frame);
        int qt = 0;
        while (qt < ntables && !same_tables(table_frame[qt], b))
            ++qt;
        if (qt == smol::kJpegMaxTables) {
            const int rc = flush();
            if (rc != SMOL_OK)
                return rc;
            qt = 0;
        }
        if (qt == ntables) {
            table_frame[ntables++] = b;
            const uint16_t *t = tables(b);
            for (int k = 0; k < 128; ++k)
                a.q[qt][k / 64][k % 64] = (uint8_t)t[k];
        }
        const Blocks &g = blk[(size_t)b];
        smol::JpegRun &r = a.run[a.runs];
        r.coef = coef_offsets[b];
        r.coef_stride = cs;
        r.out = y_offsets[b];
        r.out_stride = os;
        r.cboff = cb_offsets[b] - y_offsets[b];
        r.croff = cr_offsets[b] - y_offsets[b];
        r.W = (int32_t)g.W;
        r.H = (int32_t)g.H;
        r.wx0 = (int16_t)g.wx0;
        r.wy0 = (int16_t)g.wy0;
        r.wmx = (int16_t)g.wmx;
        r.wmy = (int16_t)g.wmy;
        r.lbx0 = (int16_t)g.lbx0;
        r.lby0 = (int16_t)g.lby0;
        r.lnbx = (int16_t)g.lnbx;
        r.lnby = (int16_t)g.lnby;
        r.cbx0 = (int16_t)g.cbx0;
        r.cby0 = (int16_t)g.cby0;
        r.cnbx = (int16_t)g.cnbx;
        r.cnby = (int16_t)g.cnby;

        // jobs of the kernel: groups of up to eight blocks along block rows
        jobs += per_frame * (e - b);
        r.jobs_end = (uint32_t)jobs;
        // lg, cg <= 1025 (11 bits each); the last group of a row holds 1..8
        const uint32_t lg = (uint32_t)((g.lnbx + 7) / 8), cg = (uint32_t)((g.cnbx + 7) / 8);
        const uint32_t lrem = (uint32_t)g.lnbx - 8 * (lg - 1), crem = (uint32_t)g.cnbx - 8 * (cg - 1);
        r.lum = lg * (uint32_t)g.lnby;
        r.chr = cg * (uint32_t)g.cnby;
        r.groups = lg | cg << 11 | lrem << 22 | crem << 26;
        uint32_t s_pf, s_lg, s_cg;
        smol::magic_divisor((uint32_t)per_frame, &r.m_pf, &s_pf);
        smol::magic_divisor(lg, &r.m_lg, &s_lg);
        smol::magic_divisor(cg, &r.m_cg, &s_cg);
        r.shifts = s_pf | s_lg << 8 | s_cg << 16 | (uint32_t)qt << 24;
        if (++a.runs == smol::kJpegMaxRuns) {
            const int rc = flush();
            if (rc != SMOL_OK)
                return rc;
        }
        b = e;
    }
    const int rc = flush();
    if (rc != SMOL_OK)
        return rc;
    return SMOL_OK;
}

int64_t smol_jpeg_workspace_bytes(int32_t n, const int32_t *widths, const int32_t *heights)
{
    if (n < 1 || !widths || !heights)
        return 0;
    int64_t total = 0;
    for (int32_t i = 0; i < n; ++i) {
        if (widths[i] < 1 || heights[i] < 1)
            return 0;
        total += frame_bytes(widths[i], heights[i]);
    }
    return ((total + 15) & ~(int64_t)15) + 16;
}

int smol_jpeg_roi_preprocess_batch(const int16_t *coef, int64_t coef_elems,
                                   const int64_t *coef_offsets, const uint16_t *qtables,
                                   int32_t n_qtables, const int32_t *widths,
                                   const int32_t *heights, int32_t n,
                                   int32_t coef_layout, const smol_params *p,
                                   const smol_options *opts, void *workspace,
                                   int64_t workspace_bytes, void *out, void *stream)
{
    smol::clear_error();
    if (n < 0 || n > SMOL_MAX_BATCH)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "n = %d outside 0..%d", n, SMOL_MAX_BATCH);
    if (n == 0)
        return SMOL_OK;
    if (!widths || !heights || !p)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "widths, heights or params is NULL");
    smol_options o = {};
    if (opts)
        o = *opts;
    if (o.chroma_siting != SMOL_CHROMA_CENTER)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "JPEG chroma is centred: chroma_siting "
                               "must be SMOL_CHROMA_CENTER");
    if (o.layout != SMOL_LAYOUT_NCHW && o.layout != SMOL_LAYOUT_NHWC)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "layout %d unknown", o.layout);
    for (int i = 0; i < 5; ++i)
        if (o.reserved[i])
            return smol::set_error(SMOL_ERR_INVALID_ARG, "options reserved[%d] is not zero", i);
    const int64_t need = smol_jpeg_workspace_bytes(n, widths, heights);
    if (!workspace || workspace_bytes < need || need == 0)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "workspace of %lld bytes, %lld needed",
                               (long long)workspace_bytes, (long long)need);
    if (((uintptr_t)workspace & 15) != 0)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    std::vector<int32_t> rects(4 * (size_t)n);
    std::vector<int64_t> yo((size_t)n), bo((size_t)n), ro((size_t)n);
    int64_t cur = 0;
    for (int32_t i = 0; i < n; ++i) {
        // validates the size and the preprocessing parameters for this frame
        const int rc = smol_jpeg_mcu_rect(widths[i], heights[i], p, &o, &rects[4 * (size_t)i]);
        if (rc)
            return rc;
        const int64_t W = widths[i], H = heights[i];
        yo[(size_t)i] = cur;
        bo[(size_t)i] = cur + W * H;
        ro[(size_t)i] = bo[(size_t)i] + ((W + 1) / 2) * ((H + 1) / 2);
        cur += frame_bytes(W, H);
    }
    t_decode_launches = 0;
    int rc = smol_jpeg_decode_i420(coef, coef_elems, coef_offsets, qtables, n_qtables, widths,
                                   heights, rects.data(), n, coef_layout,
                                   (uint8_t *)workspace, workspace_bytes, yo.data(), bo.data(),
                                   ro.data(), stream);
    if (rc)
        return rc;
    const int decode_launches = t_decode_launches;
    rc = smol_yuv420_preprocess_batch_ex((const uint8_t *)workspace, workspace_bytes, yo.data(),
                                         bo.data(), ro.data(), widths, heights, nullptr, n, p,
                                         &o, out, stream);
    if (rc == SMOL_OK)
        smol::add_plan_launches(decode_launches);  // the plan reports both stages
    return rc;
}

}  // extern "C"
