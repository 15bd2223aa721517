// smol_host.cpp -- C ABI of libsmol: validation, per-image geometry,
// descriptor staging and kernel dispatch. Everything per element runs in the
// kernels (smol_kernels.hip); this file handles per-image scalars only.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cfloat>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "smol.h"
#include "smol_internal.h"

namespace {

using smol::BatchArgs;
using smol::Desc;

thread_local std::string g_last_error;
thread_local smol_plan g_last_plan = {};

int fail(int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

std::atomic<int> g_path{0}, g_band_rows{0}, g_lds_budget{0}, g_wg_per_cu{0}, g_exact{0},
    g_row_order{0}, g_upload{0};

// True while this thread runs smol_preprocess_batch_noalloc: descriptor tables
// then go to the fixed device array of smol_scratch.hip, not to the staging
// ring and device buffer the other calls allocate.
thread_local bool t_noalloc = false;

constexpr int kDefaultLdsBudget = 64 * 1024;
constexpr int kMaxBandRows = 64;
constexpr int kMaxWorkgroupsPerCu = 16;
constexpr int kDefaultBandRows = 2;
constexpr long long kRowsMinPerWave = 3;  // rows per wave a launch aims for (row streaming)
constexpr int kGatherPassPixels = 2048;  // 256 threads x 4 pairs x 2 pixels
// Row-streaming waves per compute unit for long staged rows (4 KiB chunk
// groups): more waves would each walk fewer rows, and every wave pays its
// column taps and one exposed load latency to start.
constexpr int kRowsWavesPerCu = 8;

// Per-device facts the planner needs, queried once.
struct DeviceInfo {
    int cus = 0;
    int lds_per_cu = 0;
    int lds_per_block = 0;
};
std::mutex g_dev_mu;
std::vector<DeviceInfo> g_dev_info;

hipError_t device_info(int device, DeviceInfo *out)
{
    std::lock_guard<std::mutex> lk(g_dev_mu);
    if ((int)g_dev_info.size() <= device)
        g_dev_info.resize(device + 1);
    DeviceInfo &di = g_dev_info[device];
    if (di.cus == 0) {
        int cus = 0, lds = 0;
        hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
        if (e != hipSuccess)
            return e;
        e = hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor,
                                  device);
        if (e != hipSuccess)
            return e;
        int lpb = 0;
        e = hipDeviceGetAttribute(&lpb, hipDeviceAttributeMaxSharedMemoryPerBlock, device);
        if (e != hipSuccess)
            return e;
        di.cus = cus;
        di.lds_per_cu = lds > 0 ? lds : 65536;
        di.lds_per_block = lpb > 0 ? lpb : 65536;
    }
    *out = di;
    return hipSuccess;
}

// ---------------------------------------------------------------------------
// Geometry (section 2 step 2; Algorithm 1 for the crop offsets)
// ---------------------------------------------------------------------------

struct Geo {
    int64_t Wr, Hr, left, top;
};

// Short side -> S, long side floor(S * long / short).
// a / b for a >= 0, b > 0: a 32-bit division when both fit (several times
// cheaper than a 64-bit one on x86, and per image the host does five)
inline int64_t udiv(int64_t a, int64_t b)
{
    if (((uint64_t)a | (uint64_t)b) >> 32 == 0)
        return (int64_t)((uint32_t)a / (uint32_t)b);
    return a / b;
}

void resized(int64_t W, int64_t H, int64_t S, int64_t *Wr, int64_t *Hr)
{
    if (W <= H) {
        *Wr = S;
        *Hr = udiv(S * H, W);
    } else {
        *Hr = S;
        *Wr = udiv(S * W, H);
    }
}

// Host copy of the half-pixel tap (integer part only) for footprint queries
// and LDS planning: floor of ((2x+1)*in - out) / (2*out), clamped.
void tap_index(int64_t x, int64_t in, int64_t out, int64_t *x0, int64_t *x1)
{
    const int64_t num = (2 * x + 1) * in - out;
    if (num <= 0) {
        *x0 = *x1 = 0;
        return;
    }
    const int64_t q = udiv(num, 2 * out);
    if (q >= in - 1) {
        *x0 = *x1 = in - 1;
        return;
    }
    *x0 = q;
    *x1 = q + 1;
}

// Chroma tap index for luma index x: floor((2x - 1) / 4) for centred siting,
// floor(2x / 4) for co-sited (left), clamped to [0, n-1].
void chroma_index(int64_t x, int64_t n, int64_t *c0, int64_t *c1, int left = 0)
{
    const int64_t num = 2 * x - 1 + left;
    if (num <= 0) {
        *c0 = *c1 = 0;
        return;
    }
    const int64_t q = num >> 2;
    if (q >= n - 1) {
        *c0 = *c1 = n - 1;
        return;
    }
    *c0 = q;
    *c1 = q + 1;
}

int check_params(const smol_params *p)
{
    if (!p)
        return fail(SMOL_ERR_INVALID_ARG, "params is NULL");
    if (p->resize_short < 1 || p->resize_short > SMOL_MAX_RESIZED)
        return fail(SMOL_ERR_INVALID_ARG, "resize_short %d out of range", p->resize_short);
    if (p->crop_h < 1 || p->crop_w < 1)
        return fail(SMOL_ERR_INVALID_ARG, "crop %dx%d must be positive", p->crop_h, p->crop_w);
    if (p->out_dtype != SMOL_OUT_F32 && p->out_dtype != SMOL_OUT_F16 &&
        p->out_dtype != SMOL_OUT_U8)
        return fail(SMOL_ERR_INVALID_ARG, "out_dtype %d unknown", p->out_dtype);
    if (p->out_dtype == SMOL_OUT_U8)
        return SMOL_OK;  // mean and std are not used
    for (int c = 0; c < 3; ++c) {
        if (!std::isfinite(p->mean[c]) || !std::isfinite(p->std[c]) || p->std[c] == 0.0f)
            return fail(SMOL_ERR_INVALID_ARG, "mean/std of channel %d not finite or std == 0", c);
        const float r = 1.0f / p->std[c];
        if (!std::isfinite(r) || std::fabs(r) < FLT_MIN ||
            !std::isfinite((float)((std::fabs((double)p->mean[c]) + 255.0) * (double)r)))
            return fail(SMOL_ERR_INVALID_ARG,
                        "1/std of channel %d is not a normal number or the output overflows", c);
    }
    return SMOL_OK;
}

int check_options(const smol_options *o, smol_options *out)
{
    std::memset(out, 0, sizeof *out);
    if (!o)
        return SMOL_OK;
    if (o->resize_mode != SMOL_RESIZE_SHORT_CROP && o->resize_mode != SMOL_RESIZE_DIRECT)
        return fail(SMOL_ERR_INVALID_ARG, "resize_mode %d unknown", o->resize_mode);
    if (o->layout != SMOL_LAYOUT_NCHW && o->layout != SMOL_LAYOUT_NHWC)
        return fail(SMOL_ERR_INVALID_ARG, "layout %d unknown", o->layout);
    if (o->chroma_siting != SMOL_CHROMA_CENTER && o->chroma_siting != SMOL_CHROMA_LEFT)
        return fail(SMOL_ERR_INVALID_ARG, "chroma_siting %d unknown", o->chroma_siting);
    for (int k = 0; k < 5; ++k)
        if (o->reserved[k] != 0)
            return fail(SMOL_ERR_INVALID_ARG, "options: reserved[%d] is not zero", k);
    *out = *o;
    return SMOL_OK;
}

// The processed region of image i: its ROI (rois[4i..4i+3]) or the whole
// W x H image.
int region(const int32_t *rois, int64_t i, int64_t W, int64_t H, int64_t *rx, int64_t *ry,
           int64_t *rw, int64_t *rh)
{
    if (!rois) {
        *rx = *ry = 0;
        *rw = W;
        *rh = H;
        return SMOL_OK;
    }
    const int32_t *r = rois + 4 * i;
    if (r[0] < 0 || r[1] < 0 || r[2] < 1 || r[3] < 1 || (int64_t)r[0] + r[2] > W ||
        (int64_t)r[1] + r[3] > H)
        return fail(SMOL_ERR_INVALID_ARG, "image %lld: ROI (%d, %d, %d, %d) not inside %lldx%lld",
                    (long long)i, r[0], r[1], r[2], r[3], (long long)W, (long long)H);
    *rx = r[0];
    *ry = r[1];
    *rw = r[2];
    *rh = r[3];
    return SMOL_OK;
}

int image_geo(int64_t W, int64_t H, const smol_params *p, int mode, Geo *g, int64_t i)
{
    if (W < 1 || H < 1 || W > SMOL_MAX_DIM || H > SMOL_MAX_DIM)
        return fail(SMOL_ERR_INVALID_ARG, "image %lld: size %lldx%lld outside 1..%d",
                    (long long)i, (long long)W, (long long)H, SMOL_MAX_DIM);
    if (mode == SMOL_RESIZE_DIRECT) {
        if (p->crop_w > SMOL_MAX_RESIZED || p->crop_h > SMOL_MAX_RESIZED)
            return fail(SMOL_ERR_UNSUPPORTED, "output %dx%d beyond %d", p->crop_w, p->crop_h,
                        SMOL_MAX_RESIZED);
        g->Wr = p->crop_w;
        g->Hr = p->crop_h;
        g->left = g->top = 0;
        return SMOL_OK;
    }
    resized(W, H, p->resize_short, &g->Wr, &g->Hr);
    if (g->Wr > SMOL_MAX_RESIZED || g->Hr > SMOL_MAX_RESIZED)
        return fail(SMOL_ERR_UNSUPPORTED, "image %lld: resized size %lldx%lld beyond %d",
                    (long long)i, (long long)g->Wr, (long long)g->Hr, SMOL_MAX_RESIZED);
    if (p->crop_w > g->Wr || p->crop_h > g->Hr)
        return fail(SMOL_ERR_INVALID_ARG, "image %lld: crop %dx%d larger than resized %lldx%lld",
                    (long long)i, p->crop_w, p->crop_h, (long long)g->Wr, (long long)g->Hr);
    g->left = (g->Wr - p->crop_w) / 2;
    g->top = (g->Hr - p->crop_h) / 2;
    return SMOL_OK;
}

// Source columns [x_first, x_last] read by the crop's columns.
void x_span(const Desc &d, int Cw, int64_t *first, int64_t *last)
{
    int64_t a, b;
    tap_index(d.left, d.W, d.Wr, first, &a);
    tap_index(d.left + Cw - 1, d.W, d.Wr, &b, last);
}

int64_t distinct_rows(int64_t top, int64_t Ch, int64_t H, int64_t Hr)
{
    int64_t count = 0, last = -1;
    for (int64_t r = 0; r < Ch; ++r) {
        int64_t y0, y1;
        tap_index(top + r, H, Hr, &y0, &y1);
        if (y0 > last) {
            ++count;
            last = y0;
        }
        if (y1 > last) {
            ++count;
            last = y1;
        }
    }
    return count;
}

// ---------------------------------------------------------------------------
// Per-device descriptor staging: pinned host ring + device ring. A ragged
// batch's table is copied on the library's own copy stream (a DMA engine, so
// the copy runs while the caller's stream is still busy with earlier work);
// the caller's stream waits for that copy before the kernel. A slot is
// reused once the kernel that read it has completed (the host waits for
// that kernel's event; the kernel itself waited for the slot's copy).
// ---------------------------------------------------------------------------

struct Staging {
    static constexpr int kSlots = 16;
    std::mutex mu;
    size_t slot_cap = 0;
    uint8_t *host = nullptr;
    uint8_t *host_dev = nullptr;     // the host ring as the device addresses it
    uint8_t *dev = nullptr;
    hipStream_t copy = nullptr;      // default priority, non-blocking
    hipEvent_t ev[kSlots] = {};      // after the kernel that read slot k
    bool pending[kSlots] = {};
    hipEvent_t up[kSlots] = {};      // after the copy into slot k
    bool up_pending[kSlots] = {};
    int next = 0;
};

std::mutex g_staging_mu;
std::vector<Staging *> g_staging;  // by device ordinal; never freed

Staging *staging_for(int device)
{
    std::lock_guard<std::mutex> lk(g_staging_mu);
    if ((int)g_staging.size() <= device)
        g_staging.resize(device + 1, nullptr);
    if (!g_staging[device])
        g_staging[device] = new Staging();
    return g_staging[device];
}

// Grow the ring so each slot holds `bytes` (and create the copy stream on
// first use). Caller holds st->mu.
hipError_t staging_reserve(Staging *st, size_t bytes)
{
    if (!st->copy) {
        hipError_t e = hipStreamCreateWithFlags(&st->copy, hipStreamNonBlocking);
        if (e != hipSuccess)
            return e;
    }
    if (bytes <= st->slot_cap)
        return hipSuccess;
    for (int i = 0; i < Staging::kSlots; ++i) {
        if (st->pending[i]) {
            hipError_t e = hipEventSynchronize(st->ev[i]);
            if (e != hipSuccess)
                return e;
            st->pending[i] = false;
        }
        if (st->up_pending[i]) {
            hipError_t e = hipEventSynchronize(st->up[i]);
            if (e != hipSuccess)
                return e;
            st->up_pending[i] = false;
        }
    }
    if (st->host)
        (void)hipHostFree(st->host);
    if (st->dev)
        (void)hipFree(st->dev);
    st->host = nullptr;
    st->dev = nullptr;
    st->slot_cap = 0;
    size_t cap = 64 * 1024;
    while (cap < bytes)
        cap *= 2;
    hipError_t e = hipHostMalloc((void **)&st->host, cap * Staging::kSlots, hipHostMallocDefault);
    if (e != hipSuccess)
        return e;
    e = hipHostGetDevicePointer((void **)&st->host_dev, st->host, 0);
    if (e != hipSuccess)
        return e;
    e = hipMalloc((void **)&st->dev, cap * Staging::kSlots);
    if (e != hipSuccess)
        return e;
    for (int i = 0; i < Staging::kSlots; ++i) {
        if (!st->ev[i]) {
            e = hipEventCreateWithFlags(&st->ev[i], hipEventDisableTiming);
            if (e != hipSuccess)
                return e;
        }
        if (!st->up[i]) {
            e = hipEventCreateWithFlags(&st->up[i], hipEventDisableTiming);
            if (e != hipSuccess)
                return e;
        }
    }
    st->slot_cap = cap;
    return hipSuccess;
}

// ---------------------------------------------------------------------------
// Planning and launch
// ---------------------------------------------------------------------------

struct Plan {
    int path;  // smol::PATH_DIRECT, _LDS, _GATHER or _ROWS
    // R: output rows per band (LDS) or row-pair slots per wave (ROWS)
    int R;
    size_t lds_bytes;
    int grid;
    int f16;
};

size_t align16(size_t v) { return (v + 15) & ~(size_t)15; }

// LDS layout of the RGB kernel: two buffers per workgroup, each
//   colx/colw [Cw] | rowa0/rowa1/twy [R] | 2R row slots.
size_t rgb_lds_bytes(int Cw, int R, int slot_bytes, int *slots_off, int *buf_bytes)
{
    const size_t head = align16((size_t)8 * Cw + (size_t)12 * R);
    const size_t buf = align16(head + (size_t)2 * R * slot_bytes);
    *slots_off = (int)head;
    *buf_bytes = (int)buf;
    return 2 * buf;
}

int slot_bytes_for(int64_t span_bytes)
{
    // aligned-down start adds up to 15 bytes; 16 more cover the dword reads
    // past the last pixel pair.
    return (int)(16 * ((span_bytes + 15 + 15) / 16) + 16);
}

Plan plan_rgb(int64_t max_span_bytes, int Ch, int Cw, int *slot_bytes, int *slots_off,
              int *stage_bytes)
{
    Plan pl{smol::PATH_DIRECT, 0, 0, 0, 0};
    const int forced = g_path.load();
    if (forced == smol::PATH_DIRECT)
        return pl;
    const int budget = g_lds_budget.load() > 0 ? g_lds_budget.load() : kDefaultLdsBudget;
    if (max_span_bytes > (1 << 20))
        return pl;
    const int sb = slot_bytes_for(max_span_bytes);
    int off, stage;
    int R = g_band_rows.load();
    if (R <= 0) {
        R = kDefaultBandRows;
        while (R > 1 && rgb_lds_bytes(Cw, R, sb, &off, &stage) > (size_t)budget)
            --R;
    }
    R = std::min(R, Ch);
    const size_t bytes = rgb_lds_bytes(Cw, R, sb, &off, &stage);
    if (bytes > (size_t)budget)
        return pl;
    pl.path = smol::PATH_LDS;
    pl.R = R;
    pl.lds_bytes = bytes;
    *slot_bytes = sb;
    *slots_off = off;
    *stage_bytes = stage;
    return pl;
}

void fill_norm(const smol_params *p, BatchArgs &a)
{
    for (int c = 0; c < 3; ++c) {
        a.mean[c] = p->mean[c];
        a.stdv[c] = p->std[c];
        // fp32 division on the host: the correctly rounded reciprocal the
        // kernels' quotient correction needs (not 1/(double), which would
        // round twice).
        volatile float one = 1.0f;
        a.rcp[c] = one / p->std[c];
        a.bias[c] = (float)(-(double)p->mean[c] / (double)p->std[c]);
    }
    a.exact = g_exact.load();
}

int hip_fail(hipError_t e, const char *what)
{
    return fail(SMOL_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool is_uniform(const std::vector<Desc> &d, size_t first, size_t count, int nofs,
                int64_t *stride);

// Shared tail of both entry points: uniform-batch detection, descriptor
// upload for ragged batches and the launch, for images
// [first, first + count) of descs (written to output images first.. on).
template <class Launch>
int run_batch(const std::vector<Desc> &descs, size_t first, size_t count, int nofs,
              BatchArgs a, Plan pl, void *stream, Launch launch, smol_plan *info)
{
    hipStream_t s = (hipStream_t)stream;
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    DeviceInfo di;
    e = device_info(device, &di);
    if (e != hipSuccess)
        return hip_fail(e, "hipDeviceGetAttribute");

    const int n = (int)count;
    int64_t stride = 0;
    const bool uniform = is_uniform(descs, first, count, nofs, &stride);
    a.n = n;
    a.img_base = (int)first;
    long long items;
    if (pl.path != smol::PATH_DIRECT && pl.lds_bytes > (size_t)di.lds_per_block)
        return fail(SMOL_ERR_UNSUPPORTED, "LDS plan of %zu bytes exceeds the device's %d per "
                    "workgroup", pl.lds_bytes, di.lds_per_block);
    const bool rows = pl.path == smol::PATH_ROWS || pl.path == smol::PATH_YUV_ROWS;
    {
        // Row order of the row-streaming kernels: interleaved across waves
        // for uniform batches of long staged rows (memory-bound: the waves
        // then stream neighbouring rows), contiguous ranges otherwise. (Set
        // before the occupancy query: the two walks are different kernels.)
        const int order = g_row_order.load();
        a.interleave = pl.f16 != SMOL_OUT_U8 &&
                       (order == 2 || (order == 0 && uniform && pl.path == smol::PATH_ROWS &&
                                       a.row_groups >= 4));
    }
    if (pl.path == smol::PATH_LDS || pl.path == smol::PATH_GATHER || rows) {
        a.wpg = rows ? smol::kRowsMaxWavesPerGroup : 1;
        int per_cu = 0;
        const int oc = pl.path == smol::PATH_LDS
                           ? smol::occupancy_rgb_lds(pl.f16, pl.lds_bytes, &per_cu)
                       : pl.path == smol::PATH_GATHER
                           ? smol::occupancy_rgb_gather(pl.f16, pl.lds_bytes, &per_cu)
                       : pl.path == smol::PATH_ROWS
                           ? smol::occupancy_rgb_rows(a, pl.f16, pl.lds_bytes, &per_cu)
                           : smol::occupancy_yuv_rows(a, pl.f16, pl.lds_bytes, &per_cu);
        if (oc != (int)hipSuccess)
            return hip_fail((hipError_t)oc, "hipOccupancyMaxActiveBlocksPerMultiprocessor");
        if (per_cu < 1)
            return fail(SMOL_ERR_UNSUPPORTED, "kernel cannot be resident with %zu bytes of LDS",
                        pl.lds_bytes);
        const int forced = g_wg_per_cu.load();
        if (rows) {
            // Waves per compute unit (the tuning knob counts waves here).
            int waves = per_cu * a.wpg;
            items = (long long)n * a.Ch;
            if (forced > 0) {
                waves = std::min(waves, forced);
            } else {
                if (pl.path == smol::PATH_ROWS && a.row_groups >= 4)
                    waves = std::min(waves, kRowsWavesPerCu);
                // Small launches: at least about three rows per wave, in
                // multiples of 4 waves per compute unit (a wave's set-up and
                // first load cost about a row; 7,168 rows of 224 columns take
                // 8.1 us on 5,120 waves and 6.7 us on 2,048).
                const long long by_rows = items / kRowsMinPerWave / di.cus;
                if (by_rows < waves)
                    waves = (int)std::min<long long>(waves,
                                                     std::max<long long>(4, by_rows & ~3LL));
            }
            // Workgroups of 4 (or 2) waves when that count allows, so each
            // compute unit still holds at most `waves` of them.
            a.wpg = waves % 4 == 0 ? 4 : waves % 2 == 0 ? 2 : 1;
            long long w = std::min<long long>(items, (long long)di.cus * waves);
            if (w >= a.wpg)
                w -= w % a.wpg;
            else
                a.wpg = 1;
            pl.grid = (int)w;
            // the rows each wave walks (q >= 1: w <= items, and the kernels
            // rely on every wave having a row), and the strided walk's step
            const long long q = items / w;
            if (q >= INT32_MAX)
                return fail(SMOL_ERR_UNSUPPORTED, "%lld output rows for %lld waves", items, w);
            a.rows_q = (int)q;
            a.rows_r = (int)(items - q * w);
            a.step_di = (int)(w / a.Ch);
            a.step_dr = (int)(w % a.Ch);
            if (uniform) {
                // |quotients| <= H + 1: |step_dr - Ch| <= Ch <= Hr
                const Desc &d = descs[first];
                const int64_t den = 2 * (int64_t)d.Hr;
                const int64_t nums[2] = {2 * (int64_t)d.H * a.step_dr,
                                         2 * (int64_t)d.H * (a.step_dr - a.Ch)};
                int32_t qr[4];
                for (int k = 0; k < 2; ++k) {
                    int64_t q = nums[k] / den, r = nums[k] - q * den;
                    if (r < 0) {
                        --q;
                        r += den;
                    }
                    qr[2 * k] = (int32_t)q;
                    qr[2 * k + 1] = (int32_t)r;
                }
                a.vq_s = qr[0];
                a.vr_s = qr[1];
                a.vq_w = qr[2];
                a.vr_w = qr[3];
            }
        } else {
            if (forced > 0)
                per_cu = std::min(per_cu, forced);
            items = pl.path == smol::PATH_LDS ? (long long)n * a.bands
                                              : (long long)n * (((long long)a.Ch * a.Cw +
                                                                 kGatherPassPixels - 1) /
                                                                kGatherPassPixels);
            pl.grid = (int)std::min<long long>(items, (long long)di.cus * per_cu);
        }
        a.grid = pl.grid;
    } else {
        items = (long long)n * a.Ch * a.Cw;
        pl.grid = 0;
    }

    // The plan reports the first launch of the most specialised kernel.
    if (info->launches == 0 || (info->path == smol::PATH_DIRECT && pl.path != smol::PATH_DIRECT)) {
        info->path = pl.path == smol::PATH_YUV_ROWS ? smol::PATH_ROWS : pl.path;
        info->band_rows = pl.path == smol::PATH_LDS ? pl.R : 0;
        info->lds_bytes = (int)pl.lds_bytes;
        info->grid = pl.grid;
        info->work_items = items;
    }
    info->uploaded_descriptors |= uniform ? 0 : 1;

    Staging *st = nullptr;
    std::unique_lock<std::mutex> lk;
    int slot = -1;
    if (!uniform && t_noalloc) {
        // The call's tables sit side by side in the device's fixed array (a
        // run of images [first, first + count) at descriptor `first`); calls on
        // one stream reuse it in stream order.
        if (first + count > (size_t)smol::kNoallocMaxImages)
            return fail(SMOL_ERR_UNSUPPORTED, "descriptor table of %zu images exceeds the "
                        "no-allocation limit of %d", first + count, smol::kNoallocMaxImages);
        void *table = nullptr;
        const int rc = smol::scratch_table(device, &table);
        if (rc != (int)hipSuccess)
            return hip_fail((hipError_t)rc, "hipGetSymbolAddress(descriptor table)");
        uint8_t *dv = (uint8_t *)table + first * sizeof(Desc);
        e = hipMemcpyAsync(dv, descs.data() + first, sizeof(Desc) * count,
                           hipMemcpyHostToDevice, s);
        if (e != hipSuccess)
            return hip_fail(e, "hipMemcpyAsync(descriptors)");
        a.table = (const Desc *)dv;
    } else if (!uniform) {
        st = staging_for(device);
        lk = std::unique_lock<std::mutex>(st->mu);
        const size_t bytes = sizeof(Desc) * count;
        e = staging_reserve(st, bytes);
        if (e != hipSuccess)
            return hip_fail(e, "descriptor staging allocation");
        slot = st->next;
        st->next = (st->next + 1) % Staging::kSlots;
        // The slot's last kernel waited for the slot's last copy, so once that
        // kernel is done both the host and the device slot are free. (Waiting
        // on the kernel's event, not on the copy's, keeps the host on the
        // compute queue's completion signal.)
        if (st->pending[slot]) {
            e = hipEventSynchronize(st->ev[slot]);
            if (e != hipSuccess)
                return hip_fail(e, "hipEventSynchronize");
            st->pending[slot] = false;
            st->up_pending[slot] = false;
        }
        uint8_t *h = st->host + (size_t)slot * st->slot_cap;
        uint8_t *dv = st->dev + (size_t)slot * st->slot_cap;
        std::memcpy(h, descs.data() + first, bytes);
        // By default the kernel reads the table from the pinned slot over the
        // bus (one launch per call; measured: 256 ROIs 24.6 against 26.2 us
        // per call, 256 ragged images 52.9 against 53.9, with no slower
        // kernel). The alternatives: a copy kernel on the caller's stream
        // that moves the slot to device memory first (one launch more, about
        // 4 us of GPU time under the tracer), or a DMA copy on the copy
        // stream that the caller's stream waits for, which costs more host
        // time per call than a short kernel takes (34 against 26 us of host
        // time per call for 256 ROIs).
        const int upload = g_upload.load();
        if (upload == 0 || upload == 3) {
            // the kernel reads the pinned slot itself, over the bus: one
            // launch (the slot is reused only after that kernel completes)
            dv = st->host_dev + (size_t)slot * st->slot_cap;
        } else if (upload == 2) {
            const int rc = smol::launch_table_copy(st->host_dev + (size_t)slot * st->slot_cap, dv,
                                                   bytes, stream);
            if (rc != (int)hipSuccess)
                return hip_fail((hipError_t)rc, "descriptor copy kernel");
            info->launches += 1;
        } else {
            e = hipMemcpyAsync(dv, h, bytes, hipMemcpyHostToDevice, st->copy);
            if (e != hipSuccess)
                return hip_fail(e, "hipMemcpyAsync(descriptors)");
            e = hipEventRecord(st->up[slot], st->copy);
            if (e != hipSuccess)
                return hip_fail(e, "hipEventRecord(copy)");
            st->up_pending[slot] = true;
            e = hipStreamWaitEvent(s, st->up[slot], 0);
            if (e != hipSuccess)
                return hip_fail(e, "hipStreamWaitEvent");
        }
        a.table = (const Desc *)dv;
    } else {
        a.table = nullptr;
        a.uni = descs[first];
        a.stride = stride;
    }

    // The slot's event rides on the kernel's own dispatch: a separate event
    // record behind the kernel is a packet of its own, which holds the queue
    // about 5 us before the next dispatch (measured on 256 ROIs per call:
    // 23.2 against 20.3 us per call).
    const int rc = launch(a, pl, stream, st ? (void *)st->ev[slot] : nullptr);
    if (st) {
        if (rc == (int)hipSuccess) {
            st->pending[slot] = true;
        } else {
            // The launch failed, but the table copy enqueued above may still
            // read the slot: its next use waits for an event recorded now.
            e = hipEventRecord(st->ev[slot], s);
            if (e == hipSuccess)
                st->pending[slot] = true;
        }
    }
    if (rc != (int)hipSuccess)
        return hip_fail((hipError_t)rc, "kernel launch");
    info->launches += 1;
    return SMOL_OK;
}

bool is_uniform(const std::vector<Desc> &d, size_t first, size_t count, int nofs,
                int64_t *stride)
{
    *stride = 0;
    if (count <= 1)
        return true;
    const Desc &d0 = d[first];
    const int64_t st = d[first + 1].off[0] - d0.off[0];
    for (size_t i = 0; i < count; ++i) {
        const Desc &x = d[first + i];
        if (x.W != d0.W || x.H != d0.H || x.pitch != d0.pitch || x.rx != d0.rx ||
            x.ry != d0.ry || x.fh != d0.fh)
            return false;
        for (int k = 0; k < nofs; ++k)
            if (x.off[k] != d0.off[k] + (int64_t)i * st)
                return false;
    }
    *stride = st;
    return true;
}

int common_checks(const void *src, int64_t src_bytes, const void *out, int32_t n,
                  const smol_params *p)
{
    int rc = check_params(p);
    if (rc)
        return rc;
    if (n < 0 || n > SMOL_MAX_BATCH)
        return fail(SMOL_ERR_INVALID_ARG, "n = %d outside 0..%d", n, SMOL_MAX_BATCH);
    if (n == 0)
        return SMOL_OK;
    if (!src || !out)
        return fail(SMOL_ERR_INVALID_ARG, "src or out is NULL");
    if (src_bytes < 1)
        return fail(SMOL_ERR_INVALID_ARG, "src_bytes must be positive");
    if (((uintptr_t)out & 15) != 0)
        return fail(SMOL_ERR_INVALID_ARG, "out must be 16-byte aligned");
    return SMOL_OK;
}

}  // namespace

extern "C" {

// RGB batch: the whole image i must lie inside src; its region (ROI or the
// whole image) becomes the descriptor's image.
static int rgb_batch(const uint8_t *src, int64_t src_bytes, const int64_t *offsets,
                     const int32_t *widths, const int32_t *heights, const int32_t *row_pitch,
                     const int32_t *rois, int32_t n, const smol_params *p,
                     const smol_options *opts, void *out, void *stream)
{
    g_last_error.clear();
    int rc = common_checks(src, src_bytes, out, n, p);
    if (rc || n == 0)
        return rc;
    smol_options o;
    rc = check_options(opts, &o);
    if (rc)
        return rc;
    if (!offsets || !widths || !heights)
        return fail(SMOL_ERR_INVALID_ARG, "offsets, widths or heights is NULL");

    std::vector<Desc> descs((size_t)n);
    std::vector<uint8_t> inside((size_t)n);  // every 8-byte source window lies in src
    int64_t max_span = 0;
    // The geometry of a region depends on its size only: the previous
    // image's is reused when the size repeats (a uniform batch computes it
    // once).
    int64_t memo_w = -1, memo_h = -1, memo_xf = 0, memo_xl = 0, memo_yf = 0, memo_yl = 0;
    Geo memo_g{};
    for (int32_t i = 0; i < n; ++i) {
        Geo g;
        const int64_t FW = widths[i], FH = heights[i];
        if (FW < 1 || FH < 1 || FW > SMOL_MAX_DIM || FH > SMOL_MAX_DIM)
            return fail(SMOL_ERR_INVALID_ARG, "image %d: size %lldx%lld outside 1..%d", i,
                        (long long)FW, (long long)FH, SMOL_MAX_DIM);
        const int64_t pitch = row_pitch ? row_pitch[i] : 3 * FW;
        if (pitch < 3 * FW || pitch > INT32_MAX)
            return fail(SMOL_ERR_INVALID_ARG, "image %d: row pitch %lld < 3*width", i,
                        (long long)pitch);
        if (offsets[i] < 0 || offsets[i] > src_bytes ||
            (FH - 1) * pitch + 3 * FW > src_bytes - offsets[i])
            return fail(SMOL_ERR_INVALID_ARG, "image %d: bytes [%lld, +%lld) outside src (%lld)",
                        i, (long long)offsets[i], (long long)((FH - 1) * pitch + 3 * FW),
                        (long long)src_bytes);
        int64_t rx, ry, W, H;
        rc = region(rois, i, FW, FH, &rx, &ry, &W, &H);
        if (rc)
            return rc;
        int64_t xf, xl, yf, yl;
        if (W == memo_w && H == memo_h) {
            g = memo_g;
            xf = memo_xf;
            xl = memo_xl;
            yf = memo_yf;
            yl = memo_yl;
        } else {
            rc = image_geo(W, H, p, o.resize_mode, &g, i);
            if (rc)
                return rc;
            int64_t a, b;
            tap_index(g.left, W, g.Wr, &xf, &a);
            tap_index(g.left + p->crop_w - 1, W, g.Wr, &b, &xl);
            tap_index(g.top, H, g.Hr, &yf, &a);
            tap_index(g.top + p->crop_h - 1, H, g.Hr, &b, &yl);
            memo_w = W;
            memo_h = H;
            memo_g = g;
            memo_xf = xf;
            memo_xl = xl;
            memo_yf = yf;
            memo_yl = yl;
        }
        const int64_t off = offsets[i] + ry * pitch + 3 * rx;  // the region's first pixel
        Desc &d = descs[i];
        std::memset(&d, 0, sizeof d);
        d.off[0] = off;
        d.fh = (int32_t)H;
        d.W = (int32_t)W;
        d.H = (int32_t)H;
        d.pitch = (int32_t)pitch;
        d.Wr = (int32_t)g.Wr;
        d.Hr = (int32_t)g.Hr;
        d.left = (int32_t)g.left;
        d.top = (int32_t)g.top;
        d.xf = (int32_t)xf;
        d.span = (int32_t)std::min<int64_t>(3 * (xl - xf + 1), INT32_MAX);
        {
            // every 16-byte chunk holding a staged byte lies inside src
            const uintptr_t base = (uintptr_t)src + (uintptr_t)off + 3 * (uintptr_t)xf;
            const uintptr_t first = (base + (uintptr_t)yf * (uintptr_t)pitch) & ~(uintptr_t)15;
            const uintptr_t last =
                base + (uintptr_t)yl * (uintptr_t)pitch + 3 * (uintptr_t)(xl - xf + 1);
            const uintptr_t end = (last + 15) & ~(uintptr_t)15;
            d.safe = first >= (uintptr_t)src && end <= (uintptr_t)src + (uintptr_t)src_bytes;
        }
        max_span = std::max(max_span, 3 * (xl - xf + 1));
        inside[i] = off + (H - 1) * pitch + 3 * xl + 8 <= src_bytes;
    }
    // Maximal runs of images whose windows do / do not all lie inside src. In
    // a packed batch only the image that ends at the end of src is outside,
    // so there are one or two runs.
    std::vector<std::pair<size_t, size_t>> runs;  // [begin, end)
    bool any_inside = false;
    for (size_t i = 0; i < (size_t)n; ++i) {
        if (i == 0 || inside[i] != inside[i - 1])
            runs.push_back({i, i});
        runs.back().second = i + 1;
        any_inside = any_inside || inside[i];
    }

    BatchArgs a;
    std::memset(&a, 0, sizeof a);
    a.src = src;
    a.src_bytes = src_bytes;
    a.out = out;
    a.Ch = p->crop_h;
    a.Cw = p->crop_w;
    a.nhwc = o.layout == SMOL_LAYOUT_NHWC;
    fill_norm(p, a);
    // output type: 0 fp32, 1 fp16, 2 uint8 (row-streaming and direct kernels)
    const int f16 = p->out_dtype;
    const bool u8 = p->out_dtype == SMOL_OUT_U8;
    smol_plan info = {};
    const int forced = g_path.load();
    if (a.nhwc && (forced == smol::PATH_LDS || forced == smol::PATH_GATHER))
        return fail(SMOL_ERR_UNSUPPORTED, "NHWC output runs on the row-streaming and direct "
                    "kernels only");
    if (u8 && (forced == smol::PATH_LDS || forced == smol::PATH_GATHER))
        return fail(SMOL_ERR_UNSUPPORTED, "uint8 output runs on the row-streaming and direct "
                    "kernels only");

    auto direct = [f16](const BatchArgs &x, const Plan &, void *s, void *done) {
        return smol::launch_rgb_direct(x, f16, s, done);
    };
    // Register-gather path: the gather kernel for runs of images whose windows
    // lie inside src, the direct kernel for the others.
    // Row-streaming path: the row-streaming kernel for runs of images whose
    // staged chunks lie inside src, the direct kernel for the others.
    {
        int device = 0;
        DeviceInfo di;
        const bool have_dev =
            hipGetDevice(&device) == hipSuccess && device_info(device, &di) == hipSuccess;
        const int col_iters = p->crop_w <= 128 ? 1 : p->crop_w <= 256 ? 2 : 4;
        // A staged row: up to 15 bytes before the span (16-byte aligned
        // chunks), the span, and the 12-byte read of the last column's taps,
        // in groups of 64 chunks (1 KiB).
        const int64_t groups = (max_span + 32 + 1023) / 1024;
        const int64_t lds_bytes = 2 * 1024 * (groups <= 1 ? 1 : groups <= 2 ? 2 : 4);
        const int64_t budget = std::min<int64_t>(
            have_dev ? di.lds_per_block : 65536,
            g_lds_budget.load() > 0 ? g_lds_budget.load() : INT64_MAX);
        bool any_safe = false, runs_ok = true;
        size_t nruns = 0;
        for (int32_t i = 0; i < n; ++i) {
            any_safe = any_safe || descs[(size_t)i].safe;
            nruns += (i == 0 || descs[(size_t)i].safe != descs[(size_t)i - 1].safe) ? 1 : 0;
        }
        runs_ok = nruns <= 3;
        const bool rows_ok = have_dev && p->crop_w <= 128 * smol::kRowsMaxColIters &&
                             groups <= smol::kRowsMaxGroups && lds_bytes <= budget;
        if (forced == smol::PATH_ROWS && !rows_ok)
            return fail(SMOL_ERR_UNSUPPORTED, "row-streaming path forced but the crop width or "
                        "source span does not fit (crop_w <= %d, span + 32 <= %d bytes, "
                        "%lld bytes of LDS)",
                        128 * smol::kRowsMaxColIters, 1024 * smol::kRowsMaxGroups,
                        (long long)lds_bytes);
        if (rows_ok && (forced == smol::PATH_ROWS ||
                        (forced == smol::PATH_AUTO && any_safe && runs_ok))) {
            Plan pr{smol::PATH_ROWS, 0, (size_t)lds_bytes, 0, f16};
            a.col_iters = col_iters;
            a.row_groups = (int)(lds_bytes / 2048);
            // Prefetch depth (band_rows 1 or 2 forces it): long staged rows
            // keep one row in flight per wave, short ones two.
            const int br = g_band_rows.load();
            a.prefetch = br == 1 || br == 2 ? br : a.row_groups >= 4 ? 1 : 2;
            auto rows = [f16](const BatchArgs &x, const Plan &q, void *s, void *done) {
                return smol::launch_rgb_rows(x, f16, q.lds_bytes, s, done);
            };
            auto direct_run = [f16](const BatchArgs &x, const Plan &, void *s, void *done) {
                return smol::launch_rgb_direct(x, f16, s, done);
            };
            for (int32_t b = 0; b < n;) {
                int32_t e = b + 1;
                while (e < n && descs[(size_t)e].safe == descs[(size_t)b].safe)
                    ++e;
                rc = descs[(size_t)b].safe
                         ? run_batch(descs, (size_t)b, (size_t)(e - b), 1, a, pr, stream, rows,
                                     &info)
                         : run_batch(descs, (size_t)b, (size_t)(e - b), 1, a,
                                     Plan{smol::PATH_DIRECT, 0, 0, 0, f16}, stream, direct_run,
                                     &info);
                if (rc)
                    return rc;
                b = e;
            }
            g_last_plan = info;
            return SMOL_OK;
        }
    }

    Plan pg{smol::PATH_GATHER, 0, 0, 0, f16};
    const size_t head = align16((size_t)8 * p->crop_w);
    pg.lds_bytes = head + (size_t)20 * p->crop_h;  // column and row tap tables
    bool gather_fits = false;
    {
        int device = 0;
        DeviceInfo di;
        if (hipGetDevice(&device) == hipSuccess && device_info(device, &di) == hipSuccess)
            gather_fits = pg.lds_bytes <= (size_t)di.lds_per_block;
    }
    if (a.nhwc || u8) {
        rc = run_batch(descs, 0, (size_t)n, 1, a, Plan{smol::PATH_DIRECT, 0, 0, 0, f16}, stream,
                       direct, &info);
        if (!rc)
            g_last_plan = info;
        return rc;
    }
    if (forced == smol::PATH_GATHER ||
        (forced == smol::PATH_AUTO && gather_fits && any_inside && runs.size() <= 3)) {
        a.slots_off = (int)head;
        auto gather = [f16](const BatchArgs &x, const Plan &q, void *s, void *done) {
            return smol::launch_rgb_gather(x, f16, q.lds_bytes, s, done);
        };
        for (const auto &r : runs) {
            const size_t cnt = r.second - r.first;
            rc = inside[r.first]
                     ? run_batch(descs, r.first, cnt, 1, a, pg, stream, gather, &info)
                     : run_batch(descs, r.first, cnt, 1, a, Plan{smol::PATH_DIRECT, 0, 0, 0, f16},
                                 stream, direct, &info);
            if (rc)
                return rc;
        }
        g_last_plan = info;
        return SMOL_OK;
    }
    int slot_bytes = 0, slots_off = 0, stage_bytes = 0;
    Plan pl = plan_rgb(max_span, p->crop_h, p->crop_w, &slot_bytes, &slots_off, &stage_bytes);
    pl.f16 = f16;
    if (forced == smol::PATH_LDS && pl.path != smol::PATH_LDS)
        return fail(SMOL_ERR_UNSUPPORTED, "LDS path forced but the source span does not fit");
    if (pl.path == smol::PATH_LDS) {
        a.R = pl.R;
        a.bands = (p->crop_h + pl.R - 1) / pl.R;
        a.slot_bytes = slot_bytes;
        a.slots_off = slots_off;
        a.stage_bytes = stage_bytes;
    }
    rc = run_batch(descs, 0, (size_t)n, 1, a, pl, stream,
                   [f16](const BatchArgs &x, const Plan &q, void *s, void *done) {
                       return q.path == smol::PATH_LDS
                                  ? smol::launch_rgb_lds(x, f16, q.lds_bytes, s, done)
                                  : smol::launch_rgb_direct(x, f16, s, done);
                   },
                   &info);
    if (!rc)
        g_last_plan = info;
    return rc;
}

// I420 batch: every plane of frame i must lie inside src; the descriptor
// holds the frame's planes and the processed region (ROI or whole frame).
static int yuv_batch(const uint8_t *src, int64_t src_bytes, const int64_t *y_offsets,
                     const int64_t *cb_offsets, const int64_t *cr_offsets, const int32_t *widths,
                     const int32_t *heights, const int32_t *rois, int32_t n, const smol_params *p,
                     const smol_options *opts, void *out, void *stream)
{
    g_last_error.clear();
    int rc = common_checks(src, src_bytes, out, n, p);
    if (rc || n == 0)
        return rc;
    smol_options o;
    rc = check_options(opts, &o);
    if (rc)
        return rc;
    if (!y_offsets || !cb_offsets || !cr_offsets || !widths || !heights)
        return fail(SMOL_ERR_INVALID_ARG, "an offset table, widths or heights is NULL");
    const int left = o.chroma_siting == SMOL_CHROMA_LEFT;

    std::vector<Desc> descs((size_t)n);
    int64_t max_yspan = 0, max_cspan = 0;
    for (int32_t i = 0; i < n; ++i) {
        Geo g;
        const int64_t FW = widths[i], FH = heights[i];
        if (FW < 1 || FH < 1 || FW > SMOL_MAX_DIM || FH > SMOL_MAX_DIM)
            return fail(SMOL_ERR_INVALID_ARG, "frame %d: size %lldx%lld outside 1..%d", i,
                        (long long)FW, (long long)FH, SMOL_MAX_DIM);
        int64_t rx, ry, W, H;
        rc = region(rois, i, FW, FH, &rx, &ry, &W, &H);
        if (rc)
            return rc;
        rc = image_geo(W, H, p, o.resize_mode, &g, i);
        if (rc)
            return rc;
        const int64_t cbytes = ((FW + 1) / 2) * ((FH + 1) / 2);
        const int64_t offs[3] = {y_offsets[i], cb_offsets[i], cr_offsets[i]};
        const int64_t sizes[3] = {FW * FH, cbytes, cbytes};
        for (int k = 0; k < 3; ++k)
            if (offs[k] < 0 || offs[k] > src_bytes || sizes[k] > src_bytes - offs[k])
                return fail(SMOL_ERR_INVALID_ARG, "frame %d: plane %d [%lld, +%lld) outside src",
                            i, k, (long long)offs[k], (long long)sizes[k]);
        Desc &d = descs[i];
        std::memset(&d, 0, sizeof d);
        for (int k = 0; k < 3; ++k)
            d.off[k] = offs[k];
        d.W = (int32_t)W;
        d.H = (int32_t)H;
        d.pitch = (int32_t)FW;
        d.fh = (int32_t)FH;
        d.rx = (int32_t)rx;
        d.ry = (int32_t)ry;
        d.Wr = (int32_t)g.Wr;
        d.Hr = (int32_t)g.Hr;
        d.left = (int32_t)g.left;
        d.top = (int32_t)g.top;
        int64_t xf, xl, c0, c1, e0, e1;
        x_span(d, p->crop_w, &xf, &xl);
        chroma_index(rx + xf, (FW + 1) / 2, &c0, &c1, left);
        chroma_index(rx + xl, (FW + 1) / 2, &e0, &e1, left);
        d.xf = (int32_t)xf;
        d.span = (int32_t)(xl - xf + 1);
        max_yspan = std::max(max_yspan, xl - xf + 1);
        max_cspan = std::max(max_cspan, e1 - c0 + 1);
        // every 16-byte chunk of every plane lies inside src
        bool safe = true;
        for (int k = 0; k < 3; ++k) {
            const uintptr_t b = (uintptr_t)src + (uintptr_t)offs[k];
            safe = safe && (b & ~(uintptr_t)15) >= (uintptr_t)src &&
                   ((b + (uintptr_t)sizes[k] + 15) & ~(uintptr_t)15) <=
                       (uintptr_t)src + (uintptr_t)src_bytes;
        }
        d.safe = safe;
    }
    BatchArgs a;
    std::memset(&a, 0, sizeof a);
    a.src = src;
    a.src_bytes = src_bytes;
    a.out = out;
    a.Ch = p->crop_h;
    a.Cw = p->crop_w;
    a.nhwc = o.layout == SMOL_LAYOUT_NHWC;
    a.siting = left;
    fill_norm(p, a);
    const int forced = g_path.load();
    if (forced == smol::PATH_LDS || forced == smol::PATH_GATHER)
        return fail(SMOL_ERR_UNSUPPORTED, "no LDS-staged or register-gather I420 kernel");
    const int f16 = p->out_dtype == SMOL_OUT_F16;
    smol_plan info = {};
    auto direct = [f16](const BatchArgs &x, const Plan &, void *s, void *done) {
        return smol::launch_yuv_direct(x, f16, s, done);
    };
    if (p->out_dtype == SMOL_OUT_U8) {
        if (forced != smol::PATH_AUTO && forced != smol::PATH_DIRECT)
            return fail(SMOL_ERR_UNSUPPORTED, "uint8 output runs on the direct kernels only");
        rc = run_batch(descs, 0, (size_t)n, 3, a, Plan{smol::PATH_DIRECT, 0, 0, 0, 0}, stream,
                       [](const BatchArgs &x, const Plan &, void *s, void *done) {
                           return smol::launch_yuv_direct(x, SMOL_OUT_U8, s, done);
                       },
                       &info);
        if (!rc)
            g_last_plan = info;
        return rc;
    }
    // Row-streaming kernel: staged luma rows of at most 2 KiB and chroma rows
    // of at most 1 KiB (span + 32 bytes), crops up to 512 columns; frames
    // whose planes' chunks cross an end of src go to the direct kernel.
    const bool rows_ok = p->crop_w <= 128 * smol::kRowsMaxColIters && max_yspan + 32 <= 2048 &&
                         max_cspan + 32 <= 1024;
    if (forced == smol::PATH_ROWS && !rows_ok)
        return fail(SMOL_ERR_UNSUPPORTED, "row-streaming I420 path forced but the crop is wider "
                    "than %d columns, the luma span exceeds 2016 bytes or the chroma span 992",
                    128 * smol::kRowsMaxColIters);
    if (rows_ok && (forced == smol::PATH_ROWS || forced == smol::PATH_AUTO)) {
        a.col_iters = p->crop_w <= 128 ? 1 : p->crop_w <= 256 ? 2 : 4;
        // luma segments of 1 or 2 KiB, six chroma segments of 1 KiB per wave
        a.row_groups = max_yspan + 32 <= 1024 ? 1 : 2;
        const Plan pr{smol::PATH_YUV_ROWS, 0, (size_t)(2 * a.row_groups + 6) * 1024, 0, f16};
        auto rows = [f16](const BatchArgs &x, const Plan &q, void *s, void *done) {
            return smol::launch_yuv_rows(x, f16, q.lds_bytes, s, done);
        };
        for (int32_t b = 0; b < n;) {
            int32_t e = b + 1;
            while (e < n && descs[(size_t)e].safe == descs[(size_t)b].safe)
                ++e;
            rc = descs[(size_t)b].safe
                     ? run_batch(descs, (size_t)b, (size_t)(e - b), 3, a, pr, stream, rows, &info)
                     : run_batch(descs, (size_t)b, (size_t)(e - b), 3, a,
                                 Plan{smol::PATH_DIRECT, 0, 0, 0, f16}, stream, direct, &info);
            if (rc)
                return rc;
            b = e;
        }
        g_last_plan = info;
        return SMOL_OK;
    }
    rc = run_batch(descs, 0, (size_t)n, 3, a, Plan{smol::PATH_DIRECT, 0, 0, 0, f16}, stream,
                   direct, &info);
    if (!rc)
        g_last_plan = info;
    return rc;
}

int smol_image_geometry_ex(int32_t frame_w, int32_t frame_h, int32_t yuv420, const int32_t *roi,
                           const smol_params *p, const smol_options *opts, smol_geometry *g)
{
    g_last_error.clear();
    int rc = check_params(p);
    if (rc)
        return rc;
    smol_options o;
    rc = check_options(opts, &o);
    if (rc)
        return rc;
    if (!g)
        return fail(SMOL_ERR_INVALID_ARG, "geometry output is NULL");
    if (frame_w < 1 || frame_h < 1 || frame_w > SMOL_MAX_DIM || frame_h > SMOL_MAX_DIM)
        return fail(SMOL_ERR_INVALID_ARG, "size %dx%d outside 1..%d", frame_w, frame_h,
                    SMOL_MAX_DIM);
    int64_t rx, ry, rw, rh;
    rc = region(roi, 0, frame_w, frame_h, &rx, &ry, &rw, &rh);
    if (rc)
        return rc;
    const int32_t width = (int32_t)rw, height = (int32_t)rh;
    const int left = o.chroma_siting == SMOL_CHROMA_LEFT;
    Geo geo;
    rc = image_geo(width, height, p, o.resize_mode, &geo, 0);
    if (rc)
        return rc;
    std::memset(g, 0, sizeof *g);
    g->resized_w = (int32_t)geo.Wr;
    g->resized_h = (int32_t)geo.Hr;
    g->crop_left = (int32_t)geo.left;
    g->crop_top = (int32_t)geo.top;
    Desc d;
    std::memset(&d, 0, sizeof d);
    d.W = width;
    d.H = height;
    d.Wr = (int32_t)geo.Wr;
    d.Hr = (int32_t)geo.Hr;
    d.left = (int32_t)geo.left;
    d.top = (int32_t)geo.top;
    int64_t xf, xl;
    x_span(d, p->crop_w, &xf, &xl);
    g->src_x_first = (int32_t)(rx + xf);
    g->src_x_last = (int32_t)(rx + xl);
    g->src_rows = (int32_t)distinct_rows(geo.top, p->crop_h, height, geo.Hr);
    if (yuv420) {
        const int64_t Wc = (frame_w + 1) / 2, Hc = (frame_h + 1) / 2;
        int64_t c0, c1, e0, e1;
        chroma_index(rx + xf, Wc, &c0, &c1, left);
        chroma_index(rx + xl, Wc, &e0, &e1, left);
        g->chroma_x_first = (int32_t)c0;
        g->chroma_x_last = (int32_t)e1;
        // distinct chroma rows over every luma row the vertical taps read
        int64_t count = 0, last = -1;
        for (int64_t r = 0; r < p->crop_h; ++r) {
            int64_t y0, y1;
            tap_index(geo.top + r, height, geo.Hr, &y0, &y1);
            const int64_t ys[2] = {ry + y0, ry + y1};
            for (int k = 0; k < 2; ++k) {
                int64_t a, b;
                chroma_index(ys[k], Hc, &a, &b);
                if (a > last) {
                    ++count;
                    last = a;
                }
                if (b > last) {
                    ++count;
                    last = b;
                }
            }
        }
        g->chroma_rows = (int32_t)count;
    }
    return SMOL_OK;
}

int smol_image_geometry(int32_t width, int32_t height, int32_t yuv420, const smol_params *p,
                        smol_geometry *g)
{
    return smol_image_geometry_ex(width, height, yuv420, nullptr, p, nullptr, g);
}

int smol_preprocess_batch(const uint8_t *src, int64_t src_bytes, const int64_t *offsets,
                          const int32_t *widths, const int32_t *heights,
                          const int32_t *row_pitch, int32_t n, const smol_params *p, void *out,
                          void *stream)
{
    return rgb_batch(src, src_bytes, offsets, widths, heights, row_pitch, nullptr, n, p, nullptr,
                     out, stream);
}

int smol_preprocess_batch_noalloc(const uint8_t *src, int64_t src_bytes, const int64_t *offsets,
                                  const int32_t *widths, const int32_t *heights,
                                  const int32_t *row_pitch, int32_t n, const smol_params *p,
                                  void *out, void *stream)
{
    g_last_error.clear();
    if (n > SMOL_NOALLOC_MAX_IMAGES)
        return fail(SMOL_ERR_UNSUPPORTED, "n = %d exceeds the %d images of the no-allocation "
                    "call's descriptor table", n, SMOL_NOALLOC_MAX_IMAGES);
    struct Scope {
        Scope() { t_noalloc = true; }
        ~Scope() { t_noalloc = false; }
    } scope;
    return rgb_batch(src, src_bytes, offsets, widths, heights, row_pitch, nullptr, n, p, nullptr,
                     out, stream);
}

int smol_preprocess_batch_ex(const uint8_t *src, int64_t src_bytes, const int64_t *offsets,
                             const int32_t *widths, const int32_t *heights,
                             const int32_t *row_pitch, const int32_t *rois, int32_t n,
                             const smol_params *p, const smol_options *opts, void *out,
                             void *stream)
{
    return rgb_batch(src, src_bytes, offsets, widths, heights, row_pitch, rois, n, p, opts, out,
                     stream);
}

int smol_yuv420_preprocess_batch(const uint8_t *src, int64_t src_bytes, const int64_t *y_offsets,
                                 const int64_t *cb_offsets, const int64_t *cr_offsets,
                                 const int32_t *widths, const int32_t *heights, int32_t n,
                                 const smol_params *p, void *out, void *stream)
{
    return yuv_batch(src, src_bytes, y_offsets, cb_offsets, cr_offsets, widths, heights, nullptr,
                     n, p, nullptr, out, stream);
}

int smol_yuv420_preprocess_batch_ex(const uint8_t *src, int64_t src_bytes,
                                    const int64_t *y_offsets, const int64_t *cb_offsets,
                                    const int64_t *cr_offsets, const int32_t *widths,
                                    const int32_t *heights, const int32_t *rois, int32_t n,
                                    const smol_params *p, const smol_options *opts, void *out,
                                    void *stream)
{
    return yuv_batch(src, src_bytes, y_offsets, cb_offsets, cr_offsets, widths, heights, rois, n,
                     p, opts, out, stream);
}

int64_t smol_lowres_workspace_bytes(int32_t n, int32_t low_res)
{
    if (n < 1 || low_res < 1)
        return 0;
    // the images, then 16-byte chunks past the last one so that the second
    // step reads the last image like the others
    return (((int64_t)n * 3 * low_res * low_res + 15) & ~(int64_t)15) + 16;
}

// Low-resolution augmentation, shared checks and the second step: the r x r
// uint8 HWC images packed in the workspace, preprocessed as one uniform
// batch.
static int lowres_check(int32_t n, int32_t low_res, const smol_params *p, const void *workspace,
                        int64_t workspace_bytes, smol_params *lo)
{
    g_last_error.clear();
    int rc = check_params(p);
    if (rc)
        return rc;
    if (p->out_dtype == SMOL_OUT_U8)
        return fail(SMOL_ERR_INVALID_ARG, "the augmented output is normalised: out_dtype must be "
                    "SMOL_OUT_F32 or SMOL_OUT_F16");
    if (low_res < 1 || low_res > SMOL_MAX_DIM)
        return fail(SMOL_ERR_INVALID_ARG, "low_res %d outside 1..%d", low_res, SMOL_MAX_DIM);
    if (n < 0 || n > SMOL_MAX_BATCH)
        return fail(SMOL_ERR_INVALID_ARG, "n = %d outside 0..%d", n, SMOL_MAX_BATCH);
    const int64_t need = smol_lowres_workspace_bytes(n, low_res);
    if (n > 0 && (!workspace || workspace_bytes < need))
        return fail(SMOL_ERR_INVALID_ARG, "workspace of %lld bytes, %lld needed",
                    (long long)workspace_bytes, (long long)need);
    if (((uintptr_t)workspace & 15) != 0)
        return fail(SMOL_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    Geo g;  // the second step's geometry, checked before the first launch
    rc = image_geo(low_res, low_res, p, SMOL_RESIZE_SHORT_CROP, &g, 0);
    if (rc)
        return rc;
    *lo = *p;
    lo->resize_short = low_res;
    lo->crop_h = lo->crop_w = low_res;
    lo->out_dtype = SMOL_OUT_U8;
    return SMOL_OK;
}

static int lowres_upsample(const void *workspace, int64_t workspace_bytes, int32_t n,
                           int32_t low_res, const smol_params *p, void *out, void *stream)
{
    const int launches = g_last_plan.launches;
    std::vector<int64_t> offs((size_t)n);
    std::vector<int32_t> side((size_t)n, low_res);
    const int64_t each = (int64_t)3 * low_res * low_res;
    for (int32_t i = 0; i < n; ++i)
        offs[(size_t)i] = (int64_t)i * each;
    const int rc = rgb_batch((const uint8_t *)workspace, workspace_bytes, offs.data(),
                             side.data(), side.data(), nullptr, nullptr, n, p, nullptr, out,
                             stream);
    if (!rc)
        g_last_plan.launches += launches;
    return rc;
}

int smol_lowres_preprocess_batch(const uint8_t *src, int64_t src_bytes, const int64_t *offsets,
                                 const int32_t *widths, const int32_t *heights,
                                 const int32_t *row_pitch, int32_t n, int32_t low_res,
                                 const smol_params *p, void *workspace, int64_t workspace_bytes,
                                 void *out, void *stream)
{
    smol_params lo;
    int rc = lowres_check(n, low_res, p, workspace, workspace_bytes, &lo);
    if (rc || n == 0)
        return rc;
    const smol_options o = {SMOL_RESIZE_SHORT_CROP, SMOL_LAYOUT_NHWC, SMOL_CHROMA_CENTER, {0}};
    rc = rgb_batch(src, src_bytes, offsets, widths, heights, row_pitch, nullptr, n, &lo, &o,
                   workspace, stream);
    return rc ? rc : lowres_upsample(workspace, workspace_bytes, n, low_res, p, out, stream);
}

int smol_yuv420_lowres_preprocess_batch(const uint8_t *src, int64_t src_bytes,
                                        const int64_t *y_offsets, const int64_t *cb_offsets,
                                        const int64_t *cr_offsets, const int32_t *widths,
                                        const int32_t *heights, int32_t n, int32_t low_res,
                                        const smol_params *p, void *workspace,
                                        int64_t workspace_bytes, void *out, void *stream)
{
    smol_params lo;
    int rc = lowres_check(n, low_res, p, workspace, workspace_bytes, &lo);
    if (rc || n == 0)
        return rc;
    const smol_options o = {SMOL_RESIZE_SHORT_CROP, SMOL_LAYOUT_NHWC, SMOL_CHROMA_CENTER, {0}};
    rc = yuv_batch(src, src_bytes, y_offsets, cb_offsets, cr_offsets, widths, heights, nullptr, n,
                   &lo, &o, workspace, stream);
    return rc ? rc : lowres_upsample(workspace, workspace_bytes, n, low_res, p, out, stream);
}

int smol_set_tuning(const smol_tuning *t)
{
    g_last_error.clear();
    if (!t) {
        g_path = 0;
        g_band_rows = 0;
        g_lds_budget = 0;
        g_wg_per_cu = 0;
        g_exact = 0;
        g_row_order = 0;
        g_upload = 0;
        return SMOL_OK;
    }
    if (t->path < 0 || t->path > 4)
        return fail(SMOL_ERR_INVALID_ARG, "path %d unknown", t->path);
    if (t->band_rows < 0 || t->band_rows > kMaxBandRows)
        return fail(SMOL_ERR_INVALID_ARG, "band_rows %d outside 0..%d", t->band_rows,
                    kMaxBandRows);
    if (t->lds_budget != 0 && (t->lds_budget < 4096 || t->lds_budget > 163840))
        return fail(SMOL_ERR_INVALID_ARG, "lds_budget %d outside 4096..163840", t->lds_budget);

    if (t->workgroups_per_cu < 0 || t->workgroups_per_cu > kMaxWorkgroupsPerCu)
        return fail(SMOL_ERR_INVALID_ARG, "workgroups_per_cu %d outside 0..%d",
                    t->workgroups_per_cu, kMaxWorkgroupsPerCu);
    if (t->exact != 0 && t->exact != 1)
        return fail(SMOL_ERR_INVALID_ARG, "exact %d is neither 0 nor 1", t->exact);
    if (t->row_order < 0 || t->row_order > 2)
        return fail(SMOL_ERR_INVALID_ARG, "row_order %d outside 0..2", t->row_order);
    if (t->upload < 0 || t->upload > 3)
        return fail(SMOL_ERR_INVALID_ARG, "upload %d outside 0..3", t->upload);
    g_path = t->path;
    g_band_rows = t->band_rows;
    g_lds_budget = t->lds_budget;
    g_wg_per_cu = t->workgroups_per_cu;
    g_exact = t->exact;
    g_row_order = t->row_order;
    g_upload = t->upload;
    return SMOL_OK;
}

int smol_last_plan(smol_plan *plan)
{
    if (!plan)
        return SMOL_ERR_INVALID_ARG;
    *plan = g_last_plan;
    return SMOL_OK;
}

const char *smol_status_string(int status)
{
    switch (status) {
    case SMOL_OK:
        return "ok";
    case SMOL_ERR_INVALID_ARG:
        return "invalid argument";
    case SMOL_ERR_UNSUPPORTED:
        return "unsupported by this library";
    case SMOL_ERR_HIP:
        return "HIP runtime error";
    default:
        return "unknown status";
    }
}

const char *smol_last_error(void) { return g_last_error.c_str(); }

int smol_version(void) { return 200; }

}  // extern "C"

int smol::set_error(int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

void smol::clear_error() { g_last_error.clear(); }

int smol::mcu_rect(int64_t W, int64_t H, const smol_params *p, int resize_mode, int32_t rect[4])
{
    // the parameters as the batch calls check them (a zero crop would make
    // the resized size of a direct resize zero)
    int rc = check_params(p);
    if (rc)
        return rc;
    Geo g;
    rc = image_geo(W, H, p, resize_mode, &g, 0);
    if (rc)
        return rc;
    int64_t xf, xl, yf, yl, a, b, c0, c1, d0, d1;
    tap_index(g.left, W, g.Wr, &xf, &a);
    tap_index(g.left + p->crop_w - 1, W, g.Wr, &b, &xl);
    tap_index(g.top, H, g.Hr, &yf, &a);
    tap_index(g.top + p->crop_h - 1, H, g.Hr, &b, &yl);
    // the chroma samples of the first and last luma column and row (centred
    // siting), as luma columns and rows
    chroma_index(xf, (W + 1) / 2, &c0, &a);
    chroma_index(xl, (W + 1) / 2, &a, &c1);
    chroma_index(yf, (H + 1) / 2, &d0, &a);
    chroma_index(yl, (H + 1) / 2, &a, &d1);
    const int64_t x0 = std::min(xf, 2 * c0) / 16 * 16, y0 = std::min(yf, 2 * d0) / 16 * 16;
    const int64_t x1 = (std::max(xl, 2 * c1 + 1) / 16 + 1) * 16;
    const int64_t y1 = (std::max(yl, 2 * d1 + 1) / 16 + 1) * 16;
    rect[0] = (int32_t)x0;
    rect[1] = (int32_t)y0;
    rect[2] = (int32_t)(std::min(x1, W) - x0);
    rect[3] = (int32_t)(std::min(y1, H) - y0);
    return SMOL_OK;
}

void smol::add_plan_launches(int k) { g_last_plan.launches += k; }

namespace smol {
// The workgroups_per_cu knob (0: automatic), read by block decoding's launch
// (smol_jpeg.cpp).
int tuned_workgroups_per_cu() { return g_wg_per_cu.load(); }
}  // namespace smol

int smol::device_cus()
{
    int device = 0;
    DeviceInfo di;
    if (hipGetDevice(&device) != hipSuccess || device_info(device, &di) != hipSuccess)
        return 0;
    return di.cus;
}
