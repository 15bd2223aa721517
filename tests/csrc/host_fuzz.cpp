// Drives the library's host code built with the address and undefined-behaviour
// sanitizers (g++, host_stub.cpp in place of the HIP runtime): the T.81 stream
// parser and entropy decoder on seed JPEG streams and seeded mutations of
// them, and the C ABI's validation and geometry on seeded random arguments.
// Any sanitizer report aborts the process (-fno-sanitize-recover).
//
// usage: host_fuzz SEED MUTATIONS_PER_STREAM ABI_CALLS stream.jpg ...
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <vector>

#include "smol.h"
#include "smol_jpeg.h"

namespace {

long g_decoded = 0;  // streams whose whole-frame entropy decoding succeeded

struct Rng {  // xorshift64*
    uint64_t s;
    explicit Rng(uint64_t seed) : s(seed * 0x9E3779B97F4A7C15ull + 1) {}
    uint64_t next()
    {
        s ^= s >> 12;
        s ^= s << 25;
        s ^= s >> 27;
        return s * 0x2545F4914F6CDD1Dull;
    }
    int64_t range(int64_t lo, int64_t hi) { return lo + (int64_t)(next() % (uint64_t)(hi - lo + 1)); }
    bool coin(int pct) { return (int)(next() % 100) < pct; }
};

std::vector<uint8_t> read_file(const char *path)
{
    std::vector<uint8_t> d;
    FILE *f = fopen(path, "rb");
    if (!f)
        return d;
    int c;
    while ((c = fgetc(f)) != EOF)
        d.push_back((uint8_t)c);
    fclose(f);
    return d;
}

smol_params random_params(Rng &r)
{
    smol_params p;
    const int32_t picks[] = {0, 1, 2, 7, 16, 161, 224, 256, 4096, 70000, -3};
    p.resize_short = r.coin(70) ? (int32_t)r.range(1, 300) : picks[r.next() % 11];
    p.crop_h = r.coin(70) ? (int32_t)r.range(1, p.resize_short > 0 ? p.resize_short : 8)
                          : picks[r.next() % 11];
    p.crop_w = r.coin(70) ? (int32_t)r.range(1, p.resize_short > 0 ? p.resize_short : 8)
                          : picks[r.next() % 11];
    p.out_dtype = r.coin(90) ? (int32_t)r.range(0, 2) : (int32_t)r.range(-2, 9);
    const float odd[] = {0.0f, -1.0f, std::numeric_limits<float>::infinity(),
                         std::numeric_limits<float>::quiet_NaN(), 1e-30f, 1e30f};
    for (int c = 0; c < 3; ++c) {
        p.mean[c] = r.coin(90) ? (float)r.range(0, 255) : odd[r.next() % 6];
        p.std[c] = r.coin(90) ? (float)r.range(1, 90) : odd[r.next() % 6];
    }
    return p;
}

smol_options random_options(Rng &r)
{
    smol_options o;
    std::memset(&o, 0, sizeof o);
    o.resize_mode = r.coin(90) ? (int32_t)r.range(0, 1) : (int32_t)r.range(-3, 5);
    o.layout = r.coin(90) ? (int32_t)r.range(0, 1) : (int32_t)r.range(-3, 5);
    o.chroma_siting = r.coin(90) ? (int32_t)r.range(0, 1) : (int32_t)r.range(-3, 5);
    if (r.coin(5))
        o.reserved[r.next() % 5] = 1;
    return o;
}

int32_t random_dim(Rng &r)
{
    const int32_t picks[] = {0, 1, 2, 3, 15, 16, 17, 65535, 65536, -1, 1 << 30};
    return r.coin(85) ? (int32_t)r.range(1, 2000) : picks[r.next() % 11];
}

// Entropy decoding of one stream: whole frame, a rectangle (frame layout) and
// the rectangle's MCU window, into buffers sized from the stream's own header
// (when it parses) and capped.
void decode_stream(const std::vector<uint8_t> &d, Rng &r)
{
    smol_jpeg_info info;
    const int64_t bytes = (int64_t)d.size();
    const uint8_t *data = d.empty() ? nullptr : d.data();
    int rc = smol_jpeg_read_info(data, bytes, &info);
    if (rc != SMOL_OK || info.width < 1 || info.height < 1 || info.width > 4096 ||
        info.height > 4096)
        return;
    const int64_t full = smol_jpeg_coef_count(info.width, info.height);
    if (full <= 0 || full > (int64_t)64 << 20)
        return;
    std::vector<int16_t> coef((size_t)full);
    std::vector<uint16_t> q(2 * 64);
    const int64_t off = 0, size = bytes, coff = 0;
    if (smol_jpeg_entropy_decode_batch(data, bytes, &off, &size, 1, nullptr, coef.data(), full,
                                       &coff, SMOL_JPEG_COEF_FRAME, q.data(), 1) == SMOL_OK)
        ++g_decoded;
    int32_t rect[4];
    rect[0] = (int32_t)r.range(0, info.width - 1);
    rect[1] = (int32_t)r.range(0, info.height - 1);
    rect[2] = (int32_t)r.range(1, info.width - rect[0]);
    rect[3] = (int32_t)r.range(1, info.height - rect[1]);
    if (r.coin(10))
        rect[r.next() % 4] = (int32_t)r.range(-5, 5000);  // possibly outside the frame
    smol_jpeg_entropy_decode_batch(data, bytes, &off, &size, 1, rect, coef.data(), full, &coff,
                                   SMOL_JPEG_COEF_FRAME, nullptr, 2);
    const int64_t win = smol_jpeg_window_coef_count(info.width, info.height, rect);
    if (win > 0 && win <= full)
        smol_jpeg_entropy_decode_batch(data, bytes, &off, &size, 1, rect, coef.data(), win, &coff,
                                       SMOL_JPEG_COEF_WINDOW, q.data(), 1);
    // a coefficient buffer one element too small must be refused, not overrun
    if (full > 1) {
        std::vector<int16_t> small((size_t)full - 1);
        smol_jpeg_entropy_decode_batch(data, bytes, &off, &size, 1, nullptr, small.data(),
                                       full - 1, &coff, SMOL_JPEG_COEF_FRAME, nullptr, 1);
    }
}

std::vector<uint8_t> mutate(const std::vector<uint8_t> &seed, Rng &r)
{
    std::vector<uint8_t> d = seed;
    const int edits = (int)r.range(1, 8);
    for (int e = 0; e < edits && !d.empty(); ++e) {
        const size_t at = (size_t)r.range(0, (int64_t)d.size() - 1);
        switch (r.next() % 7) {
        case 0: d[at] = (uint8_t)r.next(); break;
        case 1: d[at] ^= (uint8_t)(1u << (r.next() % 8)); break;
        case 2: d[at] = 0xFF; break;                        // a spurious marker prefix
        case 3: d.resize(at); break;                         // truncation
        case 4: d.insert(d.begin() + (long)at, (uint8_t)r.next()); break;
        case 5: d.erase(d.begin() + (long)at); break;
        default:                                             // a restart marker
            if (at + 1 < d.size()) {
                d[at] = 0xFF;
                d[at + 1] = (uint8_t)(0xD0 + r.next() % 8);
            }
        }
    }
    return d;
}

// The C ABI's validation and geometry on random arguments. Device pointers
// are never dereferenced on the host; with no device every call that passes
// validation ends in SMOL_ERR_HIP.
void abi_call(Rng &r)
{
    const int n = (int)r.range(0, 6);
    std::vector<int64_t> off(n + 1), off2(n + 1), off3(n + 1);
    std::vector<int32_t> w(n + 1), h(n + 1), pitch(n + 1), rois(4 * n + 4);
    int64_t src_bytes = r.coin(90) ? r.range(1, (int64_t)1 << 40) : r.range(-5, 5);
    for (int i = 0; i < n; ++i) {
        w[i] = random_dim(r);
        h[i] = random_dim(r);
        off[i] = r.coin(90) ? r.range(0, (int64_t)1 << 32) : r.range(-9, 9);
        off2[i] = off[i] + r.range(-100, 1 << 22);
        off3[i] = off2[i] + r.range(-100, 1 << 22);
        const int64_t packed = 3 * (int64_t)w[i] + r.range(0, 64);
        pitch[i] = r.coin(80) && packed <= INT32_MAX ? (int32_t)packed
                                                     : (int32_t)r.range(-5, 1 << 20);
        for (int k = 0; k < 4; ++k)
            rois[4 * i + k] = r.coin(90) ? (int32_t)r.range(0, 1500) : (int32_t)r.range(-9, 1 << 20);
    }
    smol_params p = random_params(r);
    smol_options o = random_options(r);
    const uint8_t *src = (const uint8_t *)(uintptr_t)(r.coin(95) ? 0x100000 + 16 * r.range(0, 64) : 0);
    void *out = (void *)(uintptr_t)(r.coin(95) ? 0x900000 + 16 * r.range(0, 4) : 0x900001);
    smol_geometry g;
    const int32_t roi1[4] = {rois[0], rois[1], rois[2], rois[3]};
    smol_image_geometry_ex(w[0], h[0], (int32_t)r.range(0, 1), r.coin(50) ? roi1 : nullptr, &p,
                           r.coin(80) ? &o : nullptr, &g);
    int32_t rect[4];
    smol_jpeg_mcu_rect(w[0], h[0], &p, r.coin(80) ? &o : nullptr, rect);
    smol_jpeg_coef_count(w[0], h[0]);
    smol_jpeg_window_coef_count(w[0], h[0], roi1);
    smol_jpeg_workspace_bytes(n, w.data(), h.data());
    smol_lowres_workspace_bytes(n, (int32_t)r.range(-2, 400));
    switch (r.next() % 6) {
    case 0:
        smol_preprocess_batch_ex(src, src_bytes, off.data(), w.data(), h.data(),
                                 r.coin(50) ? pitch.data() : nullptr,
                                 r.coin(50) ? rois.data() : nullptr, n, &p, &o, out, nullptr);
        break;
    case 1:
        smol_yuv420_preprocess_batch_ex(src, src_bytes, off.data(), off2.data(), off3.data(),
                                        w.data(), h.data(), r.coin(50) ? rois.data() : nullptr, n,
                                        &p, &o, out, nullptr);
        break;
    case 2:
        smol_lowres_preprocess_batch(src, src_bytes, off.data(), w.data(), h.data(),
                                     r.coin(50) ? pitch.data() : nullptr, n,
                                     (int32_t)r.range(-2, 300), &p, (void *)0x700000,
                                     r.range(-5, (int64_t)1 << 34), out, nullptr);
        break;
    case 3:
        smol_preprocess_batch_noalloc(src, src_bytes, off.data(), w.data(), h.data(),
                                      r.coin(50) ? pitch.data() : nullptr, n, &p, out, nullptr);
        break;
    case 4: {
        std::vector<uint16_t> q(2 * 64 * (n + 1));
        for (auto &v : q)
            v = (uint16_t)(r.coin(95) ? r.range(1, 255) : r.range(0, 70000));
        smol_jpeg_roi_preprocess_batch((const int16_t *)src, src_bytes / 2, off.data(), q.data(),
                                       (int32_t)r.range(0, n + 1), w.data(), h.data(), n,
                                       (int32_t)r.range(-1, 2), &p, &o, (void *)0x700000,
                                       r.range(-5, (int64_t)1 << 34), out, nullptr);
        break;
    }
    default: {
        smol_tuning t;
        std::memset(&t, 0, sizeof t);
        t.path = (int32_t)r.range(-1, 6);
        t.band_rows = (int32_t)r.range(-1, 70);
        t.workgroups_per_cu = (int32_t)r.range(-1, 20);
        t.exact = (int32_t)r.range(-1, 2);
        t.row_order = (int32_t)r.range(-1, 3);
        t.upload = (int32_t)r.range(-1, 3);
        if (smol_set_tuning(&t) == SMOL_OK)
            smol_preprocess_batch(src, src_bytes, off.data(), w.data(), h.data(), nullptr, n, &p,
                                  out, nullptr);
        smol_set_tuning(nullptr);
    }
    }
    smol_last_error();
}

}  // namespace

int main(int argc, char **argv)
{
    if (argc < 4) {
        fprintf(stderr, "usage: %s SEED MUTATIONS ABI_CALLS stream.jpg ...\n", argv[0]);
        return 2;
    }
    const uint64_t seed = strtoull(argv[1], nullptr, 10);
    const int mutations = atoi(argv[2]), calls = atoi(argv[3]);
    long streams = 0;
    for (int a = 4; a < argc; ++a) {
        const std::vector<uint8_t> d = read_file(argv[a]);
        Rng r(seed * 1000003ull + (uint64_t)a);
        decode_stream(d, r);
        ++streams;
        for (int m = 0; m < mutations; ++m) {
            decode_stream(mutate(d, r), r);
            ++streams;
        }
    }
    Rng r(seed);
    for (int i = 0; i < calls; ++i)
        abi_call(r);
    printf("streams %ld decoded %ld abi_calls %d\n", streams, g_decoded, calls);
    return 0;
}
