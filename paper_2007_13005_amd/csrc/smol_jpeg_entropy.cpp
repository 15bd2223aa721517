// Baseline JPEG entropy decoding on the host: the CPU stage ahead of the
// partial decode of section 6.4 ("ROI decoding", Algorithm 1). Huffman
// decoding is bit-serial, so it stays on the CPU, one image per worker
// thread; its output, int16 coefficient blocks, is what
// smol_jpeg_decode_i420 dequantises and inverse-transforms on the GPU.
//
// Partial decoding: with a rectangle, decoding stops after the last MCU that
// holds one of its blocks, and when the stream has restart intervals, the
// intervals that end before the rectangle's first MCU are skipped by
// scanning for their markers instead of being decoded (DC prediction starts
// afresh at each interval, so nothing before one is needed).
//
// Stream format: ITU-T T.81 (Annex B syntax, Annex C Huffman tables, Annex F
// sequential Huffman decoding).
#include <sched.h>

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <thread>
#include <vector>

#include "smol_internal.h"
#include "smol_jpeg.h"

namespace {

// natural index (row * 8 + column) of the k-th coefficient in zig-zag order
constexpr uint8_t kNatural[64] = {
    0,  1,  8,  16, 9,  2,  3,  10, 17, 24, 32, 25, 18, 11, 4,  5,
    12, 19, 26, 33, 40, 48, 41, 34, 27, 20, 13, 6,  7,  14, 21, 28,
    35, 42, 49, 56, 57, 50, 43, 36, 29, 22, 15, 23, 30, 37, 44, 51,
    58, 59, 52, 45, 38, 31, 39, 46, 53, 60, 61, 54, 47, 55, 62, 63};

constexpr int kLook = 10;  // bits resolved by one table lookup

// A Huffman table for decoding: codes of up to kLook bits resolve through
// `fast` (entry = length << 8 | symbol, 0 = longer code); longer codes
// through the canonical-code bounds: the codes of length l are the
// consecutive values first[l] .. last[l], symbols sym[index[l] + code -
// first[l]].
struct Huff {
    uint16_t fast[1 << kLook];
    // A code and the value bits that follow it, both within kLook bits,
    // resolved at once: the value, the zero run before it and the bits used
    // (0: not resolvable this way). Symbol 0 (AC: end of block; DC:
    // difference 0) has run 0xFF. DC tables use the entries of run 0 and
    // 0xFF (their symbols are categories).
    struct Ac {
        int16_t value;
        uint8_t run, bits;
    } fast_ac[1 << kLook];
    int32_t first[17], last[17], index[17];
    uint8_t sym[256];
    bool present = false;
};

bool build_huff(Huff &h, const uint8_t *counts, const uint8_t *symbols, int nsym)
{
    std::memset(h.fast, 0, sizeof h.fast);
    std::memcpy(h.sym, symbols, (size_t)nsym);
    int32_t code = 0;
    int k = 0;
    for (int l = 1; l <= 16; ++l) {
        h.first[l] = code;
        h.index[l] = k;
        for (int i = 0; i < counts[l - 1]; ++i, ++k, ++code) {
            if (code >= (1 << l))
                return false;  // not a prefix code
            if (l <= kLook) {
                const int shift = kLook - l;
                for (int j = 0; j < (1 << shift); ++j)
                    h.fast[(code << shift) | j] = (uint16_t)(l << 8 | symbols[k]);
            }
        }
        h.last[l] = code - 1;  // < first[l]: no codes of this length
        code <<= 1;
    }
    // a code of length l for symbol (run, size), size > 0, followed by its
    // size value bits: entries whose lookahead holds both
    for (int e = 0; e < (1 << kLook); ++e) {
        h.fast_ac[e] = {0, 0, 0};
        const int l = h.fast[e] >> 8, rs = h.fast[e] & 0xFF, size = rs & 15;
        if (l != 0 && rs == 0x00) {
            h.fast_ac[e] = {0, 0xFF, (uint8_t)l};
            continue;
        }
        if (l == 0 || size == 0 || l + size > kLook)
            continue;
        int32_t v = (e >> (kLook - l - size)) & ((1 << size) - 1);
        if (v < (1 << (size - 1)))
            v -= (1 << size) - 1;
        h.fast_ac[e] = {(int16_t)v, (uint8_t)(rs >> 4), (uint8_t)(l + size)};
    }
    h.present = true;
    return k == nsym;
}

// Entropy-coded bits, most significant first, in a 64-bit window. Stuffed
// zero bytes after 0xFF are dropped; at a marker (or the end of the data)
// zero bytes are fed instead and counted, so that decoding past the real
// bits is detected.
struct Bits {
    const uint8_t *p, *end;
    uint64_t buf = 0;
    int n = 0;          // valid bits in buf
    int fed = 0;        // zero bytes fed after a marker or the end
    bool stop = false;  // at a marker or the end

    void fill()
    {
        // whole bytes at once while the next eight hold no 0xFF
        if (!stop && n <= 56 && end - p >= 8) {
            uint64_t w;
            std::memcpy(&w, p, 8);
            const uint64_t x = ~w;  // a zero byte where w has 0xFF
            if (((x - 0x0101010101010101ULL) & ~x & 0x8080808080808080ULL) == 0) {
                const int take = (64 - n) >> 3;
                const uint64_t big = __builtin_bswap64(w) >> n;
                const int low = 64 - n - 8 * take;  // bits below the new bytes
                buf |= low ? big & (~0ULL << low) : big;
                p += take;
                n += 8 * take;
                return;
            }
        }
        while (n <= 56) {
            uint32_t b = 0;
            if (!stop) {
                if (p < end && *p != 0xFF) {
                    b = *p++;
                } else if (p + 1 < end && p[1] == 0x00) {
                    b = 0xFF;
                    p += 2;
                } else {
                    stop = true;
                }
            }
            if (stop)
                ++fed;
            buf |= (uint64_t)b << (56 - n);
            n += 8;
        }
    }
    void skip(int k)
    {
        buf <<= k;
        n -= k;
    }
    // true when bits fed after a marker have been consumed
    bool overrun() const { return fed * 8 > n; }
};

inline int decode(Bits &s, const Huff &h)
{
    if (s.n < 16)
        s.fill();
    const uint16_t e = h.fast[s.buf >> (64 - kLook)];
    if (e) {
        s.skip(e >> 8);
        return e & 0xFF;
    }
    const int32_t code16 = (int32_t)(s.buf >> 48);
    for (int l = kLook + 1; l <= 16; ++l) {
        const int32_t c = code16 >> (16 - l);
        if (c <= h.last[l] && c >= h.first[l]) {
            s.skip(l);
            return h.sym[h.index[l] + c - h.first[l]];
        }
    }
    return -1;
}

// the next t bits as T.81's signed magnitude category t value
inline int32_t receive(Bits &s, int t)
{
    if (t == 0)
        return 0;
    if (s.n < t)
        s.fill();
    int32_t v = (int32_t)(s.buf >> (64 - t));
    s.skip(t);
    return v < (1 << (t - 1)) ? v - (1 << t) + 1 : v;
}

struct Header {
    int32_t W = 0, H = 0, restart = 0;
    int64_t scan = 0;  // first byte of the entropy-coded data
    uint16_t q[2][64];
    int dc_tab[3], ac_tab[3];
    Huff dc[4], ac[4];
};

struct Failure {
    int code = SMOL_OK;
    std::string msg;
};

int fail(Failure &f, int code, const char *fmt, ...)
{
    char buf[256];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    f.code = code;
    f.msg = buf;
    return code;
}

inline int u16be(const uint8_t *p) { return p[0] << 8 | p[1]; }

// Markers up to and including SOS; `huff` false skips building the Huffman
// tables (header queries).
int parse_header(const uint8_t *d, int64_t n, Header &h, bool huff, Failure &f)
{
    if (n < 4 || d[0] != 0xFF || d[1] != 0xD8)
        return fail(f, SMOL_ERR_INVALID_ARG, "no SOI marker");
    uint8_t qraw[4][64];
    bool qok[4] = {false, false, false, false};
    int qsel[3] = {0, 0, 0}, ids[3] = {0, 0, 0};
    bool sof = false;
    int64_t p = 2;
    for (;;) {
        if (p >= n || d[p] != 0xFF)
            return fail(f, SMOL_ERR_INVALID_ARG, "expected a marker at byte %lld", (long long)p);
        while (p < n && d[p] == 0xFF)
            ++p;
        if (p + 3 > n)
            return fail(f, SMOL_ERR_INVALID_ARG, "stream ends inside the headers");
        const int m = d[p++];
        if (m == 0xD8 || m == 0xD9 || (m >= 0xD0 && m <= 0xD7) || m == 0x01)
            return fail(f, SMOL_ERR_INVALID_ARG, "marker 0x%02X before the scan", m);
        const int len = u16be(d + p);
        if (len < 2 || p + len > n)
            return fail(f, SMOL_ERR_INVALID_ARG, "segment 0x%02X: bad length", m);
        const uint8_t *s = d + p + 2;
        const int body = len - 2;
        const int64_t next = p + len;
        switch (m) {
        case 0xDB:  // quantisation tables
            for (int o = 0; o < body;) {
                const int pq = s[o] >> 4, tq = s[o] & 15;
                if (tq > 3)
                    return fail(f, SMOL_ERR_INVALID_ARG, "quantisation table id %d", tq);
                if (pq != 0)
                    return fail(f, SMOL_ERR_UNSUPPORTED, "16-bit quantisation tables");
                if (o + 65 > body)
                    return fail(f, SMOL_ERR_INVALID_ARG, "quantisation table cut short");
                std::memcpy(qraw[tq], s + o + 1, 64);
                qok[tq] = true;
                o += 65;
            }
            break;
        case 0xC4:  // Huffman tables
            for (int o = 0; o < body;) {
                if (o + 17 > body)
                    return fail(f, SMOL_ERR_INVALID_ARG, "Huffman table cut short");
                const int tc = s[o] >> 4, th = s[o] & 15;
                int cnt = 0;
                for (int i = 0; i < 16; ++i)
                    cnt += s[o + 1 + i];
                if (tc > 1 || th > 3 || cnt > 256 || o + 17 + cnt > body)
                    return fail(f, SMOL_ERR_INVALID_ARG, "bad Huffman table");
                if (huff && !build_huff(tc ? h.ac[th] : h.dc[th], s + o + 1, s + o + 17, cnt))
                    return fail(f, SMOL_ERR_INVALID_ARG, "Huffman code lengths overflow");
                if (!huff)
                    (tc ? h.ac[th] : h.dc[th]).present = true;
                o += 17 + cnt;
            }
            break;
        case 0xDD:  // restart interval
            if (body != 2)
                return fail(f, SMOL_ERR_INVALID_ARG, "bad DRI segment");
            h.restart = u16be(s);
            break;
        case 0xC0:
        case 0xC1:  // baseline / extended sequential, Huffman
            if (body < 6 || s[0] != 8)
                return fail(f, SMOL_ERR_UNSUPPORTED, "sample precision other than 8 bits");
            if (s[5] != 3 || body != 15)
                return fail(f, SMOL_ERR_UNSUPPORTED, "%d components (3 needed)", s[5]);
            h.H = u16be(s + 1);
            h.W = u16be(s + 3);
            if (h.W < 1 || h.H < 1)
                return fail(f, SMOL_ERR_UNSUPPORTED, "size %dx%d (DNL not supported)", h.W, h.H);
            for (int c = 0; c < 3; ++c) {
                ids[c] = s[6 + 3 * c];
                qsel[c] = s[8 + 3 * c];
                if (s[7 + 3 * c] != (c == 0 ? 0x22 : 0x11))
                    return fail(f, SMOL_ERR_UNSUPPORTED, "sampling other than 4:2:0");
                if (qsel[c] > 3)
                    return fail(f, SMOL_ERR_INVALID_ARG, "quantisation table id %d", qsel[c]);
            }
            if (qsel[1] != qsel[2])
                return fail(f, SMOL_ERR_UNSUPPORTED, "Cb and Cr on different tables");
            sof = true;
            break;
        case 0xDA: {  // start of scan
            if (!sof)
                return fail(f, SMOL_ERR_INVALID_ARG, "scan before the frame header");
            if (body != 10 || s[0] != 3)
                return fail(f, SMOL_ERR_UNSUPPORTED, "scan of other than 3 interleaved "
                            "components");
            if (s[7] != 0 || s[8] != 63 || s[9] != 0)
                return fail(f, SMOL_ERR_UNSUPPORTED, "spectral selection or approximation");
            for (int c = 0; c < 3; ++c) {
                if (s[1 + 2 * c] != ids[c])
                    return fail(f, SMOL_ERR_UNSUPPORTED, "scan components out of frame order");
                h.dc_tab[c] = s[2 + 2 * c] >> 4;
                h.ac_tab[c] = s[2 + 2 * c] & 15;
                if (h.dc_tab[c] > 3 || h.ac_tab[c] > 3 || !h.dc[h.dc_tab[c]].present ||
                    !h.ac[h.ac_tab[c]].present)
                    return fail(f, SMOL_ERR_INVALID_ARG, "scan names a missing Huffman table");
            }
            for (int t = 0; t < 2; ++t) {
                const int id = qsel[t];
                if (!qok[id])
                    return fail(f, SMOL_ERR_INVALID_ARG, "missing quantisation table %d", id);
                for (int k = 0; k < 64; ++k) {
                    if (qraw[id][k] == 0)
                        return fail(f, SMOL_ERR_INVALID_ARG, "quantisation table entry 0");
                    h.q[t][kNatural[k]] = qraw[id][k];
                }
            }
            h.scan = next;
            return SMOL_OK;
        }
        default:
            if ((m >= 0xC2 && m <= 0xCF) && m != 0xC4 && m != 0xC8 && m != 0xCC)
                return fail(f, SMOL_ERR_UNSUPPORTED, "frame type 0x%02X (progressive, "
                            "lossless or arithmetic coding)", m);
            break;  // APPn, COM and the like
        }
        p = next;
    }
}

// Position just past the k-th restart marker (k >= 1) after `from`, or -1.
int64_t find_restart(const uint8_t *d, int64_t n, int64_t from, int64_t k)
{
    int64_t p = from;
    while (k > 0) {
        const void *hit = std::memchr(d + p, 0xFF, (size_t)(n - p));
        if (!hit)
            return -1;
        p = (const uint8_t *)hit - d;
        if (p + 1 >= n)
            return -1;
        const uint8_t nx = d[p + 1];
        if (nx >= 0xD0 && nx <= 0xD7) {
            --k;
            p += 2;
        } else if (nx == 0xFF) {
            p += 1;  // fill byte
        } else if (nx == 0x00) {
            p += 2;  // stuffed byte
        } else {
            return -1;  // another marker: the scan ended
        }
    }
    return p;
}

// Decode one stream's coefficients into `coef` (the library's layout). With
// `rect`, only MCUs up to the last one holding its blocks are decoded, and
// only blocks of the MCU columns and rows it spans are stored.
int decode_image(const uint8_t *d, int64_t n, const int32_t *rect, bool window, int16_t *coef,
                 int64_t coef_room, uint16_t *q_out, Failure &f)
{
    Header h;
    int rc = parse_header(d, n, h, true, f);
    if (rc)
        return rc;
    if (q_out)
        std::memcpy(q_out, h.q, sizeof h.q);
    const int64_t mx = (h.W + 15) / 16, my = (h.H + 15) / 16;
    int64_t x0 = 0, x1 = mx - 1, y0 = 0, y1 = my - 1;
    if (rect) {
        if (rect[0] < 0 || rect[1] < 0 || rect[2] < 1 || rect[3] < 1 ||
            (int64_t)rect[0] + rect[2] > h.W || (int64_t)rect[1] + rect[3] > h.H)
            return fail(f, SMOL_ERR_INVALID_ARG, "rectangle outside the %dx%d frame", h.W, h.H);
        x0 = rect[0] / 16;
        x1 = ((int64_t)rect[0] + rect[2] - 1) / 16;
        y0 = rect[1] / 16;
        y1 = ((int64_t)rect[1] + rect[3] - 1) / 16;
    }
    const int64_t first = y0 * mx + x0, last = y1 * mx + x1;
    // the stored MCU grid: the whole frame or the rectangle's window
    const int64_t gx0 = window ? x0 : 0, gy0 = window ? y0 : 0;
    const int64_t gmx = window ? x1 - x0 + 1 : mx, gmy = window ? y1 - y0 + 1 : my;
    if (coef_room < 64 * 6 * gmx * gmy)
        return fail(f, SMOL_ERR_INVALID_ARG, "coefficients of a %dx%d frame outside coef", h.W,
                    h.H);
    int16_t *planes[3] = {coef, coef + 64 * 4 * gmx * gmy, coef + 64 * 5 * gmx * gmy};
    const Huff *dct[3], *act[3];
    for (int c = 0; c < 3; ++c) {
        dct[c] = &h.dc[h.dc_tab[c]];
        act[c] = &h.ac[h.ac_tab[c]];
    }
    // start at the interval holding the first MCU needed
    int64_t start = 0, pos = h.scan;
    if (h.restart > 0 && first >= h.restart) {
        const int64_t skip = first / h.restart;
        pos = find_restart(d, n, pos, skip);
        if (pos < 0)
            return fail(f, SMOL_ERR_INVALID_ARG, "restart marker %lld not found",
                        (long long)skip);
        if (d[pos - 1] != 0xD0 + (skip - 1) % 8)
            return fail(f, SMOL_ERR_INVALID_ARG, "restart markers out of sequence");
        start = skip * h.restart;
    }
    Bits s{d + pos, d + n};
    int32_t pred[3] = {0, 0, 0};
    int16_t scratch[64];
    for (int64_t mcu = start; mcu <= last; ++mcu) {
        if (h.restart > 0 && mcu % h.restart == 0 && mcu != start) {
            // end of an interval: the rest of the byte is padding, every
            // whole byte left in the window must be a fed zero, then RSTm
            if (s.n % 8)
                s.skip(s.n % 8);
            if (s.n / 8 != s.fed)
                return fail(f, SMOL_ERR_INVALID_ARG, "data before restart marker at MCU %lld",
                            (long long)mcu);
            const uint8_t *p = s.p;
            while (p + 1 < s.end && p[0] == 0xFF && p[1] == 0xFF)
                ++p;
            const int want = 0xD0 + (int)((mcu / h.restart - 1) % 8);
            if (p + 1 >= s.end || p[0] != 0xFF || p[1] != want)
                return fail(f, SMOL_ERR_INVALID_ARG, "missing restart marker at MCU %lld",
                            (long long)mcu);
            s = Bits{p + 2, s.end};
            pred[0] = pred[1] = pred[2] = 0;
        }
        const int64_t r = mcu / mx, c0 = mcu % mx;
        const bool keep = r >= y0 && r <= y1 && c0 >= x0 && c0 <= x1;
        for (int b = 0; b < 6; ++b) {
            const int c = b < 4 ? 0 : b - 3;
            int16_t *z = scratch;
            if (keep) {
                const int64_t gr = r - gy0, gc = c0 - gx0;
                z = c == 0 ? planes[0] + 64 * ((2 * gr + (b >> 1)) * 2 * gmx + 2 * gc + (b & 1))
                           : planes[c] + 64 * (gr * gmx + gc);
            }
            std::memset(z, 0, 64 * sizeof(int16_t));
            if (s.n < 32)
                s.fill();
            const Huff::Ac &fd = dct[c]->fast_ac[s.buf >> (64 - kLook)];
            if (fd.bits && (fd.run == 0 || fd.run == 0xFF)) {
                s.skip(fd.bits);  // a DC difference resolved at once
                pred[c] += fd.run == 0xFF ? 0 : fd.value;
            } else {
                const int t = decode(s, *dct[c]);
                if (t < 0 || t > 11)
                    return fail(f, SMOL_ERR_INVALID_ARG, "bad DC code at MCU %lld",
                                (long long)mcu);
                pred[c] += receive(s, t);
            }
            if (pred[c] < -32768 || pred[c] > 32767)
                return fail(f, SMOL_ERR_INVALID_ARG, "DC value out of range at MCU %lld",
                            (long long)mcu);
            z[0] = (int16_t)pred[c];
            const Huff &ac = *act[c];
            for (int k = 1; k < 64;) {
                if (s.n < 32)
                    s.fill();
                const Huff::Ac &fa = ac.fast_ac[s.buf >> (64 - kLook)];
                if (fa.bits) {
                    if (fa.run == 0xFF) {
                        s.skip(fa.bits);
                        break;  // end of block
                    }
                    k += fa.run;
                    if (k > 63)
                        return fail(f, SMOL_ERR_INVALID_ARG, "AC run past the block at MCU "
                                    "%lld", (long long)mcu);
                    z[kNatural[k]] = fa.value;
                    s.skip(fa.bits);
                    ++k;
                    continue;
                }
                const int rs = decode(s, ac);
                if (rs < 0)
                    return fail(f, SMOL_ERR_INVALID_ARG, "bad AC code at MCU %lld",
                                (long long)mcu);
                const int size = rs & 15, run = rs >> 4;
                if (size == 0) {
                    if (run != 15)
                        break;  // end of block
                    k += 16;
                    continue;
                }
                k += run;
                if (k > 63 || size > 10)
                    return fail(f, SMOL_ERR_INVALID_ARG, "AC run past the block at MCU %lld",
                                (long long)mcu);
                z[kNatural[k]] = (int16_t)receive(s, size);
                ++k;
            }
        }
        if (s.overrun())
            return fail(f, SMOL_ERR_INVALID_ARG, "stream ends inside MCU %lld", (long long)mcu);
    }
    return SMOL_OK;
}

// CPUs this process may run on (its affinity mask), else the hardware's.
int usable_cpus()
{
    cpu_set_t set;
    if (sched_getaffinity(0, sizeof set, &set) == 0) {
        const int k = CPU_COUNT(&set);
        if (k > 0)
            return k;
    }
    const unsigned hw = std::thread::hardware_concurrency();
    return hw ? (int)hw : 1;
}

}  // namespace

extern "C" {

int smol_jpeg_read_info(const uint8_t *data, int64_t bytes, smol_jpeg_info *info)
{
    smol::clear_error();
    if (!data || !info || bytes < 0)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "data or info is NULL, or bytes < 0");
    Header h;
    Failure f;
    if (parse_header(data, bytes, h, false, f))
        return smol::set_error(f.code, "%s", f.msg.c_str());
    std::memset(info, 0, sizeof *info);
    info->width = h.W;
    info->height = h.H;
    info->restart_interval = h.restart;
    info->scan_offset = h.scan;
    std::memcpy(info->qtables, h.q, sizeof h.q);
    return SMOL_OK;
}

int smol_jpeg_entropy_decode_batch(const uint8_t *data, int64_t data_bytes,
                                   const int64_t *offsets, const int64_t *sizes, int32_t n,
                                   const int32_t *rects, int16_t *coef, int64_t coef_elems,
                                   const int64_t *coef_offsets, int32_t coef_layout,
                                   uint16_t *qtables, int32_t threads)
{
    smol::clear_error();
    if (n < 0 || n > SMOL_MAX_BATCH)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "n = %d outside 0..%d", n, SMOL_MAX_BATCH);
    if (n == 0)
        return SMOL_OK;
    if (!data || !offsets || !sizes || !coef || !coef_offsets)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "a NULL pointer or table");
    if (coef_layout != SMOL_JPEG_COEF_FRAME && coef_layout != SMOL_JPEG_COEF_WINDOW)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "coef_layout %d unknown", coef_layout);
    if (coef_layout == SMOL_JPEG_COEF_WINDOW && !rects)
        return smol::set_error(SMOL_ERR_INVALID_ARG, "the window layout needs rects");
    for (int32_t i = 0; i < n; ++i) {
        if (offsets[i] < 0 || sizes[i] < 0 || offsets[i] > data_bytes ||
            sizes[i] > data_bytes - offsets[i])
            return smol::set_error(SMOL_ERR_INVALID_ARG, "image %d: stream outside data", i);
        if (coef_offsets[i] < 0 || coef_offsets[i] > coef_elems)
            return smol::set_error(SMOL_ERR_INVALID_ARG, "image %d: coefficient offset outside "
                                   "coef", i);
    }
    int t = threads > 0 ? threads : usable_cpus();
    t = std::max(1, std::min({t, (int)n, 256}));
    std::vector<Failure> fails((size_t)n);
    std::atomic<int32_t> next{0};
    auto work = [&]() {
        for (int32_t i; (i = next.fetch_add(1)) < n;)
            decode_image(data + offsets[i], sizes[i], rects ? rects + 4 * (size_t)i : nullptr,
                         coef_layout == SMOL_JPEG_COEF_WINDOW, coef + coef_offsets[i],
                         coef_elems - coef_offsets[i],
                         qtables ? qtables + 128 * (size_t)i : nullptr, fails[(size_t)i]);
    };
    if (t == 1) {
        work();
    } else {
        std::vector<std::thread> pool;
        pool.reserve((size_t)t - 1);
        try {
            for (int k = 1; k < t; ++k)
                pool.emplace_back(work);
        } catch (...) {
            // fewer threads than asked: the running ones finish the batch
        }
        work();
        for (auto &th : pool)
            th.join();
    }
    for (int32_t i = 0; i < n; ++i)
        if (fails[(size_t)i].code)
            return smol::set_error(fails[(size_t)i].code, "image %d: %s", i,
                                   fails[(size_t)i].msg.c_str());
    return SMOL_OK;
}

}  // extern "C"
