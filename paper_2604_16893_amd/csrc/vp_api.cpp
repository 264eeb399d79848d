// vp_api.cpp -- host side of the C ABI declared in include/vp.h.
//
// Host work per call: validate the items, derive grid_thw / cu_seqlens,
// build the per-axis filter tables (double precision, rounded once to
// float), pack the plan into one blob in pinned host memory, copy it into
// the caller's workspace on the caller's stream, and launch the kernels.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstring>
#include <algorithm>
#include <list>
#include <array>
#include <map>
#include <memory>
#include <tuple>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "vp.h"
#include "vp_plan.h"

namespace {

thread_local std::string g_last_error;
thread_local hipEvent_t g_timing_start = nullptr;   // vp_set_kernel_events, one call
thread_local hipEvent_t g_timing_stop = nullptr;

int32_t fail(int32_t status, const std::string& msg) {
    g_last_error = msg;
    return status;
}

// ---------------------------------------------------------------------------
// smart_resize and frame-index sampling
// ---------------------------------------------------------------------------

// Nearest integer of a double, ties to the even neighbour.
double nearest_even(double v) {
    const double lower = std::floor(v);
    const double frac = v - lower;  // exact for |v| < 2^52
    if (frac != 0.5) return frac < 0.5 ? lower : lower + 1.0;
    return std::fmod(lower, 2.0) == 0.0 ? lower : lower + 1.0;
}

// Index i of n spread evenly over [0, last], rounded half to even on the
// exact rational i * last / (n - 1).
int32_t spread_index(int64_t i, int64_t last, int64_t n) {
    if (n == 1) return 0;
    const int64_t num = i * last, den = n - 1;
    int64_t whole = num / den;
    const int64_t twice_rem = 2 * (num - whole * den);
    if (twice_rem > den || (twice_rem == den && (whole & 1))) ++whole;
    return static_cast<int32_t>(whole);
}

// ---------------------------------------------------------------------------
// Antialiased bicubic filter tables
// ---------------------------------------------------------------------------

struct AxisFilter {
    int32_t n_in = 0, n_out = 0, taps = 0;
    std::vector<int32_t> start, count;
    std::vector<float> weight;   // [n_out][taps]
    std::vector<int32_t> fixed;  // [n_out][taps]: the double weights times 2^22, rounded
};

// Keys (1981) kernel, a = -1/2, evaluated as the polynomial is written
// (left to right, no reassociation): the fixed-point weights of the uint8
// writer are rounded from these doubles, so every machine must get the same
// bits.
double cubic_a_half(double x) {
    const double t = std::fabs(x);
    if (t < 1.0) return 1.5 * t * t * t - 2.5 * t * t + 1.0;
    if (t < 2.0) return -0.5 * t * t * t + 2.5 * t * t - 4.0 * t + 2.0;
    return 0.0;
}

// Window [lo, hi) of output i; the same double expressions as the documented
// definition, in the same order, so that window bounds are reproducible.
void window(int32_t n_in, int32_t n_out, int32_t i, double* centre, double* sigma, int32_t* lo,
            int32_t* hi) {
    const double scale = static_cast<double>(n_in) / static_cast<double>(n_out);
    const double s = scale > 1.0 ? scale : 1.0;
    const double support = 2.0 * s;
    const double c = (static_cast<double>(i) + 0.5) * scale;
    double a = std::floor(c - support + 0.5);
    double b = std::floor(c + support + 0.5);
    if (a < 0.0) a = 0.0;
    if (b > n_in) b = n_in;
    *centre = c;
    *sigma = s;
    *lo = static_cast<int32_t>(a);
    *hi = static_cast<int32_t>(b);
}

int32_t axis_taps(int32_t n_in, int32_t n_out) {
    int32_t best = 0;
    for (int32_t i = 0; i < n_out; ++i) {
        double c, s;
        int32_t lo, hi;
        window(n_in, n_out, i, &c, &s, &lo, &hi);
        if (hi - lo > best) best = hi - lo;
    }
    return best;
}

void build_axis(int32_t n_in, int32_t n_out, int32_t taps, AxisFilter* f) {
    f->n_in = n_in;
    f->n_out = n_out;
    f->taps = taps;
    f->start.assign(n_out, 0);
    f->count.assign(n_out, 0);
    f->weight.assign(static_cast<size_t>(n_out) * taps, 0.0f);
    f->fixed.assign(static_cast<size_t>(n_out) * taps, 0);
    std::vector<double> raw(taps);
    for (int32_t i = 0; i < n_out; ++i) {
        double c, s;
        int32_t lo, hi;
        window(n_in, n_out, i, &c, &s, &lo, &hi);
        double sum = 0.0;
        for (int32_t j = lo; j < hi; ++j) {
            raw[j - lo] = cubic_a_half((static_cast<double>(j) + 0.5 - c) / s);
            sum += raw[j - lo];
        }
        f->start[i] = lo;
        f->count[i] = hi - lo;
        for (int32_t j = lo; j < hi; ++j) {
            const double w = raw[j - lo] / sum;
            f->weight[static_cast<size_t>(i) * taps + (j - lo)] = static_cast<float>(w);
            const double x = w * 4194304.0;   // 2^22
            f->fixed[static_cast<size_t>(i) * taps + (j - lo)] =
                static_cast<int32_t>(x < 0.0 ? x - 0.5 : x + 0.5);   // half away from zero
        }
    }
}

// ---------------------------------------------------------------------------
// Plan
// ---------------------------------------------------------------------------

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct Plan {
    std::vector<vp::DevItem> items;
    std::vector<int32_t> prefix;
    std::vector<int32_t> indices;
    // the tables section: cached table words, each placed at its word offset
    std::vector<std::pair<int32_t, std::shared_ptr<const std::vector<int32_t>>>> tables;
    size_t table_words = 0;
    std::vector<vp::StreamUnit> units;
    std::vector<uint32_t> wgs;   // streaming workgroups: unit | band << 20, grouped per launch
    std::vector<vp::StreamLaunch> launches;
    std::vector<int32_t> grid;  // [n][3]
    std::vector<int32_t> cu;    // [n + 1]
    int64_t total_rows = 0;
    std::vector<int64_t> byte_off;   // uint8 writer: [n + 1] output byte offsets of the items
    int64_t generic_cost = 0;   // source pixels the general kernel reads, roughly
    size_t off_items = 0, off_prefix = 0, off_indices = 0, off_tables = 0, off_units = 0, off_wgs = 0,
           bytes = 0;
};

int32_t item_patch(const vp_item& it) { return it.patch == 0 ? vp::kPatch : it.patch; }

// Every item of one call must share one patch size (the rows of one output
// buffer have one width).
int32_t batch_patch(const vp_item* items, int32_t n, int32_t* patch) {
    *patch = vp::kPatch;
    if (items == nullptr || n < 1) return VP_OK;   // reported by the caller's own checks
    *patch = item_patch(items[0]);
    for (int32_t b = 1; b < n; ++b)
        if (item_patch(items[b]) != *patch)
            return fail(VP_ERR_ARG, "items of one call must share one patch size (item " +
                                        std::to_string(b) + ")");
    return VP_OK;
}

int32_t validate_item(const vp_item& it, int32_t b) {
    const std::string at = "item " + std::to_string(b) + ": ";
    if (it.frames == nullptr) return fail(VP_ERR_NULL, at + "frames is NULL");
    if (it.indices == nullptr) return fail(VP_ERR_NULL, at + "indices is NULL");
    if (it.n_src < 1) return fail(VP_ERR_FRAMES, at + "n_src < 1");
    if (it.src_h < 1 || it.src_w < 1) return fail(VP_ERR_DIMS, at + "source size < 1");
    if (it.n_idx < 1) return fail(VP_ERR_FRAMES, at + "n_idx < 1");
    if (it.patch != 0 && it.patch != 14 && it.patch != 16)
        return fail(VP_ERR_ARG, at + "patch must be 14 or 16 (0 for 16)");
    const int32_t win = 2 * item_patch(it);
    if (it.dst_h < win || it.dst_w < win || it.dst_h % win || it.dst_w % win)
        return fail(VP_ERR_DIMS, at + "target size not a positive multiple of " + std::to_string(win));
    for (int32_t k = 0; k < it.n_idx; ++k)
        if (it.indices[k] < 0 || it.indices[k] >= it.n_src)
            return fail(VP_ERR_INDEX, at + "index " + std::to_string(it.indices[k]) +
                                          " outside [0, " + std::to_string(it.n_src) + ")");
    const int64_t fb = int64_t(it.src_h) * it.src_w * 3;
    if (fb >= (int64_t(1) << 32)) return fail(VP_ERR_CAPACITY, at + "a source frame of 4 GiB or more");
    return VP_OK;
}

// Largest generic sub-tile (rh x cw output pixels) whose y-resampled column
// tile fits the kernel's LDS buffer for every merge window of the item.
bool generic_subtile(const AxisFilter& fx, int32_t win, int32_t* rh, int32_t* cw) {
    std::vector<int32_t> sizes;   // the divisors of the window edge, largest first
    for (int32_t d = win; d >= 1; --d)
        if (win % d == 0) sizes.push_back(d);
    for (int32_t r : sizes) {
        for (int32_t c : sizes) {
            int32_t worst = 0;
            for (int32_t j0 = 0; j0 < fx.n_out; j0 += c) {
                const int32_t span = fx.start[j0 + c - 1] + fx.count[j0 + c - 1] - fx.start[j0];
                if (span > worst) worst = span;
            }
            if (int64_t(r) * worst * 3 <= vp::kGenericTCap) {
                *rh = r;
                *cw = c;
                return true;
            }
        }
    }
    return false;
}

// ---------------------------------------------------------------------------
// Streaming-kernel routing and tables
// ---------------------------------------------------------------------------

// Slot table of a y axis for the streaming kernel.  Output row i lives in
// accumulator slot i mod M while it is open: from the first row of its
// window to its close row, the last row of its window or, if that is
// earlier, the close row of output row i - 1 (close rows never decrease;
// several output rows close on the same source row when the axis is
// upscaled, and at the bottom border).  M is the most output rows open at
// once (at least 4), so two open rows never share a slot.  For every source
// row y the table holds, per slot s < M, the weight of y in the output row
// that has slot s at y (zero if that row does not read y), times 2^24 (the
// kernel reads byte b as the f16 denormal b * 2^-24; the power of two is
// exact both ways), then the close row of every output row.  With `fixed`
// the weights are the int32 fixed-point weights of the uint8 writer instead.
// Returns M, or -1 if the axis needs more than kSlotWords slots (which
// kernel shapes take that many is up to the caller).
constexpr float kSlotScale = 16777216.0f;   // 2^24

int32_t build_slots(const AxisFilter& f, std::vector<int32_t>* words, bool fixed = false) {
    const int32_t n_in = f.n_in, n_out = f.n_out;
    const int32_t rows = n_in + vp::kSlotMax;
    std::vector<int32_t> close(n_out, 0);
    for (int32_t i = 0; i < n_out; ++i) {
        int32_t c = f.start[i] + f.count[i] - 1;
        if (i > 0 && c < close[i - 1]) c = close[i - 1];
        if (i > 0 && f.start[i] < f.start[i - 1]) return -1;
        close[i] = c;
    }
    if (close[n_out - 1] >= rows) return -1;
    // most rows open at once: a row is open on [start, close]
    std::vector<int32_t> delta(rows + 1, 0);
    for (int32_t i = 0; i < n_out; ++i) {
        ++delta[f.start[i]];
        --delta[close[i] + 1];
    }
    int32_t open = 0, most = 0;
    for (int32_t y = 0; y < rows; ++y) {
        open += delta[y];
        most = open > most ? open : most;
    }
    if (most > vp::kSlotWords) return -1;
    const int32_t m = most < 4 ? 4 : most;
    // close_row[n_out] and [n_out + 1]: never reached (kernels read one close row ahead)
    words->assign(size_t(rows) * vp::kSlotWords + n_out + 2, 0);
    (*words)[size_t(rows) * vp::kSlotWords + n_out] = INT32_MAX;
    (*words)[size_t(rows) * vp::kSlotWords + n_out + 1] = INT32_MAX;
    float* w = reinterpret_cast<float*>(words->data());
    for (int32_t i = 0; i < n_out; ++i)
        for (int32_t k = 0; k < f.count[i]; ++k) {
            const size_t at = size_t(f.start[i] + k) * vp::kSlotWords + i % m;
            if (fixed)
                (*words)[at] = f.fixed[size_t(i) * f.taps + k];
            else
                w[at] = f.weight[size_t(i) * f.taps + k] * kSlotScale;
        }
    std::memcpy(words->data() + size_t(rows) * vp::kSlotWords, close.data(), sizeof(int32_t) * n_out);
    return m;
}

// Column table of an x axis for the streaming kernel.  Output columns are
// cut into bands of `band`; a band's source pixels start at the window start
// of its first column, x0.  For column j: start[j] = (window start - x0),
// lowered where needed so that start[j] + kx <= row_px, and the window's
// weights shifted by the amount it was lowered, inside kx zero-padded taps.
// The caller has checked that every window ends within row_px of its x0.
void build_columns(const AxisFilter& f, int32_t kx, int32_t band, int32_t row_px,
                   std::vector<int32_t>* words) {
    words->assign(size_t(f.n_out) * (1 + kx), 0);
    int32_t* start = words->data();
    float* w = reinterpret_cast<float*>(words->data() + f.n_out);
    for (int32_t j = 0; j < f.n_out; ++j) {
        const int32_t x0 = f.start[j / band * band];
        const int32_t l = f.start[j] - x0;
        const int32_t s = l < row_px - kx ? l : row_px - kx;
        const int32_t shift = l - s;
        start[j] = s;
        for (int32_t k = 0; k < f.count[j]; ++k)
            w[size_t(j) * kx + shift + k] = f.weight[size_t(j) * f.taps + k];
    }
}

// Column table of an x axis for the uint8 streaming writer.  The kernel
// keeps each channel of a band's source row as signed bytes (value - 128),
// and column j reads kx of them from a dword-aligned start s_j (its window
// start relative to the band's x0, rounded down to a multiple of 4, lowered
// so that s_j + kx <= row_px), with the window's weights shifted to match.
// Each weight q splits into balanced base-256 digits, q = d2 2^16 + d1 2^8
// + d0 with every digit in [-128, 127], so that byte dot products (dot4 of
// four digits with four values) form the sums.  Per column: s_j / 4, then
// 128 * (sum of q) + 2^21 (the offset of the values and the rounding term),
// then for digits d0, d1, d2 the kx / 4 dwords of four taps' digits.
// Returns false if a weight does not fit three digits.
bool build_columns_dot(const AxisFilter& f, int32_t kx, int32_t band, int32_t row_px,
                       std::vector<int32_t>* words) {
    const int32_t g = kx / 4;
    const int32_t n = f.n_out;
    words->assign(size_t(n) * (2 + 3 * g), 0);
    int32_t* start = words->data();
    int32_t* cterm = start + n;
    int32_t* dig = cterm + n;
    for (int32_t j = 0; j < n; ++j) {
        const int32_t x0 = f.start[j / band * band];
        const int32_t l = f.start[j] - x0;
        const int32_t s = std::min(l & ~3, row_px - kx);
        const int32_t shift = l - s;
        if (s < 0 || shift + f.count[j] > kx) return false;
        start[j] = s / 4;
        int64_t sum = 0;
        for (int32_t k = 0; k < f.count[j]; ++k) {
            const int32_t q = f.fixed[size_t(j) * f.taps + k];
            sum += q;
            const int32_t d0 = ((q + 128) & 255) - 128;
            const int32_t q1 = (q - d0) >> 8;
            const int32_t d1 = ((q1 + 128) & 255) - 128;
            const int32_t d2 = (q1 - d1) >> 8;
            if (d2 < -128 || d2 > 127) return false;
            const int32_t t = shift + k;
            const int32_t d[3] = {d0, d1, d2};
            for (int32_t c = 0; c < 3; ++c) {
                uint32_t& w = reinterpret_cast<uint32_t&>(dig[(size_t(j) * 3 + c) * g + t / 4]);
                w |= (static_cast<uint32_t>(d[c]) & 0xffu) << (8 * (t % 4));
            }
        }
        const int64_t ct = 128 * sum + (int64_t(1) << 21);
        if (ct > INT32_MAX || ct < INT32_MIN) return false;
        cterm[j] = static_cast<int32_t>(ct);
    }
    return true;
}

// Column table of an x axis for the uint8 writer's MFMA form.  Output
// columns go in bands of 64, each of four blocks of 16; block b's window is
// the 64 source pixels from the window start of its first column (for a
// band's last block: the 64 that end where its columns' taps end), and the
// horizontal sums of a block are a 16 x 16 x 64 byte matrix product per
// channel and weight digit.  Per band: the four window starts (absolute
// source pixels), then for each block and digit d2, d1, d0 the B operand of
// v_mfma_i32_16x16x64_i8 for every lane l (column l % 16 of the block, window
// taps 16 (l / 16) .. 16 (l / 16) + 15) as four dwords of digit bytes.  After
// the bands, per column the start value 128 * (sum of q) + 2^21.  Returns
// false if a block's columns do not fit its window or a weight its digits.
bool build_columns_mfma(const AxisFilter& f, std::vector<int32_t>* words) {
    const int32_t n = f.n_out;
    const int32_t bands = (n + 63) / 64;
    words->assign(size_t(bands) * vp::kRsMfmaBandWords + n, 0);
    int32_t* cterm = words->data() + size_t(bands) * vp::kRsMfmaBandWords;
    for (int32_t bd = 0; bd < bands; ++bd) {
        int32_t* bw = words->data() + size_t(bd) * vp::kRsMfmaBandWords;
        for (int32_t blk = 0; blk < 4; ++blk) {
            const int32_t j0 = bd * 64 + blk * 16;
            int32_t xb = j0 < n ? f.start[j0] : (blk > 0 ? bw[blk - 1] : 0);
            // the band's last block ends its window where its columns' taps
            // end: its pixels past that belong to the next band, whose own
            // wave reads them
            const bool last = j0 < n && (blk == 3 || j0 + 16 >= n);
            if (last) {
                int32_t end = 0;
                for (int32_t j = j0; j < j0 + 16 && j < n; ++j) end = std::max(end, f.start[j] + f.count[j]);
                xb = std::max(0, std::min(xb, end - 64));
            }
            bw[blk] = xb;
            for (int32_t nn = 0; nn < 16 && j0 + nn < n; ++nn) {
                const int32_t j = j0 + nn;
                if (f.start[j] + f.count[j] - xb > 64) return false;
                int64_t sum = 0;
                for (int32_t t = 0; t < f.count[j]; ++t) {
                    const int32_t q = f.fixed[size_t(j) * f.taps + t];
                    sum += q;
                    const int32_t d0 = ((q + 128) & 255) - 128;
                    const int32_t q1 = (q - d0) >> 8;
                    const int32_t d1 = ((q1 + 128) & 255) - 128;
                    const int32_t d2 = (q1 - d1) >> 8;
                    if (d2 < -128 || d2 > 127) return false;
                    const int32_t k = f.start[j] + t - xb;        // tap position in the window
                    const int32_t lane = (k / 16) * 16 + nn;       // the lane holding (k, column nn)
                    const int32_t byte = k % 16;
                    const int32_t d[3] = {d2, d1, d0};
                    for (int32_t dg = 0; dg < 3; ++dg) {
                        uint32_t& w = reinterpret_cast<uint32_t&>(
                            bw[4 + ((blk * 3 + dg) * 64 + lane) * 4 + byte / 4]);
                        w |= (static_cast<uint32_t>(d[dg]) & 0xffu) << (8 * (byte % 4));
                    }
                }
                const int64_t ct = 128 * sum + (int64_t(1) << 21);
                if (ct > INT32_MAX || ct < INT32_MIN) return false;
                cterm[j] = static_cast<int32_t>(ct);
            }
        }
    }
    return true;
}

struct StreamShape {
    int32_t m = 0, kx = 0, px = 0, band = 0, bands = 0;
};

int32_t round_up(int32_t v, int32_t q) { return (v + q - 1) / q * q; }

// Widest span of source pixels that one band of output columns reads.
int32_t band_span(const AxisFilter& fx, int32_t band) {
    int32_t worst = 0;
    for (int32_t j0 = 0; j0 < fx.n_out; j0 += band) {
        const int32_t j1 = (j0 + band < fx.n_out ? j0 + band : fx.n_out) - 1;
        const int32_t span = fx.start[j1] + fx.count[j1] - fx.start[j0];
        worst = span > worst ? span : worst;
    }
    return worst;
}

// Whether an item can take the streaming kernel, and with which shape: the
// output width is cut into bands of 1 to 4 whole patches (16 to 64 columns,
// or 14 to 56 for patch 14;
// one single-wave workgroup each, one lane per column in the x pass), each
// band's source pixels must fit 64 lanes of px pixels, and among the shapes
// that fit, the one with the least estimated lane work is taken.  The LDS
// budget is checked with float32 staging, so the routing does not depend on
// the output type.
bool stream_shape(const vp_item& it, const AxisFilter& fx, int32_t m, int32_t patch, StreamShape* sh) {
    if (m < 4 || m > vp::kSlotWords) return false;
    const int32_t mm = m;
    // windows up to 16 taps run their own tap count (at least 4), longer ones a multiple of 4
    const int32_t kx = fx.taps <= 16 ? std::max<int32_t>(fx.taps, 4) : round_up(fx.taps, 4);
    // every load of a frame row (up to kSlotMax + 8 rows past the last one) stays below 4 GiB
    if (int64_t(it.src_h + vp::kSlotMax + 8) * it.src_w * 3 + 64 >= (int64_t(1) << 32)) return false;
    int64_t best = -1;
    for (int32_t band = 4 * patch; band >= patch; band -= patch) {
        const int32_t waves = (it.dst_w + band - 1) / band;
        if (waves > vp::kWgBandMax) continue;   // the band index field of a workgroup entry
        const int32_t span = band_span(fx, band);
        for (int32_t px = 2; px <= 4; ++px) {
            if (!vp::stream_shape_supported(mm, kx, px)) continue;
            if (span > 64 * px || kx > 64 * px) continue;
            if (vp::stream_wave_bytes(px, kx, 4, patch) > vp::kStreamLdsBudget) continue;
            // vector instructions per wave: per source row 3 px M
            // multiply-adds, about 2 px unpacks and 4 more; per output row
            // the x pass (3 kx FMAs, kx LDS reads), the slot's 3 px clears
            // and about 12 more
            const int64_t cost = int64_t(waves) * (int64_t(it.src_h) * (3 * px * mm + 2 * px + 4) +
                                                    int64_t(it.dst_h) * (4 * kx + 3 * px + 12));
            if (best < 0 || cost < best) {
                best = cost;
                sh->m = mm;
                sh->kx = kx;
                sh->px = px;
                sh->band = band;
                sh->bands = waves;
            }
            break;   // a wider px only adds idle lanes
        }
    }
    return best >= 0;
}

// The x-first streaming kernel (patch 16) for an item, if it can take it:
// 4 to 12 taps (the window's own count, at least 4), M slots.  With
// `pairs`, windows of 6 to 8 taps -- x scales of about 1.3 to 2 -- whose
// starts in each pair of columns (2i, 2i + 1) lie 0 to 2 pixels apart take
// one column pair per lane and 128 columns per wave; else a lane takes one
// column and a wave 64.  (A single column's window of 6 or more taps takes a
// second load of 8 bytes or more per row, which pairs save; shorter windows
// ran slower in pairs, at the lower occupancy of their larger register set.)
// The last band is narrower where the width is not a multiple of the band.
// Its shape is recorded with px = xfirst_px(0), or xfirst_px(2) for pairs.
bool xfirst_shape(const vp_item& it, const AxisFilter& fx, int32_t m, bool pairs_ok, StreamShape* sh) {
    const int32_t kx = std::max<int32_t>(fx.taps, 4);
    bool pairs = pairs_ok && vp::xfirst_shape_supported(m, kx, 2) && fx.n_out % 2 == 0;
    for (int32_t j = 0; pairs && j + 1 < fx.n_out; j += 2) {
        const int32_t d = fx.start[j + 1] - fx.start[j];
        pairs = d >= 0 && d <= 2;
    }
    const int32_t db = pairs ? 2 : 0;
    if (!vp::xfirst_shape_supported(m, kx, db)) return false;
    // every load of a frame row (a window of up to 3 (kx + db) + 6 bytes past
    // its start, up to kSlotMax + 8 rows past the last one) stays below 4 GiB
    if (int64_t(it.src_h + vp::kSlotMax + 8) * it.src_w * 3 + 3 * kx + 64 >= (int64_t(1) << 32)) return false;
    const int32_t band = db > 0 ? 128 : 64;
    const int32_t waves = (it.dst_w + band - 1) / band;
    if (waves > vp::kWgBandMax) return false;
    sh->m = m;
    sh->kx = kx;
    sh->px = vp::xfirst_px(db);
    sh->band = band;
    sh->bands = waves;
    return true;
}

// Vertical scales up to this one (source rows per output row) take the
// x-first kernel where it fits: an output row closes on almost every source
// row there, and the y-first kernel's gathers of each closed row from LDS
// bound it.
constexpr double kXFirstMaxScale = 1.6;

// Process-wide cache of per-axis tables.  The same axes recur from call to
// call (an RL loop preprocesses batches of the same shapes every step), and
// building them is most of the host's work for a batch of many shapes.
// Entries are immutable once built and shared by pointer; a cache is
// cleared when it reaches kTableCacheMax entries.
struct AxisEntry {
    AxisFilter f;
    std::vector<int32_t> words;         // the window table: start, count, weight
    std::vector<int32_t> fixed_words;   // the same with the fixed-point weights
};
struct SlotEntry {
    int32_t m = -1;               // slots, or -1 if the axis needs too many
    std::vector<int32_t> words;
};
using ColumnKey = std::tuple<int32_t, int32_t, int32_t, int32_t, int32_t, bool>;   // n_in, n_out, kx, band, row_px, fixed
using SlotKey = std::tuple<int32_t, int32_t, bool>;                                 // n_in, n_out, fixed

constexpr size_t kTableCacheMax = 4096;
std::mutex g_cache_mu;
std::map<std::pair<int32_t, int32_t>, std::shared_ptr<const AxisEntry>> g_axis_cache;
std::map<SlotKey, std::shared_ptr<const SlotEntry>> g_slot_cache;
std::map<ColumnKey, std::shared_ptr<const std::vector<int32_t>>> g_column_cache;

// The entry for `key`, built by `make` (outside the lock) on a miss.  If two
// threads miss together, the first entry stored wins; both are identical.
template <class Map, class Make>
typename Map::mapped_type cached(Map& map, const typename Map::key_type& key, Make make) {
    {
        std::lock_guard<std::mutex> lk(g_cache_mu);
        auto it = map.find(key);
        if (it != map.end()) return it->second;
    }
    typename Map::mapped_type v = make();
    std::lock_guard<std::mutex> lk(g_cache_mu);
    if (map.size() >= kTableCacheMax) map.clear();
    return map.emplace(key, std::move(v)).first->second;
}

std::shared_ptr<const AxisEntry> make_axis_entry(int32_t n_in, int32_t n_out) {
    auto e = std::make_shared<AxisEntry>();
    build_axis(n_in, n_out, axis_taps(n_in, n_out), &e->f);
    const AxisFilter& f = e->f;
    e->words.reserve(2 * f.start.size() + f.weight.size());
    e->words.insert(e->words.end(), f.start.begin(), f.start.end());
    e->words.insert(e->words.end(), f.count.begin(), f.count.end());
    const size_t wbase = e->words.size();
    e->words.resize(wbase + f.weight.size());
    std::memcpy(e->words.data() + wbase, f.weight.data(), f.weight.size() * sizeof(float));
    e->fixed_words.reserve(e->words.size());
    e->fixed_words.insert(e->fixed_words.end(), f.start.begin(), f.start.end());
    e->fixed_words.insert(e->fixed_words.end(), f.count.begin(), f.count.end());
    e->fixed_words.insert(e->fixed_words.end(), f.fixed.begin(), f.fixed.end());
    return e;
}

// One streaming work unit with its kernel shape, before the workgroup list
// is laid out.
struct Keyed {
    std::tuple<int32_t, int32_t, int32_t> key;   // kernel shape (m, kx, px)
    int32_t bands;                               // column bands (workgroups) of the unit
    vp::StreamUnit unit;
    int64_t cost;
};

// Output rows per streaming unit of an item: at most about max_src_rows
// source rows, at least min_windows windows of source rows, a multiple of
// `group` rows (the kernel's store group), and at least 16 rows (28 for
// groups of 14).
int64_t unit_row_band(const vp::DevItem& d, int64_t max_src_rows, int64_t group, int64_t min_windows = 10) {
    int64_t band = max_src_rows * d.h / d.H;
    const int64_t min_band = (min_windows * d.ky * d.h + d.H - 1) / d.H;
    band = std::max(band, min_band);
    band = std::max<int64_t>((band + group - 1) / group * group, group == 4 ? 16 : 2 * group);
    return std::min<int64_t>(band, d.h);
}

// A frame's h output rows cut into n = ceil(h / band) units whose boundaries
// fall on whole store groups of `group` rows, as evenly as that allows:
// lengths differ by at most one group, and the last unit also takes the rows
// past the last whole group.  Units of one frame are neighbours in the
// workgroup list, and a long unit followed by a short remainder (a 320-row
// frame at a 296-row cap: 296 + 24) would load the XCDs unevenly.
struct UnitSplit {
    int64_t h, group, groups, n;
    UnitSplit(int64_t h_, int64_t band, int64_t group_) : h(h_), group(group_), groups(h_ / group_) {
        n = std::max<int64_t>(1, std::min<int64_t>((h + band - 1) / band, groups));
    }
    int32_t begin(int64_t u) const { return static_cast<int32_t>(group * (groups * u / n)); }
    int32_t end(int64_t u) const { return static_cast<int32_t>(u + 1 == n ? h : group * (groups * (u + 1) / n)); }
};

// Lays out the streaming units as launches and their workgroup lists.
int32_t assemble_launches(const std::vector<Keyed>& keyed, int32_t P, Plan* p) {
    // Units of one kernel shape form one launch, whatever their widths.  Its
    // workgroups are listed explicitly: entry g (unit index | band << 20, or
    // kNoWork) runs as workgroup g, and consecutive workgroups go to the
    // eight XCDs in turn.  Units are taken eight at a time, and their bands
    // are listed round by round (band 0 of all eight, then band 1, ...), so
    // that all bands of one unit run on one XCD and share the source pixels
    // of neighbouring bands through its L2; a unit with fewer bands than the
    // others of its eight leaves empty entries.  Units are sorted by band
    // count first, which keeps those rare.  The XCD of the x-th unit of the
    // g-th eight is (x + g) mod 8: a pattern in the units' lengths that
    // repeats every few units (the units of one frame) then spreads over all
    // eight XCDs instead of loading some more than others.
    if (keyed.size() > vp::kWgUnitMask + 1)
        return fail(VP_ERR_CAPACITY, "batch has more than 2^20 streaming work units");
    // order: by shape, then band count, then as generated (a grouping: the
    // units of one item are consecutive and share both)
    std::map<std::pair<std::tuple<int32_t, int32_t, int32_t>, int32_t>, std::vector<uint32_t>> groups;
    for (size_t k = 0; k < keyed.size();) {
        size_t k1 = k + 1;
        while (k1 < keyed.size() && keyed[k1].key == keyed[k].key && keyed[k1].bands == keyed[k].bands) ++k1;
        auto& g = groups[std::make_pair(keyed[k].key, keyed[k].bands)];
        for (; k < k1; ++k) g.push_back(static_cast<uint32_t>(k));
    }
    std::vector<uint32_t> order;
    order.reserve(keyed.size());
    for (const auto& g : groups) order.insert(order.end(), g.second.begin(), g.second.end());
    p->units.clear();
    p->wgs.clear();
    p->launches.clear();
    p->units.reserve(keyed.size());
    p->wgs.reserve(keyed.size() * 8);
    for (size_t k0 = 0; k0 < order.size();) {
        const auto& key0 = keyed[order[k0]].key;
        size_t k1 = k0;
        while (k1 < order.size() && keyed[order[k1]].key == key0) ++k1;
        vp::StreamLaunch L{};
        L.first = static_cast<int32_t>(p->wgs.size());
        L.m = std::get<0>(key0);
        L.kx = std::get<1>(key0);
        L.px = std::get<2>(key0);
        L.patch = P;
        for (size_t c0 = k0, g = 0; c0 < k1; c0 += 8, ++g) {
            const size_t c1 = std::min(c0 + 8, k1);
            int32_t rounds = 0;
            for (size_t k = c0; k < c1; ++k) rounds = std::max(rounds, keyed[order[k]].bands);
            const uint32_t u0 = static_cast<uint32_t>(p->units.size());
            for (size_t k = c0; k < c1; ++k) {
                const Keyed& e = keyed[order[k]];
                p->units.push_back(e.unit);
                L.cost += e.cost * e.bands;
            }
            for (int32_t r = 0; r < rounds; ++r)
                for (size_t col = 0; col < 8; ++col) {
                    const size_t x = (col + 8 - g % 8) % 8;   // the unit on XCD col
                    const size_t k = c0 + x;
                    p->wgs.push_back(k < c1 && r < keyed[order[k]].bands
                                         ? (u0 + static_cast<uint32_t>(x)) | (static_cast<uint32_t>(r) << vp::kWgBandShift)
                                         : vp::kNoWork);
                }
        }
        L.count = static_cast<int32_t>(p->wgs.size()) - L.first;
        p->launches.push_back(L);
        k0 = k1;
    }

    return VP_OK;
}

int32_t build_plan(const vp_item* items, int32_t n, Plan* p) {
    if (items == nullptr) return fail(VP_ERR_NULL, "items is NULL");
    if (n < 1) return fail(VP_ERR_ARG, "n_items < 1");
    int32_t P = vp::kPatch;
    if (const int32_t st = batch_patch(items, n, &P); st != VP_OK) return st;
    p->items.assign(n, vp::DevItem{});
    p->generic_cost = 0;
    p->prefix.assign(n + 1, 0);
    p->grid.assign(size_t(n) * 3, 0);
    p->cu.assign(n + 1, 0);
    p->indices.clear();
    p->tables.clear();
    p->table_words = 0;
    // Tables come from the process-wide cache; each one used by the batch is
    // copied into the plan once, and the per-call maps keep the cache
    // entries alive while the call uses them.
    auto append = [&](std::shared_ptr<const std::vector<int32_t>> words) -> int32_t {
        const int32_t o = static_cast<int32_t>(p->table_words);
        p->table_words += words->size();
        p->tables.emplace_back(o, std::move(words));
        return o;
    };
    std::map<std::pair<int32_t, int32_t>, std::pair<int32_t, std::shared_ptr<const AxisEntry>>> axes;
    auto table_for = [&](int32_t n_in, int32_t n_out, int32_t* off) -> const AxisFilter* {
        const auto key = std::make_pair(n_in, n_out);
        auto found = axes.find(key);
        if (found == axes.end()) {
            auto e = cached(g_axis_cache, key, [&] { return make_axis_entry(n_in, n_out); });
            const int32_t o = append(std::shared_ptr<const std::vector<int32_t>>(e, &e->words));
            found = axes.emplace(key, std::make_pair(o, e)).first;
        }
        *off = found->second.first;
        return &found->second.second->f;
    };
    std::map<SlotKey, std::pair<int32_t, std::shared_ptr<const SlotEntry>>> slot_tables;
    auto slots_for = [&](const AxisFilter& f, int32_t* off, int32_t* m) -> bool {
        const SlotKey key = std::make_tuple(f.n_in, f.n_out, false);
        auto found = slot_tables.find(key);
        if (found == slot_tables.end()) {
            auto e = cached(g_slot_cache, key, [&] {
                auto v = std::make_shared<SlotEntry>();
                v->m = build_slots(f, &v->words);
                return std::shared_ptr<const SlotEntry>(std::move(v));
            });
            const int32_t o = e->m > 0 ? append(std::shared_ptr<const std::vector<int32_t>>(e, &e->words)) : -1;
            found = slot_tables.emplace(key, std::make_pair(o, e)).first;
        }
        *off = found->second.first;
        *m = found->second.second->m;
        return found->second.first >= 0;
    };
    std::map<ColumnKey, int32_t> column_tables;
    auto columns_for = [&](const AxisFilter& f, int32_t kx, int32_t band, int32_t row_px) -> int32_t {
        const ColumnKey key = std::make_tuple(f.n_in, f.n_out, kx, band, row_px, false);
        auto found = column_tables.find(key);
        if (found == column_tables.end()) {
            auto e = cached(g_column_cache, key, [&] {
                auto v = std::make_shared<std::vector<int32_t>>();
                build_columns(f, kx, band, row_px, v.get());
                return std::shared_ptr<const std::vector<int32_t>>(std::move(v));
            });
            found = column_tables.emplace(key, append(e)).first;
        }
        return found->second;
    };
    std::vector<StreamShape> shapes(n);
    std::vector<const AxisFilter*> x_axes(n, nullptr);

    int64_t rows = 0, tiles = 0;
    for (int32_t b = 0; b < n; ++b) {
        const vp_item& it = items[b];
        int32_t st = validate_item(it, b);
        if (st != VP_OK) return st;
        vp::DevItem& d = p->items[b];
        d.frames = it.frames;
        d.frame_bytes = int64_t(it.src_h) * it.src_w * 3;
        d.H = it.src_h;
        d.W = it.src_w;
        d.h = it.dst_h;
        d.w = it.dst_w;
        d.t = (it.n_idx + 1) / 2;
        d.patch = P;
        d.hm = it.dst_h / (2 * P);
        d.wm = it.dst_w / (2 * P);
        d.idx_off = static_cast<int32_t>(p->indices.size());
        for (int32_t k = 0; k < 2 * d.t; ++k)
            p->indices.push_back(it.indices[k < it.n_idx ? k : it.n_idx - 1]);
        const AxisFilter* fy = table_for(it.src_h, it.dst_h, &d.ty_off);
        const AxisFilter* fx = table_for(it.src_w, it.dst_w, &d.tx_off);
        d.ky = fy->taps;
        d.kx = fx->taps;
        d.route = vp::kRouteGeneric;
        int32_t m = 0;
        StreamShape sh;
        const bool slots = slots_for(*fy, &d.sy_off, &m);
        const bool near_one = P == 16 && double(it.src_h) <= kXFirstMaxScale * double(it.dst_h);
        if (slots && ((near_one && xfirst_shape(it, *fx, m, false, &sh)) || stream_shape(it, *fx, m, P, &sh))) {
            d.route = vp::kRouteStream;   // (band and column table below, once the shape is final)
            shapes[b] = sh;
            x_axes[b] = fx;
        } else if (!generic_subtile(*fx, 2 * P, &d.rh, &d.cw)) {
            return fail(VP_ERR_CAPACITY, "item " + std::to_string(b) +
                                             ": horizontal filter window too long (downscale too large)");
        }
        d.row_off = rows;
        const int64_t item_rows = int64_t(d.t) * (it.dst_h / P) * (it.dst_w / P);
        p->grid[3 * b + 0] = d.t;
        p->grid[3 * b + 1] = it.dst_h / P;
        p->grid[3 * b + 2] = it.dst_w / P;
        rows += item_rows;
        if (d.route == vp::kRouteGeneric) {
            tiles += int64_t(d.t) * d.hm * d.wm;
            p->generic_cost += int64_t(2) * d.t * d.H * d.W;
        }
        if (rows > INT32_MAX || tiles > INT32_MAX)
            return fail(VP_ERR_CAPACITY, "batch has more than 2^31-1 rows");
        p->cu[b + 1] = static_cast<int32_t>(rows);
        p->prefix[b + 1] = static_cast<int32_t>(tiles);
    }
    p->total_rows = rows;

    // Streaming units: one per (item, distinct frame of a pair, band of output
    // rows); for patch 14 one per (item, pair, band), its frames on the two
    // waves of one workgroup.  A workgroup streams the source rows of its unit top to bottom,
    // so its life is about proportional to those rows.  To end the batch
    // evenly -- many kernel shapes run side by side, and a small launch lasts
    // as long as its longest unit -- no unit reads more than an eighth of the
    // source rows per wave slot of the whole batch (256 CUs x 20 waves), in
    // bands of output rows that are multiples of 4 (one 64-value run per
    // store).  A band re-reads the source rows that its first window shares
    // with the band above, so none spans fewer than ten windows of source
    // rows, or fifteen where the batch still gives every wave slot four
    // workgroups at that length (shorter units re-read more rows -- about a
    // tenth at ten windows -- but in a batch of few workgroups they end it
    // more evenly, which is worth more).
    constexpr int64_t kWaveSlots = 256 * 20;
    int64_t stream_frames = 0;
    auto source_row_cap = [&] {
        int64_t wave_rows = 0;   // source rows that all workgroups stream, whole frames
        stream_frames = 0;
        for (int32_t b = 0; b < n; ++b) {
            const vp::DevItem& d = p->items[b];
            if (d.route != vp::kRouteStream) continue;
            for (int32_t tt = 0; tt < d.t; ++tt) {
                const bool same = p->indices[d.idx_off + 2 * tt] == p->indices[d.idx_off + 2 * tt + 1];
                wave_rows += int64_t(same ? 1 : 2) * shapes[b].bands * d.H;
                stream_frames += same ? 1 : 2;
            }
        }
        return wave_rows / (kWaveSlots * 8);
    };
    auto workgroup_waves = [&](int64_t min_windows, int64_t max_src_rows) {
        int64_t waves = 0;
        for (int32_t b = 0; b < n; ++b) {
            const vp::DevItem& d = p->items[b];
            if (d.route != vp::kRouteStream) continue;
            const int64_t group = d.patch == 16 ? 4 : d.patch;
            const int64_t units = UnitSplit(d.h, unit_row_band(d, max_src_rows, group, min_windows), group).n;
            int64_t frames = 0;   // units per row band: one per distinct frame (patch 14: per pair)
            for (int32_t tt = 0; tt < d.t; ++tt)
                frames += d.patch == 14 || p->indices[d.idx_off + 2 * tt] == p->indices[d.idx_off + 2 * tt + 1]
                              ? 1 : 2;
            const int64_t per_unit = d.patch == 14 ? 4 * ((shapes[b].bands + 1) / 2) : shapes[b].bands;
            waves += frames * units * per_unit;
        }
        return waves;
    };
    // Column pairs halve an x-first item's workgroups: taken only where the
    // batch gives every wave slot four workgroups with single columns.
    if (workgroup_waves(10, source_row_cap()) >= 4 * kWaveSlots) {
        for (int32_t b = 0; b < n; ++b) {
            StreamShape sh;
            if (p->items[b].route == vp::kRouteStream && shapes[b].px == vp::xfirst_px(0) &&
                xfirst_shape(items[b], *x_axes[b], shapes[b].m, true, &sh))
                shapes[b] = sh;
        }
    }
    for (int32_t b = 0; b < n; ++b) {
        vp::DevItem& d = p->items[b];
        if (d.route != vp::kRouteStream) continue;
        const StreamShape& sh = shapes[b];
        d.band = sh.band;
        d.row_px = sh.px > 0 ? 64 * sh.px : d.W + sh.kx;
        d.sx_off = columns_for(*x_axes[b], sh.kx, sh.band, d.row_px);
    }
    const int64_t max_src_rows = source_row_cap();
    const int64_t min_windows = workgroup_waves(15, max_src_rows) >= 4 * kWaveSlots ? 15 : 10;
    std::vector<Keyed> keyed;
    keyed.reserve(static_cast<size_t>(stream_frames));
    for (int32_t b = 0; b < n; ++b) {
        const vp::DevItem& d = p->items[b];
        if (d.route != vp::kRouteStream) continue;
        const StreamShape& sh = shapes[b];
        // whole store groups: multiples of 4 rows for patch 16, whole
        // patch rows (14 output rows, stored at once) for patch 14
        const int64_t group = d.patch == 16 ? 4 : d.patch;
        const UnitSplit split(d.h, unit_row_band(d, max_src_rows, group, min_windows), group);
        for (int32_t tt = 0; tt < d.t; ++tt) {
            const bool same = p->indices[d.idx_off + 2 * tt] == p->indices[d.idx_off + 2 * tt + 1];
            const bool pair_units = d.patch == 14;   // both frames in one unit
            for (int32_t dt = 0; dt < (same || pair_units ? 1 : 2); ++dt) {
                for (int64_t u = 0; u < split.n; ++u) {
                    const int32_t i0 = split.begin(u), i1 = split.end(u);
                    Keyed k;
                    k.key = std::make_tuple(sh.m, sh.kx, sh.px);
                    k.bands = d.patch == 14 ? (sh.bands + 1) / 2 : sh.bands;   // patch 14: bands in pairs
                    k.unit.item = b;
                    k.unit.p_flags = (2 * tt + dt) | (same ? vp::kUnitBoth : 0);
                    k.unit.i0 = i0;
                    k.unit.i1 = i1;
                    k.cost = int64_t(i1 - i0) * d.H / d.h * d.W   // source pixels read, roughly
                             * (pair_units && !same ? 2 : 1);
                    keyed.push_back(k);
                }
            }
        }
    }
    if (const int32_t st = assemble_launches(keyed, P, p); st != VP_OK) return st;

    p->off_items = 0;
    p->off_prefix = align_up(p->off_items + sizeof(vp::DevItem) * p->items.size());
    p->off_indices = align_up(p->off_prefix + sizeof(int32_t) * p->prefix.size());
    p->off_tables = align_up(p->off_indices + sizeof(int32_t) * p->indices.size());
    p->off_units = align_up(p->off_tables + sizeof(int32_t) * p->table_words);
    p->off_wgs = align_up(p->off_units + sizeof(vp::StreamUnit) * p->units.size());
    p->bytes = align_up(p->off_wgs + sizeof(uint32_t) * p->wgs.size());
    return VP_OK;
}

// Plan of vp_patchify_batch: items whose frames are already at the target
// size; one workgroup per merge-window row (32 pixel rows) of a frame pair.
int32_t build_patch_plan(const vp_item* items, int32_t n, Plan* p) {
    if (items == nullptr) return fail(VP_ERR_NULL, "items is NULL");
    if (n < 1) return fail(VP_ERR_ARG, "n_items < 1");
    int32_t P = vp::kPatch;
    if (const int32_t st = batch_patch(items, n, &P); st != VP_OK) return st;
    p->items.assign(n, vp::DevItem{});
    p->prefix.assign(n + 1, 0);
    p->grid.assign(size_t(n) * 3, 0);
    p->cu.assign(n + 1, 0);
    p->indices.clear();
    p->tables.clear();
    p->table_words = 0;
    p->units.clear();
    p->wgs.clear();
    p->launches.clear();
    p->generic_cost = 0;
    int64_t rows = 0, tiles = 0;
    for (int32_t b = 0; b < n; ++b) {
        const vp_item& it = items[b];
        int32_t st = validate_item(it, b);
        if (st != VP_OK) return st;
        const std::string at = "item " + std::to_string(b) + ": ";
        if (it.dst_h != it.src_h || it.dst_w != it.src_w)
            return fail(VP_ERR_DIMS, at + "vp_patchify_batch needs frames already at the target size");
        if (reinterpret_cast<uintptr_t>(it.frames) % 4 != 0)
            return fail(VP_ERR_ARG, at + "frames must be 4-byte aligned");
        vp::DevItem& d = p->items[b];
        d.frames = it.frames;
        d.frame_bytes = int64_t(it.src_h) * it.src_w * 3;
        d.H = d.h = it.dst_h;
        d.W = d.w = it.dst_w;
        d.t = (it.n_idx + 1) / 2;
        d.patch = P;
        d.hm = it.dst_h / (2 * P);
        d.wm = it.dst_w / (2 * P);
        d.idx_off = static_cast<int32_t>(p->indices.size());
        for (int32_t k = 0; k < 2 * d.t; ++k)
            p->indices.push_back(it.indices[k < it.n_idx ? k : it.n_idx - 1]);
        d.route = vp::kRoutePatch;
        d.row_off = rows;
        p->grid[3 * b + 0] = d.t;
        p->grid[3 * b + 1] = it.dst_h / P;
        p->grid[3 * b + 2] = it.dst_w / P;
        rows += int64_t(d.t) * (it.dst_h / P) * (it.dst_w / P);
        tiles += int64_t(d.t) * d.hm;
        if (rows > INT32_MAX || tiles > INT32_MAX)
            return fail(VP_ERR_CAPACITY, "batch has more than 2^31-1 rows");
        p->cu[b + 1] = static_cast<int32_t>(rows);
        p->prefix[b + 1] = static_cast<int32_t>(tiles);
    }
    p->total_rows = rows;
    p->off_items = 0;
    p->off_prefix = align_up(p->off_items + sizeof(vp::DevItem) * p->items.size());
    p->off_indices = align_up(p->off_prefix + sizeof(int32_t) * p->prefix.size());
    p->off_tables = align_up(p->off_indices + sizeof(int32_t) * p->indices.size());
    p->off_units = p->off_tables;
    p->off_wgs = p->off_tables;
    p->bytes = p->off_tables;
    return VP_OK;
}

// Plan of the row tables (vp_position_ids): per item its grid, with the
// items' row offsets (cu) as the prefix the kernel searches.
int32_t build_rows_plan(const vp_item* items, int32_t n, Plan* p) {
    if (items == nullptr) return fail(VP_ERR_NULL, "items is NULL");
    if (n < 1) return fail(VP_ERR_ARG, "n_items < 1");
    int32_t P = vp::kPatch;
    if (const int32_t st = batch_patch(items, n, &P); st != VP_OK) return st;
    p->items.assign(n, vp::DevItem{});
    p->grid.assign(size_t(n) * 3, 0);
    p->cu.assign(n + 1, 0);
    p->indices.clear();
    p->tables.clear();
    p->table_words = 0;
    p->units.clear();
    p->wgs.clear();
    p->launches.clear();
    p->generic_cost = 0;
    int64_t rows = 0;
    for (int32_t b = 0; b < n; ++b) {
        const vp_item& it = items[b];
        const int32_t st = validate_item(it, b);
        if (st != VP_OK) return st;
        vp::DevItem& d = p->items[b];
        d.h = it.dst_h;
        d.w = it.dst_w;
        d.t = (it.n_idx + 1) / 2;
        d.patch = P;
        d.hm = it.dst_h / (2 * P);
        d.wm = it.dst_w / (2 * P);
        d.row_off = rows;
        p->grid[3 * b + 0] = d.t;
        p->grid[3 * b + 1] = it.dst_h / P;
        p->grid[3 * b + 2] = it.dst_w / P;
        rows += int64_t(d.t) * (it.dst_h / P) * (it.dst_w / P);
        if (rows > INT32_MAX) return fail(VP_ERR_CAPACITY, "batch has more than 2^31-1 rows");
        p->cu[b + 1] = static_cast<int32_t>(rows);
    }
    p->prefix = p->cu;
    p->total_rows = rows;
    p->off_items = 0;
    p->off_prefix = align_up(p->off_items + sizeof(vp::DevItem) * p->items.size());
    p->off_indices = align_up(p->off_prefix + sizeof(int32_t) * p->prefix.size());
    p->off_tables = p->off_indices;
    p->off_units = p->off_indices;
    p->off_wgs = p->off_indices;
    p->bytes = p->off_indices;
    return VP_OK;
}

// Output tile of the uint8 writer for an item: the largest rows x columns
// (rows from 32 down, then columns from 64 down) whose horizontal-pass rows,
// staged source span and weights fit the kernel's LDS budgets.
bool resize_tiles(const AxisFilter& fy, const AxisFilter& fx, int32_t* rb, int32_t* cb) {
    static const int32_t kRows[] = {32, 16, 8, 4, 2, 1};
    static const int32_t kCols[] = {64, 32, 16, 8};
    for (int32_t r : kRows) {
        if (int64_t(r) * fy.taps > vp::kRsQ) continue;
        int64_t rows = 0;   // source rows the tile's horizontal pass produces
        for (int32_t i0 = 0; i0 < fy.n_out; i0 += r) {
            const int32_t i1 = std::min(i0 + r, fy.n_out) - 1;
            rows = std::max<int64_t>(rows, fy.start[i1] + fy.count[i1] - fy.start[i0]);
        }
        for (int32_t c : kCols) {
            if (int64_t(c) * fx.taps > vp::kRsQ) continue;
            int64_t span = 0;   // source pixels the tile's columns read
            for (int32_t j0 = 0; j0 < fx.n_out; j0 += c) {
                const int32_t j1 = std::min(j0 + c, fx.n_out) - 1;
                span = std::max<int64_t>(span, fx.start[j1] + fx.count[j1] - fx.start[j0]);
            }
            if (rows * c * 3 <= vp::kRsMid && span * 3 + 6 <= vp::kRsSrcRow) {
                *rb = r;
                *cb = c;
                return true;
            }
        }
    }
    return false;
}

// Shape of the uint8 streaming writer for an item, if it can take it: the
// output width in bands of 64 columns (down to 16), each band's source span
// within 64 lanes of px pixels, the column taps rounded up to 4, M slots.
// The widest band that fits is taken: the horizontal pass costs the same per
// output column whatever the band, and fewer bands unpack fewer pixels.
bool resize_stream_shape(const vp_item& it, const AxisFilter& fx, int32_t m, StreamShape* sh) {
    if (m < 4 || m > vp::kSlotWords) return false;
    const int32_t kx = round_up(fx.taps + 3, 4);   // any window start, rounded down to a dword
    if (!vp::resize_stream_supported(m, kx, vp::kRsPx)) return false;
    if (int64_t(it.src_h + vp::kSlotMax + 8) * it.src_w * 3 + 64 >= (int64_t(1) << 32)) return false;
    for (int32_t band = 64; band >= 16; band -= 16) {
        if (band_span(fx, band) > 64 * vp::kRsPx) continue;
        if ((it.dst_w + band - 1) / band > vp::kWgBandMax) continue;
        sh->m = m;
        sh->kx = kx;
        sh->px = vp::kRsPx;
        sh->band = band;
        sh->bands = (it.dst_w + band - 1) / band;
        return true;
    }
    return false;
}

// Plan of vp_resize_batch: per item its frames in index order (no padding),
// fixed-point tables, the route (streaming, or the tile kernel where an axis
// does not fit the streaming shapes) and its output byte offset.
int32_t build_resize_plan(const vp_item* items, int32_t n, Plan* p) {
    if (items == nullptr) return fail(VP_ERR_NULL, "items is NULL");
    if (n < 1) return fail(VP_ERR_ARG, "n_items < 1");
    int32_t P = vp::kPatch;
    if (const int32_t st = batch_patch(items, n, &P); st != VP_OK) return st;
    p->items.assign(n, vp::DevItem{});
    p->prefix.assign(n + 1, 0);
    p->byte_off.assign(n + 1, 0);
    p->grid.clear();
    p->cu.clear();
    p->indices.clear();
    p->tables.clear();
    p->table_words = 0;
    p->units.clear();
    p->wgs.clear();
    p->launches.clear();
    p->generic_cost = 0;
    std::map<std::pair<int32_t, int32_t>, std::pair<int32_t, std::shared_ptr<const AxisEntry>>> axes;
    auto append = [&](std::shared_ptr<const std::vector<int32_t>> words) -> int32_t {
        const int32_t o = static_cast<int32_t>(p->table_words);
        p->table_words += words->size();
        p->tables.emplace_back(o, std::move(words));
        return o;
    };
    auto table_for = [&](int32_t n_in, int32_t n_out, int32_t* off) -> const AxisFilter* {
        const auto key = std::make_pair(n_in, n_out);
        auto found = axes.find(key);
        if (found == axes.end()) {
            auto e = cached(g_axis_cache, key, [&] { return make_axis_entry(n_in, n_out); });
            const int32_t o = append(std::shared_ptr<const std::vector<int32_t>>(e, &e->fixed_words));
            found = axes.emplace(key, std::make_pair(o, e)).first;
        }
        *off = found->second.first;
        return &found->second.second->f;
    };
    std::map<SlotKey, std::pair<int32_t, std::shared_ptr<const SlotEntry>>> slot_tables;
    auto slots_for = [&](const AxisFilter& f, int32_t* off, int32_t* m) -> bool {
        const SlotKey key = std::make_tuple(f.n_in, f.n_out, true);
        auto found = slot_tables.find(key);
        if (found == slot_tables.end()) {
            auto e = cached(g_slot_cache, key, [&] {
                auto v = std::make_shared<SlotEntry>();
                v->m = build_slots(f, &v->words, true);
                return std::shared_ptr<const SlotEntry>(std::move(v));
            });
            const int32_t o = e->m > 0 ? append(std::shared_ptr<const std::vector<int32_t>>(e, &e->words)) : -1;
            found = slot_tables.emplace(key, std::make_pair(o, e)).first;
        }
        *off = found->second.first;
        *m = found->second.second->m;
        return found->second.first >= 0;
    };
    std::map<ColumnKey, int32_t> column_tables;
    // the dot-product column table, or -1 if a weight does not fit its digits
    auto columns_for = [&](const AxisFilter& f, int32_t kx, int32_t band, int32_t row_px) -> int32_t {
        const ColumnKey key = std::make_tuple(f.n_in, f.n_out, kx, band, row_px, true);
        auto found = column_tables.find(key);
        if (found == column_tables.end()) {
            auto e = cached(g_column_cache, key, [&] {
                auto v = std::make_shared<std::vector<int32_t>>();
                if (!build_columns_dot(f, kx, band, row_px, v.get())) v->clear();
                return std::shared_ptr<const std::vector<int32_t>>(std::move(v));
            });
            found = column_tables.emplace(key, e->empty() ? -1 : append(e)).first;
        }
        return found->second;
    };
    std::map<std::pair<int32_t, int32_t>, int32_t> mfma_tables;
    // the MFMA column table, or -1 if a block's columns do not fit its window
    auto mfma_columns_for = [&](const AxisFilter& f) -> int32_t {
        const ColumnKey key = std::make_tuple(f.n_in, f.n_out, vp::kRsMfmaWindow, 64, 0, true);
        auto found = mfma_tables.find(std::make_pair(f.n_in, f.n_out));
        if (found == mfma_tables.end()) {
            auto e = cached(g_column_cache, key, [&] {
                auto v = std::make_shared<std::vector<int32_t>>();
                if (!build_columns_mfma(f, v.get())) v->clear();
                return std::shared_ptr<const std::vector<int32_t>>(std::move(v));
            });
            found = mfma_tables.emplace(std::make_pair(f.n_in, f.n_out), e->empty() ? -1 : append(e)).first;
        }
        return found->second;
    };
    std::vector<StreamShape> shapes(n);
    int64_t bytes = 0, tiles = 0;
    for (int32_t b = 0; b < n; ++b) {
        const vp_item& it = items[b];
        int32_t st = validate_item(it, b);
        if (st != VP_OK) return st;
        vp::DevItem& d = p->items[b];
        d.frames = it.frames;
        d.frame_bytes = int64_t(it.src_h) * it.src_w * 3;
        d.H = it.src_h;
        d.W = it.src_w;
        d.h = it.dst_h;
        d.w = it.dst_w;
        d.t = it.n_idx;
        d.idx_off = static_cast<int32_t>(p->indices.size());
        p->indices.insert(p->indices.end(), it.indices, it.indices + it.n_idx);
        const AxisFilter* fy = table_for(it.src_h, it.dst_h, &d.ty_off);
        const AxisFilter* fx = table_for(it.src_w, it.dst_w, &d.tx_off);
        d.ky = fy->taps;
        d.kx = fx->taps;
        d.patch = P;
        d.row_off = bytes;   // output byte offset of the item
        bytes += int64_t(it.n_idx) * it.dst_h * it.dst_w * 3;
        int32_t m = 0;
        StreamShape sh;
        const bool slots = slots_for(*fy, &d.sy_off, &m);
        // The MFMA form costs about the same per source row whatever the
        // window; byte dot products cost in proportion to it.  Measured, the
        // MFMA form wins from 16 dot-product taps (windows of 10 or more).
        const bool long_x = round_up(fx->taps + 3, 4) >= 16;
        if (slots && long_x && m >= 4 && m <= vp::kSlotWords && (it.dst_w + 63) / 64 <= vp::kWgBandMax &&
            (d.sx_off = mfma_columns_for(*fx)) >= 0 &&
            int64_t(it.src_h + vp::kSlotMax + 20) * it.src_w * 3 + 256 < (int64_t(1) << 32)) {
            // the MFMA form: bands of 64 columns, blocks of 16 with 64-pixel windows
            d.route = vp::kRouteStream;
            d.band = 64;
            d.row_px = 0;
            sh.m = m;
            sh.kx = vp::kRsMfmaWindow;
            sh.px = vp::kRsPx;
            sh.band = 64;
            sh.bands = (it.dst_w + 63) / 64;
            shapes[b] = sh;
        } else if (slots && resize_stream_shape(it, *fx, m, &sh) &&
            (d.sx_off = columns_for(*fx, sh.kx, sh.band, 64 * sh.px)) >= 0) {
            d.route = vp::kRouteStream;
            d.band = sh.band;
            d.row_px = 64 * sh.px;
            shapes[b] = sh;
        } else {
            if (!resize_tiles(*fy, *fx, &d.rh, &d.cw))
                return fail(VP_ERR_CAPACITY, "item " + std::to_string(b) +
                                                 ": filter window too long for the uint8 writer's tiles");
            d.hm = (it.dst_h + d.rh - 1) / d.rh;
            d.wm = (it.dst_w + d.cw - 1) / d.cw;
            d.route = vp::kRouteResize;
            tiles += int64_t(it.n_idx) * d.hm * d.wm;
            p->generic_cost += int64_t(8) * it.n_idx * it.src_h * it.src_w;   // about 8x the streaming cost per pixel
        }
        if (tiles > INT32_MAX) return fail(VP_ERR_CAPACITY, "batch has more than 2^31-1 tiles");
        p->byte_off[b + 1] = bytes;
        p->prefix[b + 1] = static_cast<int32_t>(tiles);
    }
    p->total_rows = 0;

    // Streaming units: one per (item, frame, band of output rows), the
    // bands sized as for the float path (multiples of the kernel's store
    // group of 4 rows).
    constexpr int64_t kWaveSlots = 256 * 20;
    int64_t wave_rows = 0;
    for (int32_t b = 0; b < n; ++b) {
        const vp::DevItem& d = p->items[b];
        if (d.route == vp::kRouteStream) wave_rows += int64_t(d.t) * shapes[b].bands * d.H;
    }
    const int64_t max_src_rows = wave_rows / (kWaveSlots * 8);
    std::vector<Keyed> keyed;
    for (int32_t b = 0; b < n; ++b) {
        const vp::DevItem& d = p->items[b];
        if (d.route != vp::kRouteStream) continue;
        const StreamShape& sh = shapes[b];
        const UnitSplit split(d.h, unit_row_band(d, max_src_rows, 4), 4);
        for (int32_t k = 0; k < d.t; ++k) {
            for (int64_t u = 0; u < split.n; ++u) {
                const int32_t i0 = split.begin(u), i1 = split.end(u);
                Keyed e;
                e.key = std::make_tuple(sh.m, sh.kx, sh.px);
                e.bands = sh.bands;
                e.unit.item = b;
                e.unit.p_flags = k;
                e.unit.i0 = i0;
                e.unit.i1 = i1;
                e.cost = int64_t(i1 - i0) * d.H / d.h * d.W;
                keyed.push_back(e);
            }
        }
    }
    if (const int32_t st = assemble_launches(keyed, P, p); st != VP_OK) return st;

    p->off_items = 0;
    p->off_prefix = align_up(p->off_items + sizeof(vp::DevItem) * p->items.size());
    p->off_indices = align_up(p->off_prefix + sizeof(int32_t) * p->prefix.size());
    p->off_tables = align_up(p->off_indices + sizeof(int32_t) * p->indices.size());
    p->off_units = align_up(p->off_tables + sizeof(int32_t) * p->table_words);
    p->off_wgs = align_up(p->off_units + sizeof(vp::StreamUnit) * p->units.size());
    p->bytes = align_up(p->off_wgs + sizeof(uint32_t) * p->wgs.size());
    return VP_OK;
}

// ---------------------------------------------------------------------------
// Plan cache.  An RL loop or a serving loop hands the library the same batch
// (the same frame buffers, sizes and index lists) call after call; its plan
// is a pure function of those, so the last few plans are kept and reused
// when every field and every index matches.  Entries are immutable and
// shared by pointer; a cache holds kPlanCacheMax plans, the most recently
// used first.
// ---------------------------------------------------------------------------

enum class PlanKind : int64_t { kBatch = 1, kPatch = 2, kResize = 3, kRows = 4 };

constexpr size_t kPlanCacheMax = 8;
std::mutex g_plan_mu;
std::list<std::pair<std::vector<int64_t>, std::shared_ptr<const Plan>>> g_plans;

int32_t build_kind(PlanKind kind, const vp_item* items, int32_t n, Plan* p) {
    switch (kind) {
        case PlanKind::kBatch: return build_plan(items, n, p);
        case PlanKind::kPatch: return build_patch_plan(items, n, p);
        case PlanKind::kResize: return build_resize_plan(items, n, p);
        case PlanKind::kRows: return build_rows_plan(items, n, p);
    }
    return fail(VP_ERR_ARG, "unknown plan kind");
}

// The plan of `items` for `kind`: from the cache if an identical batch was
// planned recently, else built (and cached if valid).  Errors are those of
// the builder; nothing invalid is cached.
int32_t get_plan(PlanKind kind, const vp_item* items, int32_t n, std::shared_ptr<const Plan>* out) {
    bool cacheable = items != nullptr && n >= 1;
    for (int32_t b = 0; cacheable && b < n; ++b)
        cacheable = items[b].indices != nullptr && items[b].n_idx >= 1;
    if (!cacheable) {   // the builder reports the error
        Plan p;
        const int32_t st = build_kind(kind, items, n, &p);
        if (st == VP_OK) *out = std::make_shared<const Plan>(std::move(p));
        return st;
    }
    std::vector<int64_t> key;
    key.reserve(2 + size_t(n) * 8);
    key.push_back(static_cast<int64_t>(kind));
    key.push_back(n);
    for (int32_t b = 0; b < n; ++b) {
        const vp_item& it = items[b];
        key.insert(key.end(), {static_cast<int64_t>(reinterpret_cast<uintptr_t>(it.frames)), it.n_src,
                               it.src_h, it.src_w, it.n_idx, it.dst_h, it.dst_w, it.patch});
        key.insert(key.end(), it.indices, it.indices + it.n_idx);
    }
    {
        std::lock_guard<std::mutex> lk(g_plan_mu);
        for (auto e = g_plans.begin(); e != g_plans.end(); ++e)
            if (e->first == key) {
                g_plans.splice(g_plans.begin(), g_plans, e);   // most recent first
                *out = e->second;
                return VP_OK;
            }
    }
    Plan p;
    const int32_t st = build_kind(kind, items, n, &p);
    if (st != VP_OK) return st;
    auto plan = std::make_shared<const Plan>(std::move(p));
    std::lock_guard<std::mutex> lk(g_plan_mu);
    g_plans.emplace_front(std::move(key), plan);
    if (g_plans.size() > kPlanCacheMax) g_plans.pop_back();
    *out = std::move(plan);
    return VP_OK;
}

// ---------------------------------------------------------------------------
// Pinned staging ring: the plan blob is written into pinned host memory and
// copied asynchronously; a slot is reused only after the copy that read it
// has completed.
// ---------------------------------------------------------------------------

struct Slot {
    void* host = nullptr;
    size_t cap = 0;
    hipEvent_t done = nullptr;
    bool pending = false;
};

struct Ring {
    std::mutex mu;
    Slot slots[4];
    int next = 0;
};

std::mutex g_rings_mu;
std::map<int, Ring*> g_rings;

Ring* ring_for_device(int dev) {
    std::lock_guard<std::mutex> lk(g_rings_mu);
    Ring*& r = g_rings[dev];
    if (r == nullptr) r = new Ring();  // lives until process exit
    return r;
}

int32_t hip_fail(hipError_t e, const char* what) {
    return fail(VP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Writes the plan blob (p.bytes bytes, the layout of vp_plan.h) to `base`:
// each section, then zeros up to the next one (the gaps are never read;
// zeroing them keeps the blob deterministic).
void pack_plan(const Plan& p, uint8_t* base) {
    auto put = [&](size_t off, const void* src, size_t n, size_t next) {
        if (n != 0) std::memcpy(base + off, src, n);
        std::memset(base + off + n, 0, next - off - n);
    };
    put(p.off_items, p.items.data(), sizeof(vp::DevItem) * p.items.size(), p.off_prefix);
    put(p.off_prefix, p.prefix.data(), sizeof(int32_t) * p.prefix.size(), p.off_indices);
    put(p.off_indices, p.indices.data(), sizeof(int32_t) * p.indices.size(), p.off_tables);
    for (const auto& part : p.tables)
        std::memcpy(base + p.off_tables + sizeof(int32_t) * part.first, part.second->data(),
                    sizeof(int32_t) * part.second->size());
    put(p.off_tables + sizeof(int32_t) * p.table_words, nullptr, 0, p.off_units);
    put(p.off_units, p.units.data(), sizeof(vp::StreamUnit) * p.units.size(), p.off_wgs);
    put(p.off_wgs, p.wgs.data(), sizeof(uint32_t) * p.wgs.size(), p.bytes);
}

int32_t upload_plan(const Plan& p, void* workspace, hipStream_t stream) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    Ring* ring = ring_for_device(dev);
    std::lock_guard<std::mutex> lk(ring->mu);
    Slot& s = ring->slots[ring->next];
    ring->next = (ring->next + 1) % 4;
    if (s.pending) {
        e = hipEventSynchronize(s.done);
        if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
        s.pending = false;
    }
    if (s.done == nullptr) {
        e = hipEventCreateWithFlags(&s.done, hipEventDisableTiming);
        if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
    }
    if (s.cap < p.bytes) {
        if (s.host != nullptr) (void)hipHostFree(s.host);
        s.host = nullptr;
        s.cap = 0;
        size_t cap = align_up(p.bytes * 2);
        e = hipHostMalloc(&s.host, cap, hipHostMallocDefault);
        if (e != hipSuccess) return hip_fail(e, "hipHostMalloc");
        s.cap = cap;
    }
    pack_plan(p, static_cast<uint8_t*>(s.host));
    e = hipMemcpyAsync(workspace, s.host, p.bytes, hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
    e = hipEventRecord(s.done, stream);
    if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
    s.pending = true;
    return VP_OK;
}

// ---------------------------------------------------------------------------
// Side streams.  The launches of one call (one per streaming-kernel shape,
// plus the general kernel) are independent of each other; on the caller's
// stream alone they would run one after another, and a small launch leaves
// most of the chip idle for the whole life of its longest workgroup.  Calls
// with several launches therefore fork to up to kSideStreams more streams of
// the device and join back with events, so the call stays one ordered step
// of the caller's stream.  The streams (default priority) and events are
// created on first use and kept until the process ends.
// ---------------------------------------------------------------------------

constexpr int kSideStreams = 3;

struct Side {
    std::mutex mu;   // held from fork to join: the events are shared by all calls
    bool ready = false;
    hipStream_t s[kSideStreams] = {};
    hipEvent_t fork = nullptr;
    hipEvent_t join[kSideStreams] = {};
};

std::mutex g_side_mu;
std::map<int, Side*> g_side;

int32_t side_for_device(int dev, Side** out) {
    Side* side = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_side_mu);
        Side*& r = g_side[dev];
        if (r == nullptr) r = new Side();   // lives until process exit
        side = r;
    }
    std::lock_guard<std::mutex> lk(side->mu);
    if (!side->ready) {
        hipError_t e = hipEventCreateWithFlags(&side->fork, hipEventDisableTiming);
        if (e != hipSuccess) return hip_fail(e, "hipEventCreate (fork)");
        for (int i = 0; i < kSideStreams; ++i) {
            e = hipStreamCreateWithFlags(&side->s[i], hipStreamNonBlocking);
            if (e != hipSuccess) return hip_fail(e, "hipStreamCreate (side stream)");
            e = hipEventCreateWithFlags(&side->join[i], hipEventDisableTiming);
            if (e != hipSuccess) return hip_fail(e, "hipEventCreate (join)");
        }
        side->ready = true;
    }
    *out = side;
    return VP_OK;
}

// Runs the plan's launches: on the caller's stream if there is one, else
// spread over the caller's stream and the side streams, largest estimated
// work first onto the least loaded stream.
// The plan's launches (the tile kernel, if it has tiles, and one per
// streaming shape), spread over the caller's stream and the side streams by
// estimated cost.  `resize`: the uint8 writer's kernels instead of the float
// path's (out_dtype and norm unused).
// With `one_stream` every launch goes to the caller's stream, one after
// another (no side streams, nothing created).
int32_t run_launches(const Plan& p, const vp::PlanView& view, void* out_rows, int32_t out_dtype,
                     const vp::Norm& norm, hipStream_t stream, bool resize = false,
                     bool one_stream = false) {
    struct Job {
        int32_t launch;   // index into p.launches, or -1 for the general kernel
        int64_t cost;
    };
    std::vector<Job> jobs;
    if (view.n_tiles > 0) jobs.push_back(Job{-1, p.generic_cost});
    for (size_t k = 0; k < p.launches.size(); ++k)
        jobs.push_back(Job{static_cast<int32_t>(k), p.launches[k].cost});
    auto launch = [&](const Job& j, hipStream_t st) -> int32_t {
        if (resize) {
            const int err = j.launch < 0 ? vp::launch_resize(view, out_rows, st)
                                         : vp::launch_resize_stream(view, p.launches[j.launch], out_rows, st);
            if (err != 0) return hip_fail(static_cast<hipError_t>(err), "uint8 writer launch");
        } else if (j.launch < 0) {
            const int err = vp::launch_generic(view, out_rows, out_dtype, norm, st);
            if (err != 0) return hip_fail(static_cast<hipError_t>(err), "general kernel launch");
        } else {
            const int err = vp::launch_stream(view, p.launches[j.launch], out_rows, out_dtype, norm, st);
            if (err != 0) return hip_fail(static_cast<hipError_t>(err), "streaming kernel launch");
        }
        return VP_OK;
    };
    if (jobs.size() <= 1) return jobs.empty() ? VP_OK : launch(jobs[0], stream);
    if (one_stream) {
        for (const Job& j : jobs)
            if (const int32_t st = launch(j, stream); st != VP_OK) return st;
        return VP_OK;
    }

    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    Side* side = nullptr;
    int32_t st = side_for_device(dev, &side);
    if (st != VP_OK) return st;
    std::stable_sort(jobs.begin(), jobs.end(), [](const Job& a, const Job& b) { return a.cost > b.cost; });
    const int lanes = std::min<int>(static_cast<int>(jobs.size()), kSideStreams + 1);
    std::vector<int> lane_of(jobs.size(), 0);
    std::vector<int64_t> load(lanes, 0);
    for (size_t k = 0; k < jobs.size(); ++k) {
        int best = 0;
        for (int l = 1; l < lanes; ++l)
            if (load[l] < load[best]) best = l;
        lane_of[k] = best;
        load[best] += jobs[k].cost;
    }
    std::lock_guard<std::mutex> lk(side->mu);
    e = hipEventRecord(side->fork, stream);
    if (e != hipSuccess) return hip_fail(e, "hipEventRecord (fork)");
    for (int l = 1; l < lanes; ++l) {
        e = hipStreamWaitEvent(side->s[l - 1], side->fork, 0);
        if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent (fork)");
    }
    st = VP_OK;
    for (size_t k = 0; k < jobs.size() && st == VP_OK; ++k)
        st = launch(jobs[k], lane_of[k] == 0 ? stream : side->s[lane_of[k] - 1]);
    // join even after a failed launch, so that the caller's stream still
    // orders after whatever was enqueued
    for (int l = 1; l < lanes; ++l) {
        e = hipEventRecord(side->join[l - 1], side->s[l - 1]);
        if (e == hipSuccess) e = hipStreamWaitEvent(stream, side->join[l - 1], 0);
        if (e != hipSuccess && st == VP_OK) st = hip_fail(e, "join of a side stream");
    }
    return st;
}

// Shared body of vp_preprocess_batch (resample + normalise + patchify),
// vp_patchify_batch (frames already at the target size) and
// vp_preprocess_batch_noalloc (no_alloc: the plan goes to the library's
// fixed device array instead of a workspace, copied from pageable host
// memory, and every launch runs on the caller's stream).
int32_t run_batch(bool patch_only, const vp_item* items, int32_t n_items, const float* mean,
                  const float* std, int32_t out_dtype, void* out_rows, int64_t out_rows_capacity,
                  int32_t* grid_thw, int32_t* cu_seqlens, void* workspace, int64_t workspace_bytes,
                  hipStream_t stream, bool no_alloc = false) {
    if (mean == nullptr || std == nullptr || out_rows == nullptr || (!no_alloc && workspace == nullptr))
        return fail(VP_ERR_NULL, no_alloc ? "mean, std and out_rows must be non-NULL"
                                          : "mean, std, out_rows and workspace must be non-NULL");
    if (out_dtype != VP_OUT_F32 && out_dtype != VP_OUT_BF16)
        return fail(VP_ERR_ARG, "out_dtype must be VP_OUT_F32 or VP_OUT_BF16");
    if (reinterpret_cast<uintptr_t>(out_rows) % 16 != 0)
        return fail(VP_ERR_ARG, "out_rows must be 16-byte aligned");
    if (!no_alloc && reinterpret_cast<uintptr_t>(workspace) % kAlign != 0)
        return fail(VP_ERR_ARG, "workspace must be 256-byte aligned");
    vp::Norm norm;
    for (int c = 0; c < 3; ++c) {
        if (!(std[c] > 0.0f) || !std::isfinite(std[c]) || !std::isfinite(mean[c]))
            return fail(VP_ERR_ARG, "std must be positive and finite, mean finite");
        norm.a[c] = static_cast<float>(1.0 / (255.0 * static_cast<double>(std[c])));
        norm.b[c] = static_cast<float>(-static_cast<double>(mean[c]) / static_cast<double>(std[c]));
        norm.z[c] = static_cast<float>(-255.0 * static_cast<double>(mean[c]));
    }
    std::shared_ptr<const Plan> plan;
    int32_t st = get_plan(patch_only ? PlanKind::kPatch : PlanKind::kBatch, items, n_items, &plan);
    if (st != VP_OK) return st;
    const Plan& p = *plan;
    if (out_rows_capacity < p.total_rows)
        return fail(VP_ERR_CAPACITY, "out_rows holds " + std::to_string(out_rows_capacity) +
                                         " rows, batch needs " + std::to_string(p.total_rows));
    if (no_alloc) {
        if (p.bytes > static_cast<size_t>(vp::kNoAllocPlanBytes))
            return fail(VP_ERR_CAPACITY, "the plan needs " + std::to_string(p.bytes) +
                                             " bytes; the library's fixed plan memory holds " +
                                             std::to_string(vp::kNoAllocPlanBytes));
        const int err = vp::noalloc_plan_memory(&workspace);
        if (err != 0) return hip_fail(static_cast<hipError_t>(err), "hipGetSymbolAddress (plan memory)");
        // pageable host memory: the copy has read it when hipMemcpyAsync returns
        thread_local std::vector<uint8_t> blob;
        if (blob.size() < p.bytes) blob.resize(p.bytes);
        pack_plan(p, blob.data());
        const hipError_t e = hipMemcpyAsync(workspace, blob.data(), p.bytes, hipMemcpyHostToDevice, stream);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (plan)");
    } else {
        if (workspace_bytes < static_cast<int64_t>(p.bytes))
            return fail(VP_ERR_CAPACITY, "workspace holds " + std::to_string(workspace_bytes) +
                                             " bytes, plan needs " + std::to_string(p.bytes));
        st = upload_plan(p, workspace, stream);
        if (st != VP_OK) return st;
    }
    hipEvent_t t_start = g_timing_start, t_stop = g_timing_stop;
    g_timing_start = g_timing_stop = nullptr;
    if (t_start != nullptr) {
        const hipError_t e = hipEventRecord(t_start, stream);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord (timing start)");
    }
    auto* ws = static_cast<uint8_t*>(workspace);
    vp::PlanView view;
    view.items = reinterpret_cast<const vp::DevItem*>(ws + p.off_items);
    view.tile_prefix = reinterpret_cast<const int32_t*>(ws + p.off_prefix);
    view.indices = reinterpret_cast<const int32_t*>(ws + p.off_indices);
    view.tables = reinterpret_cast<const int32_t*>(ws + p.off_tables);
    view.units = reinterpret_cast<const vp::StreamUnit*>(ws + p.off_units);
    view.wgs = reinterpret_cast<const uint32_t*>(ws + p.off_wgs);
    view.n_items = n_items;
    view.n_tiles = p.prefix[n_items];
    if (patch_only) {
        const int err = vp::launch_patchify(view, out_rows, out_dtype, norm, p.items[0].patch, stream);
        if (err != 0) return hip_fail(static_cast<hipError_t>(err), "patchify kernel launch");
    } else {
        st = run_launches(p, view, out_rows, out_dtype, norm, stream, false, no_alloc);
        if (st != VP_OK) return st;
    }
    if (t_stop != nullptr) {
        const hipError_t e = hipEventRecord(t_stop, stream);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord (timing stop)");
    }
    if (grid_thw) std::memcpy(grid_thw, p.grid.data(), sizeof(int32_t) * p.grid.size());
    if (cu_seqlens) std::memcpy(cu_seqlens, p.cu.data(), sizeof(int32_t) * p.cu.size());
    g_last_error.clear();
    return VP_OK;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================

extern "C" {

int32_t vp_smart_resize_dims(int32_t height, int32_t width, int32_t factor, int64_t min_pixels,
                             int64_t max_pixels, int32_t* out_h, int32_t* out_w) {
    if (out_h == nullptr || out_w == nullptr) return fail(VP_ERR_NULL, "output pointer is NULL");
    if (height <= 0 || width <= 0 || factor <= 0 || max_pixels <= 0 || min_pixels < 0 ||
        min_pixels > max_pixels)
        return fail(VP_ERR_ARG, "smart_resize: sizes, factor and max_pixels must be positive, "
                                "0 <= min_pixels <= max_pixels");
    const double H = height, W = width, F = factor;
    const double ratio = height > width ? H / W : W / H;
    if (ratio > 200.0) return fail(VP_ERR_ASPECT, "smart_resize: aspect ratio above 200");
    int64_t h = static_cast<int64_t>(nearest_even(H / F)) * factor;
    int64_t w = static_cast<int64_t>(nearest_even(W / F)) * factor;
    if (h < factor) h = factor;
    if (w < factor) w = factor;
    if (h * w > max_pixels) {
        const double beta = std::sqrt(static_cast<double>(int64_t(height) * width) /
                                      static_cast<double>(max_pixels));
        h = static_cast<int64_t>(std::floor(H / beta / F)) * factor;
        w = static_cast<int64_t>(std::floor(W / beta / F)) * factor;
        if (h < factor) h = factor;
        if (w < factor) w = factor;
    } else if (h * w < min_pixels) {
        const double beta = std::sqrt(static_cast<double>(min_pixels) /
                                      static_cast<double>(int64_t(height) * width));
        h = static_cast<int64_t>(std::ceil(H * beta / F)) * factor;
        w = static_cast<int64_t>(std::ceil(W * beta / F)) * factor;
    }
    if (h > INT32_MAX || w > INT32_MAX) return fail(VP_ERR_DIMS, "smart_resize: result too large");
    *out_h = static_cast<int32_t>(h);
    *out_w = static_cast<int32_t>(w);
    return VP_OK;
}

int32_t vp_sample_indices(int32_t total_frames, int32_t mode, int32_t nframes, double video_fps,
                          double fps, int32_t min_frames, int32_t max_frames, int32_t* out_idx,
                          int32_t capacity, int32_t* out_count) {
    if (out_count == nullptr) return fail(VP_ERR_NULL, "out_count is NULL");
    if (total_frames < 1) return fail(VP_ERR_FRAMES, "total_frames < 1");
    int64_t n = 0;
    if (mode == VP_SAMPLE_UNIFORM) {
        if (nframes < 1 || nframes > total_frames)
            return fail(VP_ERR_FRAMES, "uniform sampling needs 1 <= nframes <= total_frames");
        n = nframes;
    } else if (mode == VP_SAMPLE_FPS) {
        if (!(video_fps > 0.0) || !(fps > 0.0) || min_frames < 1 || max_frames < min_frames)
            return fail(VP_ERR_ARG, "fps sampling needs video_fps, fps > 0 and "
                                    "1 <= min_frames <= max_frames");
        const double lo = static_cast<double>((int64_t(min_frames) + 1) / 2 * 2);
        const double hi = static_cast<double>(int64_t(max_frames) / 2 * 2);
        double want = static_cast<double>(total_frames) / video_fps * fps;
        want = want < lo ? lo : want;
        want = want > hi ? hi : want;
        want = want > total_frames ? static_cast<double>(total_frames) : want;
        n = static_cast<int64_t>(std::floor(want / 2.0)) * 2;
        if (n < 2) return fail(VP_ERR_FRAMES, "fps sampling yields fewer than 2 frames");
    } else {
        return fail(VP_ERR_ARG, "unknown sampling mode");
    }
    *out_count = static_cast<int32_t>(n);
    if (out_idx == nullptr || capacity < n)
        return fail(VP_ERR_CAPACITY, "index buffer holds " + std::to_string(capacity) + " of " +
                                         std::to_string(n) + " indices");
    for (int64_t i = 0; i < n; ++i) out_idx[i] = spread_index(i, total_frames - 1, n);
    return VP_OK;
}

int32_t vp_filter_taps(int32_t n_in, int32_t n_out, int32_t* max_taps) {
    if (max_taps == nullptr) return fail(VP_ERR_NULL, "max_taps is NULL");
    if (n_in < 1 || n_out < 1) return fail(VP_ERR_ARG, "n_in and n_out must be >= 1");
    *max_taps = axis_taps(n_in, n_out);
    return VP_OK;
}

int32_t vp_filter_table(int32_t n_in, int32_t n_out, int32_t taps, int32_t* start, int32_t* count,
                        float* weights) {
    if (start == nullptr || count == nullptr || weights == nullptr)
        return fail(VP_ERR_NULL, "output pointer is NULL");
    if (n_in < 1 || n_out < 1) return fail(VP_ERR_ARG, "n_in and n_out must be >= 1");
    const int32_t need = axis_taps(n_in, n_out);
    if (taps < need) return fail(VP_ERR_CAPACITY, "taps below the longest window");
    AxisFilter f;
    build_axis(n_in, n_out, taps, &f);
    std::memcpy(start, f.start.data(), sizeof(int32_t) * n_out);
    std::memcpy(count, f.count.data(), sizeof(int32_t) * n_out);
    std::memcpy(weights, f.weight.data(), sizeof(float) * f.weight.size());
    return VP_OK;
}

int32_t vp_filter_table_fixed(int32_t n_in, int32_t n_out, int32_t taps, int32_t* start,
                              int32_t* count, int32_t* q) {
    if (start == nullptr || count == nullptr || q == nullptr)
        return fail(VP_ERR_NULL, "output pointer is NULL");
    if (n_in < 1 || n_out < 1) return fail(VP_ERR_ARG, "n_in and n_out must be >= 1");
    const int32_t need = axis_taps(n_in, n_out);
    if (taps < need) return fail(VP_ERR_CAPACITY, "taps below the longest window");
    AxisFilter f;
    build_axis(n_in, n_out, taps, &f);
    std::memcpy(start, f.start.data(), sizeof(int32_t) * n_out);
    std::memcpy(count, f.count.data(), sizeof(int32_t) * n_out);
    std::memcpy(q, f.fixed.data(), sizeof(int32_t) * f.fixed.size());
    return VP_OK;
}

int32_t vp_batch_layout(const vp_item* items, int32_t n_items, int32_t* grid_thw,
                        int32_t* cu_seqlens, int64_t* total_rows, int64_t* workspace_bytes) {
    std::shared_ptr<const Plan> plan;
    const int32_t st = get_plan(PlanKind::kBatch, items, n_items, &plan);
    if (st != VP_OK) return st;
    const Plan& p = *plan;
    if (grid_thw) std::memcpy(grid_thw, p.grid.data(), sizeof(int32_t) * p.grid.size());
    if (cu_seqlens) std::memcpy(cu_seqlens, p.cu.data(), sizeof(int32_t) * p.cu.size());
    if (total_rows) *total_rows = p.total_rows;
    if (workspace_bytes) *workspace_bytes = static_cast<int64_t>(p.bytes);
    return VP_OK;
}

int32_t vp_batch_kernels(const vp_item* items, int32_t n_items, int32_t* launches,
                         int32_t capacity, int32_t* n_launches) {
    if (n_launches == nullptr) return fail(VP_ERR_NULL, "n_launches is NULL");
    if (capacity < 0 || (launches == nullptr && capacity > 0))
        return fail(VP_ERR_ARG, "launches must hold capacity rows of 6 int32");
    std::shared_ptr<const Plan> plan;
    const int32_t st = get_plan(PlanKind::kBatch, items, n_items, &plan);
    if (st != VP_OK) return st;
    const Plan& p = *plan;
    std::vector<std::array<int32_t, 6>> rows;
    if (p.prefix[n_items] > 0) rows.push_back({VP_KERNEL_GENERIC, 0, 0, 0, 0, p.prefix[n_items]});
    for (const vp::StreamLaunch& L : p.launches) {
        if (L.px < 0)
            rows.push_back({VP_KERNEL_XFIRST, L.m, L.kx, 0, vp::xfirst_db(L.px) > 0 ? 2 : 1, L.count});
        else
            rows.push_back({VP_KERNEL_YFIRST, L.m, L.kx, L.px, 0, L.count});
    }
    for (size_t i = 0; i < rows.size() && i < size_t(capacity); ++i)
        std::memcpy(launches + 6 * i, rows[i].data(), sizeof(int32_t) * 6);
    *n_launches = static_cast<int32_t>(rows.size());
    return VP_OK;
}

int32_t vp_preprocess_batch(const vp_item* items, int32_t n_items, const float* mean,
                            const float* std, int32_t out_dtype, void* out_rows,
                            int64_t out_rows_capacity, int32_t* grid_thw, int32_t* cu_seqlens,
                            void* workspace, int64_t workspace_bytes, hipStream_t stream) {
    return run_batch(false, items, n_items, mean, std, out_dtype, out_rows, out_rows_capacity,
                     grid_thw, cu_seqlens, workspace, workspace_bytes, stream);
}

int32_t vp_preprocess_batch_noalloc(const vp_item* items, int32_t n_items, const float* mean,
                                    const float* std, int32_t out_dtype, void* out_rows,
                                    int64_t out_rows_capacity, int32_t* grid_thw,
                                    int32_t* cu_seqlens, hipStream_t stream) {
    return run_batch(false, items, n_items, mean, std, out_dtype, out_rows, out_rows_capacity,
                     grid_thw, cu_seqlens, nullptr, 0, stream, true);
}

int32_t vp_patchify_batch(const vp_item* items, int32_t n_items, const float* mean,
                          const float* std, int32_t out_dtype, void* out_rows,
                          int64_t out_rows_capacity, int32_t* grid_thw, int32_t* cu_seqlens,
                          void* workspace, int64_t workspace_bytes, hipStream_t stream) {
    return run_batch(true, items, n_items, mean, std, out_dtype, out_rows, out_rows_capacity,
                     grid_thw, cu_seqlens, workspace, workspace_bytes, stream);
}
int32_t vp_resize_layout(const vp_item* items, int32_t n_items, int64_t* frame_off,
                         int64_t* workspace_bytes) {
    std::shared_ptr<const Plan> plan;
    const int32_t st = get_plan(PlanKind::kResize, items, n_items, &plan);
    if (st != VP_OK) return st;
    const Plan& p = *plan;
    if (frame_off) std::memcpy(frame_off, p.byte_off.data(), sizeof(int64_t) * p.byte_off.size());
    if (workspace_bytes) *workspace_bytes = static_cast<int64_t>(p.bytes);
    g_last_error.clear();
    return VP_OK;
}

int32_t vp_resize_batch(const vp_item* items, int32_t n_items, void* out_frames,
                        int64_t out_capacity, int64_t* frame_off, void* workspace,
                        int64_t workspace_bytes, hipStream_t stream) {
    if (out_frames == nullptr || workspace == nullptr)
        return fail(VP_ERR_NULL, "out_frames and workspace must be non-NULL");
    if (reinterpret_cast<uintptr_t>(out_frames) % 4 != 0)
        return fail(VP_ERR_ARG, "out_frames must be 4-byte aligned");
    if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0)
        return fail(VP_ERR_ARG, "workspace must be 256-byte aligned");
    std::shared_ptr<const Plan> plan;
    int32_t st = get_plan(PlanKind::kResize, items, n_items, &plan);
    if (st != VP_OK) return st;
    const Plan& p = *plan;
    if (out_capacity < p.byte_off[n_items])
        return fail(VP_ERR_CAPACITY, "out_frames holds " + std::to_string(out_capacity) +
                                         " bytes, batch needs " + std::to_string(p.byte_off[n_items]));
    if (workspace_bytes < static_cast<int64_t>(p.bytes))
        return fail(VP_ERR_CAPACITY, "workspace holds " + std::to_string(workspace_bytes) +
                                         " bytes, plan needs " + std::to_string(p.bytes));
    st = upload_plan(p, workspace, stream);
    if (st != VP_OK) return st;
    hipEvent_t t_start = g_timing_start, t_stop = g_timing_stop;
    g_timing_start = g_timing_stop = nullptr;
    if (t_start != nullptr) {
        const hipError_t e = hipEventRecord(t_start, stream);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord (timing start)");
    }
    auto* ws = static_cast<uint8_t*>(workspace);
    vp::PlanView view{};
    view.items = reinterpret_cast<const vp::DevItem*>(ws + p.off_items);
    view.tile_prefix = reinterpret_cast<const int32_t*>(ws + p.off_prefix);
    view.indices = reinterpret_cast<const int32_t*>(ws + p.off_indices);
    view.tables = reinterpret_cast<const int32_t*>(ws + p.off_tables);
    view.units = reinterpret_cast<const vp::StreamUnit*>(ws + p.off_units);
    view.wgs = reinterpret_cast<const uint32_t*>(ws + p.off_wgs);
    view.n_items = n_items;
    view.n_tiles = p.prefix[n_items];
    st = run_launches(p, view, out_frames, 0, vp::Norm{}, stream, true);
    if (st != VP_OK) return st;
    if (t_stop != nullptr) {
        const hipError_t e = hipEventRecord(t_stop, stream);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord (timing stop)");
    }
    if (frame_off) std::memcpy(frame_off, p.byte_off.data(), sizeof(int64_t) * p.byte_off.size());
    g_last_error.clear();
    return VP_OK;
}

int32_t vp_position_ids(const vp_item* items, int32_t n_items, int32_t* vit_pos,
                        int32_t* llm_pos, int64_t rows_capacity, int32_t* vit_cu,
                        int32_t vit_cu_capacity, int32_t* n_slices, void* workspace,
                        int64_t workspace_bytes, hipStream_t stream) {
    if (workspace == nullptr) return fail(VP_ERR_NULL, "workspace must be non-NULL");
    if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0)
        return fail(VP_ERR_ARG, "workspace must be 256-byte aligned");
    if (reinterpret_cast<uintptr_t>(vit_pos) % 4 != 0 || reinterpret_cast<uintptr_t>(llm_pos) % 4 != 0)
        return fail(VP_ERR_ARG, "vit_pos and llm_pos must be 4-byte aligned");
    std::shared_ptr<const Plan> plan;
    int32_t st = get_plan(PlanKind::kRows, items, n_items, &plan);
    if (st != VP_OK) return st;
    const Plan& p = *plan;
    if ((vit_pos != nullptr || llm_pos != nullptr) && rows_capacity < p.total_rows)
        return fail(VP_ERR_CAPACITY, "position tables hold " + std::to_string(rows_capacity) +
                                         " rows, batch needs " + std::to_string(p.total_rows));
    int64_t slices = 0;
    for (int32_t b = 0; b < n_items; ++b) slices += p.items[b].t;
    if (vit_cu != nullptr && vit_cu_capacity < slices + 1)
        return fail(VP_ERR_CAPACITY, "vit_cu holds " + std::to_string(vit_cu_capacity) +
                                         " entries, batch needs " + std::to_string(slices + 1));
    if (workspace_bytes < static_cast<int64_t>(p.bytes))
        return fail(VP_ERR_CAPACITY, "workspace holds " + std::to_string(workspace_bytes) +
                                         " bytes, plan needs " + std::to_string(p.bytes));
    hipEvent_t t_start = g_timing_start, t_stop = g_timing_stop;
    g_timing_start = g_timing_stop = nullptr;
    if (vit_pos != nullptr || llm_pos != nullptr) {
        st = upload_plan(p, workspace, stream);
        if (st != VP_OK) return st;
        if (t_start != nullptr) {
            const hipError_t e = hipEventRecord(t_start, stream);
            if (e != hipSuccess) return hip_fail(e, "hipEventRecord (timing start)");
        }
        auto* ws = static_cast<uint8_t*>(workspace);
        vp::PlanView view{};
        view.items = reinterpret_cast<const vp::DevItem*>(ws + p.off_items);
        view.tile_prefix = reinterpret_cast<const int32_t*>(ws + p.off_prefix);
        view.indices = reinterpret_cast<const int32_t*>(ws + p.off_indices);
        view.n_items = n_items;
        view.n_tiles = 0;
        const int err = vp::launch_positions(view, vit_pos, llm_pos, p.total_rows, stream);
        if (err != 0) return hip_fail(static_cast<hipError_t>(err), "position kernel launch");
        if (t_stop != nullptr) {
            const hipError_t e = hipEventRecord(t_stop, stream);
            if (e != hipSuccess) return hip_fail(e, "hipEventRecord (timing stop)");
        }
    }
    if (vit_cu != nullptr) {
        int64_t s = 0;
        vit_cu[0] = 0;
        for (int32_t b = 0; b < n_items; ++b)
            for (int32_t k = 0; k < p.items[b].t; ++k, ++s)
                vit_cu[s + 1] = vit_cu[s] + p.grid[3 * b + 1] * p.grid[3 * b + 2];
    }
    if (n_slices) *n_slices = static_cast<int32_t>(slices);
    g_last_error.clear();
    return VP_OK;
}

const char* vp_status_string(int32_t status) {
    switch (status) {
        case VP_OK: return "VP_OK";
        case VP_ERR_NULL: return "VP_ERR_NULL";
        case VP_ERR_ARG: return "VP_ERR_ARG";
        case VP_ERR_ASPECT: return "VP_ERR_ASPECT";
        case VP_ERR_DIMS: return "VP_ERR_DIMS";
        case VP_ERR_INDEX: return "VP_ERR_INDEX";
        case VP_ERR_FRAMES: return "VP_ERR_FRAMES";
        case VP_ERR_CAPACITY: return "VP_ERR_CAPACITY";
        case VP_ERR_HIP: return "VP_ERR_HIP";
        default: return "VP_ERR_UNKNOWN";
    }
}

int32_t vp_set_kernel_events(hipEvent_t start, hipEvent_t stop) {
    if ((start == nullptr) != (stop == nullptr))
        return fail(VP_ERR_NULL, "vp_set_kernel_events needs both events or neither");
    g_timing_start = start;
    g_timing_stop = stop;
    g_last_error.clear();
    return VP_OK;
}

const char* vp_last_error_message(void) { return g_last_error.c_str(); }

}  // extern "C"
