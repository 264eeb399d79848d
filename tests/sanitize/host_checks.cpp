// Host-side checks under AddressSanitizer and UndefinedBehaviorSanitizer
// (built and run by tests/test_host_sanitizers.py on the CPU; no GPU).
//
// Drives every host path of the library's C ABI -- smart_resize, index
// sampling, the float and fixed-point filter tables, the batch planner of
// every entry point (through vp_batch_layout, vp_batch_kernels,
// vp_resize_layout and the host part of vp_position_ids), the plan cache,
// column pairs of the x-first kernel in a large batch, and the checks that
// return before any HIP call -- and every function of the oracle, over
// seeded random shapes, degenerate sizes and the workloads' own batches.
// A sanitizer report aborts the run; the exit status is 0 only if every
// call returned a status and nothing was reported.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "vp.h"

extern "C" {
int oracle_smart_resize(int64_t, int64_t, int64_t, int64_t, int64_t, int64_t*, int64_t*);
int oracle_sample_uniform(int64_t, int64_t, int32_t*);
int oracle_sample_fps(int64_t, double, double, int64_t, int64_t, int32_t*, int64_t, int64_t*);
int oracle_filter(int64_t, int64_t, int64_t, int64_t*, int64_t*, double*, int64_t);
int64_t oracle_filter_max_taps(int64_t, int64_t);
int oracle_filter_table(int64_t, int64_t, int64_t*, int64_t*, double*, int64_t);
int oracle_resize_frame(const uint8_t*, int64_t, int64_t, int64_t, int64_t, double*);
double oracle_resize_pixel(const uint8_t*, int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, int64_t);
int oracle_fixed_weights(int64_t, int64_t, int64_t, int64_t*, int64_t*, int32_t*, int64_t);
int oracle_resize_u8(const uint8_t*, int64_t, int64_t, int64_t, int64_t, uint8_t*);
int oracle_resize_u8_item(const uint8_t*, int64_t, int64_t, int64_t, const int32_t*, int64_t, int64_t,
                          int64_t, int64_t, uint8_t*);
int64_t oracle_item_rows(int64_t, int64_t, int64_t, int64_t);
int oracle_preprocess_item(const uint8_t*, int64_t, int64_t, int64_t, const int32_t*, int64_t, int64_t,
                           int64_t, int64_t, const double*, const double*, double*);
int oracle_patchify_item(const uint8_t*, int64_t, int64_t, int64_t, const int32_t*, int64_t, int64_t,
                         const double*, const double*, double*);
int oracle_item_row(const uint8_t*, int64_t, int64_t, int64_t, const int32_t*, int64_t, int64_t, int64_t,
                    int64_t, const double*, const double*, int64_t, double*);
int oracle_position_ids(int64_t, const int64_t*, const int64_t*, const int64_t*, int64_t, int64_t*,
                        int64_t*, int64_t*, int64_t*);
int oracle_layout(int64_t, const int64_t*, const int64_t*, const int64_t*, int64_t, int64_t*, int64_t*);
}

namespace {

std::mt19937_64 rng(2604'16893);
int64_t calls = 0, ok_calls = 0;

int64_t uni(int64_t lo, int64_t hi) { return std::uniform_int_distribution<int64_t>(lo, hi)(rng); }

void count(int32_t st) {
    ++calls;
    ok_calls += st == VP_OK;
}

// A fake device pointer: the host paths never dereference frame pointers.
const uint8_t* fake_frames(int64_t k) { return reinterpret_cast<const uint8_t*>(uintptr_t(0x100000) + 4096 * k); }

struct Batch {
    std::vector<vp_item> items;
    std::vector<std::vector<int32_t>> idx;
};

Batch random_batch(int patch, int max_items, int max_side) {
    Batch b;
    const int n = int(uni(1, max_items));
    b.idx.resize(n);
    for (int k = 0; k < n; ++k) {
        vp_item it{};
        const int F = 2 * patch;
        it.frames = fake_frames(k);
        it.n_src = int32_t(uni(1, 300));
        it.src_h = int32_t(uni(1, max_side));
        it.src_w = int32_t(uni(1, max_side));
        const int64_t mode = uni(0, 3);
        if (mode == 0) {   // near the source size
            it.dst_h = int32_t(std::max<int64_t>(F, (it.src_h + F / 2) / F * F));
            it.dst_w = int32_t(std::max<int64_t>(F, (it.src_w + F / 2) / F * F));
        } else {
            it.dst_h = int32_t(F * uni(1, 40));
            it.dst_w = int32_t(F * uni(1, 40));
        }
        it.n_idx = int32_t(uni(1, 64));
        b.idx[k].resize(it.n_idx);
        for (auto& v : b.idx[k]) v = int32_t(uni(0, it.n_src - 1));
        if (uni(0, 20) == 0) b.idx[k][0] = it.n_src;   // an out-of-range index: VP_ERR_INDEX
        it.patch = patch == 16 && uni(0, 1) ? 0 : patch;
        b.items.push_back(it);
    }
    for (int k = 0; k < n; ++k) b.items[k].indices = b.idx[k].data();
    return b;
}

void library_host_paths() {
    // smart_resize and sampling
    for (int r = 0; r < 20000; ++r) {
        int32_t h = 0, w = 0;
        const int64_t maxp = uni(0, 2) ? uni(1, int64_t(1) << 24) : uni(-5, 5);
        count(vp_smart_resize_dims(int32_t(uni(-2, 20000)), int32_t(uni(-2, 20000)),
                                   uni(0, 1) ? 32 : 28, uni(-1, 70000), maxp, &h, &w));
        std::vector<int32_t> out(512);
        int32_t n = 0;
        count(vp_sample_indices(int32_t(uni(-1, 5000)), int32_t(uni(0, 2)), int32_t(uni(-1, 600)),
                                double(uni(-1, 60)), double(uni(-1, 8)), int32_t(uni(-1, 300)),
                                int32_t(uni(-1, 600)), out.data(), int32_t(out.size()), &n));
    }
    count(vp_sample_indices(100, VP_SAMPLE_UNIFORM, 10, 0, 0, 1, 1, nullptr, 0, nullptr));
    // filter tables, exactly sized
    for (int r = 0; r < 400; ++r) {
        const int32_t n_in = int32_t(uni(1, r % 10 == 0 ? 40000 : 4000));
        const int32_t n_out = int32_t(uni(1, 2048));
        int32_t taps = 0;
        count(vp_filter_taps(n_in, n_out, &taps));
        if (taps < 1 || int64_t(taps) * n_out > (int64_t(1) << 26)) continue;
        std::vector<int32_t> start(n_out), cnt(n_out), q(size_t(taps) * n_out);
        std::vector<float> wt(size_t(taps) * n_out);
        count(vp_filter_table(n_in, n_out, taps, start.data(), cnt.data(), wt.data()));
        count(vp_filter_table_fixed(n_in, n_out, taps, start.data(), cnt.data(), q.data()));
        count(vp_filter_table(n_in, n_out, taps - 1, start.data(), cnt.data(), wt.data()));   // too few taps
    }
    // planners of every entry point, over random ragged batches
    for (int r = 0; r < 300; ++r) {
        const int patch = r % 3 == 2 ? 14 : 16;
        Batch b = random_batch(patch, 24, r % 7 == 0 ? 6000 : 1500);
        const int32_t n = int32_t(b.items.size());
        std::vector<int32_t> grid(size_t(n) * 3), cu(n + 1);
        int64_t rows = 0, ws = 0;
        const int32_t st = vp_batch_layout(b.items.data(), n, grid.data(), cu.data(), &rows, &ws);
        count(st);
        count(vp_batch_layout(b.items.data(), n, nullptr, nullptr, nullptr, nullptr));   // a cache hit
        {
            int32_t nl = 0;
            std::vector<int32_t> launches(6 * 2);
            count(vp_batch_kernels(b.items.data(), n, launches.data(), 2, &nl));   // maybe fewer rows than launches
            launches.assign(size_t(6) * (nl > 0 ? nl : 1), 0);
            count(vp_batch_kernels(b.items.data(), n, launches.data(), nl, &nl));
        }
        std::vector<int64_t> off(n + 1);
        count(vp_resize_layout(b.items.data(), n, off.data(), &ws));
        int64_t slices = 0;
        for (const auto& it : b.items) slices += (it.n_idx + 1) / 2;
        std::vector<int32_t> vit_cu(slices + 1);
        int32_t ns = 0;
        count(vp_position_ids(b.items.data(), n, nullptr, nullptr, 0, vit_cu.data(), int32_t(vit_cu.size()),
                              &ns, reinterpret_cast<void*>(0x200000), int64_t(1) << 40, nullptr));
        // argument checks that return before any HIP call
        const float mean[3] = {0.5f, 0.5f, 0.5f}, bad_std[3] = {0.5f, 0.f, 0.5f};
        count(vp_preprocess_batch(b.items.data(), n, mean, bad_std, VP_OUT_BF16, reinterpret_cast<void*>(0x300000),
                                  int64_t(1) << 40, grid.data(), cu.data(), reinterpret_cast<void*>(0x200000),
                                  int64_t(1) << 40, nullptr));
        if (st == VP_OK) {
            count(vp_preprocess_batch(b.items.data(), n, mean, mean, VP_OUT_F32, reinterpret_cast<void*>(0x300000),
                                      rows - 1, nullptr, nullptr, reinterpret_cast<void*>(0x200000), ws, nullptr));
            count(vp_preprocess_batch(b.items.data(), n, mean, mean, VP_OUT_F32, reinterpret_cast<void*>(0x300000),
                                      rows, nullptr, nullptr, reinterpret_cast<void*>(0x200000), ws - 1, nullptr));
            count(vp_patchify_batch(b.items.data(), n, mean, mean, VP_OUT_F32, reinterpret_cast<void*>(0x300000),
                                    rows, nullptr, nullptr, reinterpret_cast<void*>(0x200000), ws, nullptr));
            count(vp_preprocess_batch_noalloc(b.items.data(), n, mean, mean, 7, reinterpret_cast<void*>(0x300000),
                                              rows, nullptr, nullptr, nullptr));
        }
    }
    // the workloads' own batches: 720p -> 256x448 (64 x 256 frames) and a mixed one
    {
        std::vector<std::vector<int32_t>> idx(64, std::vector<int32_t>(256));
        std::vector<vp_item> items(64);
        for (int k = 0; k < 64; ++k) {
            for (int i = 0; i < 256; ++i) idx[k][i] = i;
            items[k] = vp_item{fake_frames(k), idx[k].data(), 256, 720, 1280, 256, 256, 448, 16};
        }
        int64_t rows = 0, ws = 0;
        for (int rep = 0; rep < 3; ++rep) count(vp_batch_layout(items.data(), 64, nullptr, nullptr, &rows, &ws));
        count(vp_resize_layout(items.data(), 64, nullptr, &ws));
        std::vector<int32_t> grid(64 * 3), cu(65);
        for (auto& it : items) it.patch = 14, it.dst_h = 252;
        count(vp_batch_layout(items.data(), 64, grid.data(), cu.data(), &rows, &ws));
    }
    // a batch large enough for column pairs: 400 copies of a 480p pair -> 320x576
    {
        std::vector<int32_t> idx = {1, 0};
        std::vector<vp_item> items(400, vp_item{fake_frames(3), idx.data(), 2, 480, 854, 2, 320, 576, 16});
        int32_t nl = 0;
        std::vector<int32_t> launches(6 * 8);
        count(vp_batch_kernels(items.data(), 400, launches.data(), 8, &nl));
        int64_t rows = 0, ws = 0;
        count(vp_batch_layout(items.data(), 400, nullptr, nullptr, &rows, &ws));
        count(vp_batch_kernels(items.data(), 400, nullptr, 0, &nl));
    }
    // NULLs and degenerate batches
    count(vp_batch_layout(nullptr, 1, nullptr, nullptr, nullptr, nullptr));
    int32_t one = 0;
    vp_item single{fake_frames(0), &one, 1, 1, 1, 1, 32, 32, 16};
    count(vp_batch_layout(&single, 1, nullptr, nullptr, nullptr, nullptr));
    count(vp_batch_layout(&single, 0, nullptr, nullptr, nullptr, nullptr));
    int32_t nl = 0;
    count(vp_batch_kernels(&single, 1, nullptr, -1, &nl));
    count(vp_batch_kernels(&single, 1, nullptr, 0, nullptr));
    single.indices = nullptr;
    count(vp_batch_layout(&single, 1, nullptr, nullptr, nullptr, nullptr));
    for (int s = -1; s < 12; ++s) (void)vp_status_string(s);
    (void)vp_last_error_message();
}

void oracle_paths() {
    for (int r = 0; r < 20000; ++r) {
        int64_t h = 0, w = 0, c = 0;
        count(oracle_smart_resize(uni(-2, 20000), uni(-2, 20000), uni(0, 1) ? 32 : 28, uni(-1, 70000),
                                  uni(-5, int64_t(1) << 24), &h, &w));
        std::vector<int32_t> out(600);
        const int64_t total = uni(1, 5000);
        const int64_t n = uni(0, 600);
        if (n >= 1 && n <= total) count(oracle_sample_uniform(total, n, out.data()));
        count(oracle_sample_fps(total, double(uni(-1, 60)), double(uni(-1, 8)), uni(-1, 300), uni(-1, 600),
                                out.data(), int64_t(out.size()), &c));
    }
    for (int r = 0; r < 300; ++r) {
        const int64_t n_in = uni(1, 3000), n_out = uni(1, 1000);
        const int64_t taps = oracle_filter_max_taps(n_in, n_out);
        std::vector<int64_t> lo(n_out), cnt(n_out);
        std::vector<double> wt(size_t(taps) * n_out);
        count(oracle_filter_table(n_in, n_out, lo.data(), cnt.data(), wt.data(), taps));
        std::vector<double> one(taps);
        std::vector<int32_t> q(taps);
        int64_t l = 0, k = 0;
        count(oracle_filter(n_in, n_out, uni(0, n_out - 1), &l, &k, one.data(), taps));
        count(oracle_fixed_weights(n_in, n_out, uni(0, n_out - 1), &l, &k, q.data(), taps));
    }
    const double mean[3] = {0.48, 0.46, 0.41}, stdv[3] = {0.27, 0.26, 0.28};
    for (int r = 0; r < 60; ++r) {
        const int64_t patch = r % 3 == 2 ? 14 : 16, F = 2 * patch;
        const int64_t n_src = uni(1, 4), H = uni(1, 120), W = uni(1, 120);
        const int64_t h = F * uni(1, 3), w = F * uni(1, 3);
        std::vector<uint8_t> frames(size_t(n_src * H * W * 3));
        for (auto& v : frames) v = uint8_t(uni(0, 255));
        std::vector<int32_t> idx(size_t(uni(1, 5)));
        for (auto& v : idx) v = int32_t(uni(0, n_src - 1));
        const int64_t n_idx = int64_t(idx.size());
        std::vector<double> res(size_t(3 * h * w));
        count(oracle_resize_frame(frames.data(), H, W, h, w, res.data()));
        (void)oracle_resize_pixel(frames.data(), H, W, h, w, uni(0, h - 1), uni(0, w - 1), uni(0, 2));
        std::vector<uint8_t> u8(size_t(n_idx * h * w * 3));
        count(oracle_resize_u8(frames.data(), H, W, h, w, u8.data()));
        count(oracle_resize_u8_item(frames.data(), n_src, H, W, idx.data(), n_idx, h, w, patch, u8.data()));
        const int64_t rows = oracle_item_rows(n_idx, h, w, patch);
        std::vector<double> out(size_t(rows * 6 * patch * patch));
        count(oracle_preprocess_item(frames.data(), n_src, H, W, idx.data(), n_idx, h, w, patch, mean, stdv,
                                     out.data()));
        std::vector<double> row(size_t(6 * patch * patch));
        count(oracle_item_row(frames.data(), n_src, H, W, idx.data(), n_idx, h, w, patch, mean, stdv,
                              uni(0, rows - 1), row.data()));
        if (H >= h && W >= w) {   // patchify of frames at the target size: reuse the first h x w pixels' bytes
            std::vector<uint8_t> at(size_t(n_src * h * w * 3));
            for (size_t i = 0; i < at.size(); ++i) at[i] = frames[i % frames.size()];
            std::vector<double> pr(size_t(oracle_item_rows(n_idx, h, w, patch) * 6 * patch * patch));
            count(oracle_patchify_item(at.data(), n_src, h, w, idx.data(), n_idx, patch, mean, stdv, pr.data()));
        }
        const int64_t nn[2] = {n_idx, int64_t(uni(1, 9))}, hh[2] = {h, F}, ww[2] = {w, 2 * F};
        int64_t total = 0, slices = 0;
        for (int k = 0; k < 2; ++k) total += oracle_item_rows(nn[k], hh[k], ww[k], patch), slices += (nn[k] + 1) / 2;
        std::vector<int64_t> vit(size_t(total * 3)), llm(size_t(total / 4 * 3)), vcu(size_t(slices + 1)), g(6), cu(3);
        int64_t ns = 0;
        count(oracle_position_ids(2, nn, hh, ww, patch, vit.data(), llm.data(), vcu.data(), &ns));
        count(oracle_layout(2, nn, hh, ww, patch, g.data(), cu.data()));
    }
}

}  // namespace

int main() {
    library_host_paths();
    oracle_paths();
    std::printf("host checks: %lld calls, %lld returned OK\n", static_cast<long long>(calls),
                static_cast<long long>(ok_calls));
    return 0;
}
