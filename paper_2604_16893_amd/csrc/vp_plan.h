// vp_plan.h -- device-side plan of one vp_preprocess_batch call.
//
// The host planner (vp_api.cpp) validates the items, computes their filter
// tables, tile counts and row offsets, packs everything into one blob and
// copies it into the caller's workspace with a single async copy; the
// kernels (vp_kernels.hip) read it from there.  Layout of the blob, each
// section aligned to 256 bytes:
//   DevItem items[n_items]
//   int32   tile_prefix[n_items + 1]     work units of item b: [prefix[b], prefix[b+1])
//   int32   indices[sum of padded counts] frame index of every (frame pair, dt)
//   int32   tables[...]                  filter tables, 4-byte words
// A filter table of one axis (n_in -> n_out, K taps) at word offset `off`:
//   int32 start[n_out]; int32 count[n_out]; float weight[n_out][K]
// Items with the same (n_in, n_out) share one table.
#pragma once

#include <cstdint>

#include <hip/hip_runtime_api.h>

namespace vp {

constexpr int kPatch = 16;
constexpr int kWin = 32;              // merge window edge in pixels (patch * merge)
constexpr int kRow = 1536;            // 3 * 2 * 16 * 16
constexpr int kWinElems = 4 * kRow;   // one merge window of one frame pair
constexpr int kGenericThreads = 256;
constexpr int kGenericTCap = 8192;    // floats of the generic kernel's LDS column tile

// Kernel variants an item can be routed to.
enum Route : int32_t { kRouteGeneric = 0 };

struct DevItem {
    const uint8_t* frames;   // [n_src][H][W][3]
    int64_t frame_bytes;     // H * W * 3
    int64_t row_off;         // first output row of the item
    int32_t H, W, h, w;      // source and target size
    int32_t t, hm, wm;       // frame pairs, merge windows along y and x
    int32_t idx_off;         // first entry of the item in `indices` (2 * t entries)
    int32_t ty_off, tx_off;  // word offsets of the y and x filter tables
    int32_t ky, kx;          // tap stride of the y and x tables
    int32_t rh, cw;          // generic kernel: output rows / columns per LDS sub-tile
    int32_t route, pad0;
};
static_assert(sizeof(DevItem) == 88, "DevItem layout");

struct PlanView {
    const DevItem* items;
    const int32_t* tile_prefix;
    const int32_t* indices;
    const int32_t* tables;
    int32_t n_items;
    int32_t n_tiles;
};

struct Norm {
    float a[3];   // 1 / (255 * std_c)
    float b[3];   // -mean_c / std_c
};

// Kernel launchers (vp_kernels.hip).
int launch_generic(const PlanView& plan, void* out, int out_dtype, const Norm& norm,
                   hipStream_t stream);

}  // namespace vp
