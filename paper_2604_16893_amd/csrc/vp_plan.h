// vp_plan.h -- device-side plan of one vp_preprocess_batch call.
//
// The host planner (vp_api.cpp) validates the items, computes their filter
// tables, work units and row offsets, packs everything into one blob and
// copies it into the caller's workspace with a single async copy; the
// kernels (vp_kernels.hip) read it from there.  Layout of the blob, each
// section aligned to 256 bytes:
//   DevItem    items[n_items]
//   int32      tile_prefix[n_items + 1]   general-kernel work of item b: [prefix[b], prefix[b+1])
//   int32      indices[sum of padded counts]  source frame of every (frame pair, dt)
//   int32      tables[...]                filter tables, 4-byte words
//   StreamUnit units[...]                 streaming-kernel work units
//   uint32     wgs[...]                   streaming-kernel workgroups, grouped per launch:
//                                         unit index | column band << 20, or kNoWork
//
// Tables (word offsets into `tables`; items with the same axis share them):
//   window table of an axis n_in -> n_out, K taps:
//       int32 start[n_out]; int32 count[n_out]; float weight[n_out][K]
//   slot table of a y axis n_in -> n_out (streaming kernel), M slots:
//       [n_in + 6] rows of 8 words: float weight[slot]   (slots >= M zero)
//         -- output row i is accumulated in slot i mod M from the first row of
//            its window to its close row; weight[s] is 2^24 times the weight
//            of source row y in the output row that has slot s at y, or zero
//            (the kernel reads source bytes as f16 denormals, b * 2^-24)
//       int32 close_row[n_out + 1]   (the last entry is INT32_MAX)
//         -- the row after which output row i is complete: the last row of its
//            window, or the close row of output row i - 1 if that is later;
//            never decreasing, and several output rows may close on one row
//            (an upscaled axis, the bottom border)
//   fixed-point window table (uint8 writer): as the window table, with int32
//       weights in units of 2^-22
//   column table of an x axis (streaming kernels), KX taps, for output bands
//   of `band` columns whose source pixels fit a row of `row_px` pixels (the
//   y-first kernel's LDS row; the x-first kernel passes W + KX, a bound no
//   window reaches):
//       int32 start[n_out]; float weight[n_out][KX]
//     -- start is relative to the first source pixel of the output's band
//        (the window start of the band's first column) and start + KX never
//        passes row_px; weights are shifted and zero-padded to match.
#pragma once

#include <cstdint>

#include <hip/hip_runtime_api.h>

namespace vp {

constexpr int kPatch = 16;
constexpr int kWin = 32;              // merge window edge in pixels (patch * merge)
constexpr int kRow = 1536;            // 3 * 2 * 16 * 16
constexpr int kWinElems = 4 * kRow;   // one merge window of one frame pair
constexpr int kGenericThreads = 256;
constexpr int kGenericTCap = 8192;    // floats of the general kernel's LDS column tile
constexpr int kSlotWords = 8;         // words per source row of a slot table
constexpr int kSlotMax = 6;           // most output rows open at once (accumulator slots)
constexpr int kStreamLdsBudget = 64 * 1024;   // LDS of one streaming workgroup (one wave)

// LDS of one streaming workgroup.  Patch 16 (one wave): its source row (64 *
// px float4 pixels) and the stage of four output rows (3 channels x 4 rows x
// 64 columns).  Patch 14 (four waves: a pair's two frames over two bands):
// four source rows and the stage of up to eight whole output rows of 1176
// values.
constexpr int stream_wave_bytes(int px, int kx, int elem_bytes, int patch = 16) {
    return (void)kx, patch == 16 ? 64 * px * 16 + 3 * 4 * 64 * elem_bytes
                                 : 4 * 64 * px * 16 + 8 * 6 * patch * patch * elem_bytes;
}

// LDS of one x-first streaming workgroup (one wave of cpl columns per lane):
// the stage of four output rows (its lanes load their source windows from
// memory).
constexpr int xfirst_wave_bytes(int elem_bytes, int cpl) { return 3 * 4 * 64 * cpl * elem_bytes; }

// uint8 streaming writer: pixels per lane (a band's source span is at most
// 64 * kRsPx pixels), and the LDS of one workgroup (one wave): its source
// row as three byte planes and the stage of four output rows of up to 64
// RGB pixels.
constexpr int kRsPx = 4;
constexpr int resize_stream_bytes() { return 3 * 64 * kRsPx + 4 * 64 * 3; }
// The writer's MFMA form (launch shape kx = kRsMfmaWindow): column table words
// per band of 64 columns (four window starts, then 4 blocks x 3 digits x 64
// lanes x 4 dwords), and its LDS: the horizontal pass's bytes of 16 source
// rows for 64 columns and 3 channels, and the stage.
constexpr int kRsMfmaWindow = 64;
constexpr int kRsMfmaBandWords = 4 + 4 * 3 * 64 * 4;
constexpr int resize_mfma_bytes() { return 3 * 64 * 16 + 4 * 64 * 3; }

// Kernel an item is routed to.
enum Route : int32_t { kRouteGeneric = 0, kRouteStream = 1, kRoutePatch = 2, kRouteResize = 3 };

// uint8 cache writer (resize_u8_kernel): one workgroup of kRsThreads per tile
// of up to 32 output rows x 64 output columns of one frame; the host picks
// smaller tiles where these LDS budgets require it.
constexpr int kRsThreads = 256;
constexpr int kRsChunk = 4;          // source rows staged per horizontal step (kRsThreads / 64)
constexpr int kRsSrcRow = 2048;      // LDS bytes per staged source row
constexpr int kRsMid = 32768;        // LDS bytes of the horizontal pass's uint8 rows
constexpr int kRsQ = 2048;           // int32 weights of one axis per tile
constexpr int kRsRowsMax = 32;
constexpr int kRsColsMax = 64;

struct DevItem {
    const uint8_t* frames;   // [n_src][H][W][3]
    int64_t frame_bytes;     // H * W * 3
    int64_t row_off;         // first output row of the item
    int32_t H, W, h, w;      // source and target size
    int32_t t, hm, wm;       // frame pairs, merge windows along y and x
    int32_t idx_off;         // first entry of the item in `indices` (2 * t entries)
    int32_t ty_off, tx_off;  // window tables of the y and x axes
    int32_t ky, kx;          // tap stride of those tables
    int32_t rh, cw;          // general kernel: output rows / columns per LDS sub-tile
    int32_t route;
    int32_t band;            // streaming kernel: output columns per wave (16, 32, 48 or 64)
    int32_t sy_off, sx_off;  // streaming kernel: slot and column tables
    int32_t row_px;          // streaming kernels: the column table's row bound (64 * px; x-first W + kx)
    int32_t patch;           // patch edge P (16 or 14): rows of 6 P^2 values, windows of 2P
};
static_assert(sizeof(DevItem) == 104, "DevItem layout");

// One streaming work unit: output rows [i0, i1) of padded frame position p
// of an item; one workgroup per column band of the unit.  Bit kUnitBoth of
// p_flags: the pair's two frames are the same source frame (an image, or an
// odd count padded with its last index), so the unit writes both temporal
// halves of the rows.  p < 2^30 always: every frame pair owns at least four
// of the batch's at most 2^31 - 1 rows.
struct StreamUnit {
    int32_t item;
    int32_t p_flags;   // p | kUnitBoth if the pair's frames are one
    int32_t i0, i1;    // output rows [i0, i1) of the frame
};
static_assert(sizeof(StreamUnit) == 16, "StreamUnit layout");
constexpr int32_t kUnitBoth = 1 << 30;

struct PlanView {
    const DevItem* items;
    const int32_t* tile_prefix;
    const int32_t* indices;
    const int32_t* tables;
    const StreamUnit* units;
    const uint32_t* wgs;
    int32_t n_items;
    int32_t n_tiles;
};

struct Norm {
    float a[3];   // 1 / (255 * std_c)
    float b[3];   // -mean_c / std_c
    float z[3];   // -255 * mean_c: v = a_c * (R + z_c), the same value in pixel units
};

// Streaming workgroup entries: unit index in the low 20 bits, column band
// (at most kWgBandMax) above; kNoWork marks an empty workgroup.
constexpr uint32_t kWgUnitMask = (1u << 20) - 1;
constexpr int kWgBandShift = 20;
constexpr int kWgBandMax = (1 << (32 - kWgBandShift)) - 2;   // keeps entries below kNoWork
constexpr uint32_t kNoWork = 0xffffffffu;

// One launch of the streaming kernel: workgroups wgs[first, first + count),
// all with the same template shape.  px < 0 marks the x-first kernel:
// xfirst_px(0) one column per lane, xfirst_px(2) column pairs whose second
// window starts at most 2 pixels after the first's.
constexpr int32_t xfirst_px(int db) { return -1 - db; }
constexpr int xfirst_db(int32_t px) { return -1 - px; }
struct StreamLaunch {
    int32_t first, count;
    int32_t m, kx, px;       // accumulator slots, column taps, pixels per lane (or xfirst_px)
    int32_t patch;           // patch edge of the batch (16 or 14)
    int64_t cost;            // host only: estimated work (source pixels read)
};

// Fixed device memory for the plan of vp_preprocess_batch_noalloc, one array
// per device (vp_kernels.hip), and its size.  noalloc_plan_memory() gives the
// current device's copy of the array, looked up once per device; it returns
// a hipError_t value.
constexpr int64_t kNoAllocPlanBytes = int64_t(16) << 20;
int noalloc_plan_memory(void** ptr);

// Kernel launchers (vp_kernels.hip).  Return a hipError_t value.
int launch_generic(const PlanView& plan, void* out, int out_dtype, const Norm& norm,
                   hipStream_t stream);
int launch_stream(const PlanView& plan, const StreamLaunch& launch, void* out, int out_dtype,
                  const Norm& norm, hipStream_t stream);
// Normalise + patchify of frames already at the target size: one workgroup
// per merge-window row of a frame pair (tile_prefix counts them per item).
int launch_patchify(const PlanView& plan, void* out, int out_dtype, const Norm& norm, int patch,
                    hipStream_t stream);
// uint8 cache writer over tile_prefix (items with route kRouteResize: rh x cw
// output tiles, tables holding fixed-point weights); out is the byte buffer.
int launch_resize(const PlanView& plan, void* out, hipStream_t stream);
int launch_resize_stream(const PlanView& plan, const StreamLaunch& launch, void* out, hipStream_t stream);
// Shapes (slots, column taps, pixels per lane) the uint8 streaming writer is built for.
bool resize_stream_supported(int m, int kx, int px);
// Position tables: one thread per output row; tile_prefix holds the items'
// row offsets (cu).  vit / llm may be null.
int launch_positions(const PlanView& plan, int32_t* vit, int32_t* llm, int64_t rows,
                     hipStream_t stream);
// Whether a (m, kx, px) shape has a compiled streaming kernel.
bool stream_shape_supported(int m, int kx, int px);
// Whether an (m, kx, pair offset) shape has a compiled x-first kernel.
bool xfirst_shape_supported(int m, int kx, int db);

}  // namespace vp
