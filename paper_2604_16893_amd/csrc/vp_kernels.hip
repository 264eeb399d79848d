// vp_kernels.hip -- gfx950 kernels of the preprocessing path.
//
// Three kernels compute the same result (the resampled, normalised,
// merge-window rows of Section 3.1.1 of arXiv 2604.16893, laid out per the
// grid the host reports); the host routes each item to one of them.
//
// Streaming kernel, y first (the fast path for vertical downscales: items
// with at most 8 output rows open on a source row and x windows of at most
// 32 taps that the x-first kernel below does not take).  One workgroup streams
// one source frame -- or a band of its output rows -- top to bottom, one
// wave per band of up to 64 output columns; the waves never wait for each
// other:
//   * y pass first, in registers: each lane owns 2 or 3 RGB pixels of the
//     band's source span, loads them with one buffer load per row
//     (prefetched four rows ahead), unpacks the bytes two at a time into
//     f16 halves (one v_perm per pair, which also absorbs the lane's byte
//     misalignment) and adds them with wave-uniform scalar weights into M
//     accumulator slots through mixed-precision FMAs (f16 byte times f32
//     weight, exact); output row i lives in slot i mod M while it is open.
//     The source is read once.
//   * when an output row is complete its slot goes to the wave's LDS row
//     (one float4 per pixel) and the wave's x pass follows: one lane per
//     output column, one ds_read_b128 and three FMAs per tap, then the
//     normalisation FMA and the bf16/f32 conversion into the wave's stage.
//   * every four output rows the stage holds the band's part of one
//     64-value run (four patch rows of 16) of every (patch, channel) block;
//     those leave as 16-byte stores, eight lanes per 128-byte run.
//   * patch 14 is the exception to independent waves: a workgroup is four
//     waves (two neighbouring bands x a pair's two frames) that meet at a
//     barrier once per patch row, to write whole output rows.
//
// Streaming kernel, x first (patch 16, vertical scales up to 1.6, x windows
// of 4 to 12 taps): the same units, slots and store, but each lane x-filters
// its own window of every source row, loaded straight from the frame, before
// the y pass into the slots; LDS holds only the stage.
//
// General kernel (any scale factor): one workgroup per merge window of one
// frame pair; y pass from global memory into an LDS column tile, x pass,
// staging of the four rows in output order, 16-byte stores.  When the
// horizontal window of 32 output columns does not fit the tile, the host
// splits the window into rh x cw sub-tiles.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <type_traits>

#include "vp_plan.h"

// The streaming kernels' many template shapes are compiled in VP_PARTS
// translation units: this file is compiled once per part with
// -DVP_PART=k.  Part 0 holds the launchers and the kernels of a single
// shape; every part instantiates its share of the streaming shapes and
// exports a dispatcher for them (launch_stream_part<k>,
// launch_resize_stream_part<k>).  Built as one unit (no -D), part 0 is all.
#ifndef VP_PART
#define VP_PART 0
#endif
#ifndef VP_PARTS
#define VP_PARTS 1
#endif
static_assert(VP_PARTS >= 1 && VP_PARTS <= 8 && VP_PART >= 0 && VP_PART < VP_PARTS, "kernel parts");
#define VP_CAT2(a, b) a##b
#define VP_CAT(a, b) VP_CAT2(a, b)

namespace vp {
namespace {

// The plan is read-only while the kernels run: reading it through the
// constant address space lets wave-uniform reads become scalar loads, which
// neither occupy vector registers nor share the vector-memory counter with
// the frame prefetch.
template <class T>
using cptr = const __attribute__((address_space(4))) T*;

template <class T>
__device__ __forceinline__ cptr<T> as_const(const T* p) {
    return (cptr<T>)(p);
}

#if VP_PART == 0   // the kernels of a single shape: part 0 only

__device__ __forceinline__ uint32_t bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ int find_item(const int32_t* prefix, int n_items, int tile) {
    int lo = 0, hi = n_items;  // largest lo with prefix[lo] <= tile
    while (hi - lo > 1) {
        int mid = (lo + hi) >> 1;
        if (prefix[mid] <= tile) lo = mid; else hi = mid;
    }
    return lo;
}

// ===========================================================================
// General kernel
// ===========================================================================

template <int OUT_BF16>
__global__ __launch_bounds__(kGenericThreads) void generic_tile_kernel(PlanView plan, void* out,
                                                                       Norm norm) {
    __shared__ float tcol[kGenericTCap];   // y-resampled columns of one sub-tile, [r][x][c]
    __shared__ float stage[kWinElems];     // the unit's four output rows, output order (P <= 16)

    const int tile = blockIdx.x;
    const int b = find_item(plan.tile_prefix, plan.n_items, tile);
    const DevItem it = plan.items[b];
    const int local = tile - plan.tile_prefix[b];
    const int bw = local % it.wm;
    const int q = local / it.wm;
    const int bh = q % it.hm;
    const int tt = q / it.hm;

    const int32_t* ys = plan.tables + it.ty_off;
    const int32_t* yn = ys + it.h;
    const float* wy = reinterpret_cast<const float*>(yn + it.h);
    const int32_t* xs = plan.tables + it.tx_off;
    const int32_t* xn = xs + it.w;
    const float* wx = reinterpret_cast<const float*>(xn + it.w);
    const int64_t row_stride = int64_t(it.W) * 3;
    const int tid = threadIdx.x;
    const int P = it.patch, win = 2 * it.patch, row_len = 6 * it.patch * it.patch;

    // an image, or an odd count padded with its last index: both temporal
    // halves come from one frame, computed once and staged twice
    const bool same = plan.indices[it.idx_off + 2 * tt] == plan.indices[it.idx_off + 2 * tt + 1];
    for (int dt = 0; dt < (same ? 1 : 2); ++dt) {
        const int f = plan.indices[it.idx_off + 2 * tt + dt];
        const uint8_t* frame = it.frames + int64_t(f) * it.frame_bytes;
        for (int r0 = 0; r0 < win; r0 += it.rh) {
            for (int c0 = 0; c0 < win; c0 += it.cw) {
                const int i0 = win * bh + r0;
                const int j0 = win * bw + c0;
                const int x0 = xs[j0];
                const int xw = xs[j0 + it.cw - 1] + xn[j0 + it.cw - 1] - x0;
                const int span = xw * 3;
                // pass along y: tcol[r][x][c] = sum_k wy[i][k] * F[ys[i] + k][x0 + x][c]
                for (int e = tid; e < it.rh * span; e += kGenericThreads) {
                    const int r = e / span;
                    const int col = e - r * span;
                    const int i = i0 + r;
                    const int n = yn[i];
                    const float* wr = wy + int64_t(i) * it.ky;
                    const uint8_t* p = frame + int64_t(ys[i]) * row_stride + int64_t(x0) * 3 + col;
                    float acc = 0.f;
                    for (int k = 0; k < n; ++k) acc = fmaf(wr[k], float(p[k * row_stride]), acc);
                    tcol[e] = acc;
                }
                __syncthreads();
                // pass along x, normalise, stage in output order
                for (int e = tid; e < it.rh * it.cw * 3; e += kGenericThreads) {
                    const int c = e % 3;
                    const int qq = e / 3;
                    const int cc = qq % it.cw;
                    const int r = qq / it.cw;
                    const int j = j0 + cc;
                    const int n = xn[j];
                    const float* wr = wx + int64_t(j) * it.kx;
                    const float* src = tcol + r * span + (xs[j] - x0) * 3 + c;
                    float acc = 0.f;
                    for (int k = 0; k < n; ++k) acc = fmaf(wr[k], src[3 * k], acc);
                    // the normalisation every kernel uses, a_c * (R + z_c): at
                    // identity size R is the pixel itself and the paths agree
                    // bit for bit
                    const float v = (acc + norm.z[c]) * norm.a[c];
                    const int il = r0 + r, jl = c0 + cc;
                    const int sub = (il / P) * 2 + (jl / P);
                    float* st = stage + sub * row_len + ((c * 2 + dt) * P + il % P) * P + jl % P;
                    st[0] = v;
                    if (same) st[P * P] = v;   // the second temporal half
                }
                __syncthreads();
            }
        }
    }

    const int64_t row0 = it.row_off + ((int64_t(tt) * it.hm + bh) * it.wm + bw) * 4;
    // the four rows are contiguous: 4 * 6 P^2 values, a multiple of 8, and
    // they start on a 16-byte boundary (6 P^2 * 2 bytes is one for P = 14, 16)
    const int win_elems = 4 * row_len;
    if (OUT_BF16) {
        uint4* dst = reinterpret_cast<uint4*>(static_cast<uint16_t*>(out) + row0 * row_len);
        for (int e = tid; e < win_elems / 8; e += kGenericThreads) {
            const float* s = stage + e * 8;
            uint4 v;
            v.x = bf16_rne(s[0]) | (bf16_rne(s[1]) << 16);
            v.y = bf16_rne(s[2]) | (bf16_rne(s[3]) << 16);
            v.z = bf16_rne(s[4]) | (bf16_rne(s[5]) << 16);
            v.w = bf16_rne(s[6]) | (bf16_rne(s[7]) << 16);
            dst[e] = v;
        }
    } else {
        float4* dst = reinterpret_cast<float4*>(static_cast<float*>(out) + row0 * row_len);
        for (int e = tid; e < win_elems / 4; e += kGenericThreads)
            dst[e] = reinterpret_cast<const float4*>(stage)[e];
    }
}

// ===========================================================================
// Position tables
// ===========================================================================

// One thread per output row: the row's item (binary search over the row
// offsets), then its frame pair, patch row and patch column from the
// merge-window order; the first row of each window also writes the window's
// token coordinates.
__global__ __launch_bounds__(256) void positions_kernel(PlanView plan, int32_t* vit, int32_t* llm,
                                                         int64_t rows) {
    for (int64_t row = int64_t(blockIdx.x) * 256 + threadIdx.x; row < rows;
         row += int64_t(gridDim.x) * 256) {
        const int b = find_item(plan.tile_prefix, plan.n_items, static_cast<int>(row));
        const cptr<DevItem> it = as_const(plan.items) + b;
        const int local = static_cast<int>(row) - plan.tile_prefix[b];
        const int sub = local & 3, win = local >> 2;
        const int wm = it->wm, hm = it->hm;
        const int bw = win % wm;
        const int bh = (win / wm) % hm;
        const int tt = win / (wm * hm);
        if (vit != nullptr) {
            int32_t* v = vit + row * 3;
            v[0] = tt;
            v[1] = 2 * bh + (sub >> 1);
            v[2] = 2 * bw + (sub & 1);
        }
        if (llm != nullptr && sub == 0) {
            int32_t* l = llm + (row >> 2) * 3;
            l[0] = tt;
            l[1] = bh;
            l[2] = bw;
        }
    }
}

// ===========================================================================
// uint8 cache writer (fixed-point resampling)
// ===========================================================================

// round half up of a sum in units of 2^-22, clamped to a byte
__device__ __forceinline__ uint32_t fixed_to_byte(int32_t acc) {
    const int32_t v = acc + (1 << 21);
    return v < 0 ? 0u : min(static_cast<uint32_t>(v) >> 22, 255u);
}

// One workgroup per tile of up to 32 output rows x 64 output columns of one
// sampled frame.  The horizontal pass runs first (the fixed-point
// convention): the source rows the tile's vertical windows need are staged
// four at a time in LDS as bytes, and each thread (row, column) forms the
// three channels of one horizontally resampled pixel, rounded and clamped to
// a byte, into the tile's LDS rows.  The vertical pass then forms each output
// byte from those and stores them four at a time.  Sums are exact in int32:
// |q| < 2^23, bytes < 2^8, and the weights of a window sum to about 2^22.
__global__ __launch_bounds__(kRsThreads) void resize_u8_kernel(PlanView plan, uint8_t* out) {
    __shared__ __align__(16) uint32_t src32[kRsChunk][kRsSrcRow / 4];
    __shared__ __align__(16) uint8_t mid[kRsMid];
    __shared__ int32_t qx[kRsQ], qy[kRsQ];
    __shared__ int32_t col_off[kRsColsMax], col_n[kRsColsMax], row_off[kRsRowsMax], row_n[kRsRowsMax];

    const int tile = blockIdx.x;
    const int b = find_item(plan.tile_prefix, plan.n_items, tile);
    const DevItem it = plan.items[b];
    const int local = tile - plan.tile_prefix[b];
    const int tx = local % it.wm;
    const int q2 = local / it.wm;
    const int ty = q2 % it.hm;
    const int k = q2 / it.hm;
    const int RB = it.rh, CB = it.cw;
    const int i0 = ty * RB, j0 = tx * CB;
    const int nr = min(RB, it.h - i0), nc = min(CB, it.w - j0);
    const int32_t* ys = plan.tables + it.ty_off;
    const int32_t* yn = ys + it.h;
    const int32_t* yq = yn + it.h;
    const int32_t* xs = plan.tables + it.tx_off;
    const int32_t* xn = xs + it.w;
    const int32_t* xq = xn + it.w;
    // window ends never decrease, so the tile reads [ylo, yhi) x [xlo, xhi)
    const int ylo = ys[i0], yhi = ys[i0 + nr - 1] + yn[i0 + nr - 1];
    const int xlo = xs[j0], xhi = xs[j0 + nc - 1] + xn[j0 + nc - 1];
    const int tid = threadIdx.x;
    for (int e = tid; e < nc * it.kx; e += kRsThreads)
        qx[e] = xq[int64_t(j0 + e / it.kx) * it.kx + e % it.kx];
    for (int e = tid; e < nr * it.ky; e += kRsThreads)
        qy[e] = yq[int64_t(i0 + e / it.ky) * it.ky + e % it.ky];
    if (tid < nc) {
        col_off[tid] = 3 * (xs[j0 + tid] - xlo);
        col_n[tid] = xn[j0 + tid];
    }
    if (tid < nr) {
        row_off[tid] = ys[i0 + tid] - ylo;
        row_n[tid] = yn[i0 + tid];
    }

    // the frame through a buffer resource (range: the frame in whole dwords,
    // so a dword that runs past its end reads zeros)
    const int f = plan.indices[it.idx_off + k];
    const uintptr_t fa = reinterpret_cast<uintptr_t>(it.frames + int64_t(f) * it.frame_bytes);
    const uint32_t lead = static_cast<uint32_t>(fa & 3u);
    const uint32_t range = static_cast<uint32_t>((it.frame_bytes + lead + 3) & ~int64_t(3));
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(fa - lead), (short)0, static_cast<int>(range), 0x00020000);
    const uint32_t row_bytes = static_cast<uint32_t>(it.W) * 3u;
    const int span = (xhi - xlo) * 3;
    __syncthreads();

    const int r = tid >> 6, jj = tid & 63;
    for (int y0 = ylo; y0 < yhi; y0 += kRsChunk) {
        for (int e = tid; e < kRsChunk * (kRsSrcRow / 4); e += kRsThreads) {
            const int rr = e / (kRsSrcRow / 4), d = e % (kRsSrcRow / 4);
            const int y = y0 + rr;
            const uint32_t o = lead + static_cast<uint32_t>(y) * row_bytes + 3u * static_cast<uint32_t>(xlo);
            const int ndw = (span + static_cast<int>(o & 3u) + 3) >> 2;
            if (y < yhi && d < ndw)
                src32[rr][d] = static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b32(rsrc, (o & ~3u) + 4u * d, 0, 0));
        }
        __syncthreads();
        const int y = y0 + r;
        if (y < yhi && jj < nc) {
            const uint32_t o = lead + static_cast<uint32_t>(y) * row_bytes + 3u * static_cast<uint32_t>(xlo);
            const uint8_t* px = reinterpret_cast<const uint8_t*>(src32[r]) + (o & 3u) + col_off[jj];
            const int32_t* q = qx + jj * it.kx;
            const int n = col_n[jj];
            int32_t a0 = 0, a1 = 0, a2 = 0;
            for (int t = 0; t < n; ++t) {
                const int32_t w = q[t];
                a0 += __mul24(w, static_cast<int32_t>(px[3 * t]));
                a1 += __mul24(w, static_cast<int32_t>(px[3 * t + 1]));
                a2 += __mul24(w, static_cast<int32_t>(px[3 * t + 2]));
            }
            uint8_t* m = mid + ((y - ylo) * CB + jj) * 3;
            m[0] = static_cast<uint8_t>(fixed_to_byte(a0));
            m[1] = static_cast<uint8_t>(fixed_to_byte(a1));
            m[2] = static_cast<uint8_t>(fixed_to_byte(a2));
        }
        __syncthreads();
    }

    // vertical pass: four output bytes per step (the tile's row segments are
    // nc * 3 bytes, a multiple of 24, and start on 4-byte boundaries)
    const int words = nc * 3 / 4;
    uint8_t* ob = out + it.row_off + (int64_t(k) * it.h + i0) * it.w * 3 + int64_t(j0) * 3;
    for (int e = tid; e < nr * words; e += kRsThreads) {
        const int ii = e / words, d = e % words;
        const int32_t* q = qy + ii * it.ky;
        const int n = row_n[ii];
        const uint8_t* m0 = mid + row_off[ii] * CB * 3;
        uint32_t word = 0;
#pragma unroll
        for (int bb = 0; bb < 4; ++bb) {
            const int byte = 4 * d + bb;   // pixel byte / 3, channel byte % 3
            const int col = byte / 3, c = byte - 3 * col;
            const uint8_t* m = m0 + col * 3 + c;
            int32_t acc = 0;
            for (int t = 0; t < n; ++t) acc += __mul24(q[t], static_cast<int32_t>(m[t * CB * 3]));
            word |= fixed_to_byte(acc) << (8 * bb);
        }
        *reinterpret_cast<uint32_t*>(ob + int64_t(ii) * it.w * 3 + 4 * d) = word;
    }
}

// ===========================================================================
// Normalise + patchify kernel (frames already at the target size)
// ===========================================================================

// One workgroup of four waves per merge-window row (32 pixel rows) of one
// frame pair.  Wave (dt, mh) takes pixel rows 16*mh .. 16*mh + 15 of frame
// dt of the pair; lane (y, g) owns 8 pixels (24 bytes) of row y, at 8*g in
// each merge window.  Window by window along the row, with the next
// window's bytes already in flight, a lane normalises its 24 values and
// stores three 16-byte pieces of 8 values, one per channel: for a fixed
// channel the wave's stores fill two whole 512-byte blocks of output (one
// per patch of its patch row), so every store is fully coalesced.
template <int OUT_BF16>
__global__ __launch_bounds__(256) void patchify_kernel(PlanView plan, void* out, Norm norm) {
    using elem_t = typename std::conditional<OUT_BF16 != 0, uint16_t, float>::type;
    const int tile = blockIdx.x;
    const int b = find_item(plan.tile_prefix, plan.n_items, tile);
    const cptr<DevItem> it = as_const(plan.items) + b;
    const int local = tile - plan.tile_prefix[b];
    const int hm = it->hm, wm = it->wm, w = it->w;
    const int bh = local % hm;
    const int tt = local / hm;
    const int wv = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    const int lane = threadIdx.x & 63;
    const int dt = wv >> 1, mh = wv & 1;
    const int y = lane >> 2, g = lane & 3;
    const int f = as_const(plan.indices)[it->idx_off + 2 * tt + dt];
    // 4-byte aligned: the frames pointer is (checked on the host), and every
    // offset below is a multiple of 24 bytes
    const uint32_t* src = reinterpret_cast<const uint32_t*>(
        it->frames + int64_t(f) * it->frame_bytes + (int64_t(32 * bh + 16 * mh + y) * w + 8 * g) * 3);
    const int64_t row0 = it->row_off + (int64_t(tt) * hm + bh) * wm * 4 + mh * 2 + (g >> 1);
    elem_t* dst = static_cast<elem_t*>(out) + row0 * kRow + (dt * 16 + y) * 16 + (g & 1) * 8;
    const float a[3] = {norm.a[0], norm.a[1], norm.a[2]};
    const float z[3] = {norm.z[0], norm.z[1], norm.z[2]};

    uint32_t cur[6], nxt[6];
#pragma unroll
    for (int k = 0; k < 6; ++k) cur[k] = src[k];
    for (int bw = 0; bw < wm; ++bw) {
        if (bw + 1 < wm) {
#pragma unroll
            for (int k = 0; k < 6; ++k) nxt[k] = src[24 * (bw + 1) + k];   // 96 bytes per window
        }
        elem_t* d = dst + int64_t(bw) * 4 * kRow;
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            float v[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int byte = 3 * q + c;
                const float x = float((cur[byte >> 2] >> (8 * (byte & 3))) & 255u);
                v[q] = (x + z[c]) * a[c];   // (F/255 - mean)/std as a * (F - 255 mean)
            }
            using u4v = unsigned __attribute__((ext_vector_type(4)));
            if constexpr (OUT_BF16 != 0) {
                u4v pk;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    using f2 = float __attribute__((ext_vector_type(2)));
                    using b2 = __bf16 __attribute__((ext_vector_type(2)));
                    const f2 pair = {v[2 * e], v[2 * e + 1]};
                    pk[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(pair, b2));   // RNE
                }
                __builtin_nontemporal_store(pk, reinterpret_cast<u4v*>(d + c * 512));
            } else {
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const u4v pk = {__float_as_uint(v[4 * h]), __float_as_uint(v[4 * h + 1]),
                                    __float_as_uint(v[4 * h + 2]), __float_as_uint(v[4 * h + 3])};
                    __builtin_nontemporal_store(pk, reinterpret_cast<u4v*>(d + c * 512 + 4 * h));
                }
            }
        }
#pragma unroll
        for (int k = 0; k < 6; ++k) cur[k] = nxt[k];
    }
}

// The same for patches of 14 (Qwen2/2.5-VL geometry: windows of 28, rows of
// 1176).  Wave (dt, mh) as above; lane l < 56 owns one patch row, P = 14
// pixels (42 bytes): row y = l % 14 of patch mw = (l / 14) & 1 in window
// bw = 2 * step + (l / 28).  A patch row can start off a dword boundary, so
// the lane loads the 12 dwords that cover it from any offset (42 bytes plus
// up to 3) through a buffer resource (range-checked at the frame's end) and
// aligns them with v_alignbyte.  Per channel its 14 values are one contiguous run of
// the output row (4-byte aligned for bf16, 8-byte for float32).
template <int OUT_BF16>
__global__ __launch_bounds__(256) void patchify14_kernel(PlanView plan, void* out, Norm norm) {
    using elem_t = typename std::conditional<OUT_BF16 != 0, uint16_t, float>::type;
    constexpr int P = 14;
    constexpr int kRowLen = 6 * P * P;   // 1176
    const int tile = blockIdx.x;
    const int b = find_item(plan.tile_prefix, plan.n_items, tile);
    const cptr<DevItem> it = as_const(plan.items) + b;
    const int local = tile - plan.tile_prefix[b];
    const int hm = it->hm, wm = it->wm, w = it->w;
    const int bh = local % hm;
    const int tt = local / hm;
    const int wv = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    const int lane = threadIdx.x & 63;
    const int dt = wv >> 1, mh = wv & 1;
    if (lane >= 4 * P) return;   // no barrier follows
    const int y = lane % P, mw = (lane / P) & 1, par = lane / (2 * P);
    const int f = as_const(plan.indices)[it->idx_off + 2 * tt + dt];
    const uintptr_t fa = reinterpret_cast<uintptr_t>(it->frames + int64_t(f) * it->frame_bytes);
    const uint32_t lead = static_cast<uint32_t>(fa & 3u);
    const uint32_t range = static_cast<uint32_t>((it->frame_bytes + lead + 3) & ~int64_t(3));
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<void*>(fa - lead), (short)0, static_cast<int>(range), 0x00020000);
    const uint32_t row_byte0 = lead + static_cast<uint32_t>((2 * P * bh + P * mh + y) * w) * 3u;
    const float a[3] = {norm.a[0], norm.a[1], norm.a[2]};
    const float z[3] = {norm.z[0], norm.z[1], norm.z[2]};
    const int64_t row_base = it->row_off + (int64_t(tt) * hm + bh) * wm * 4 + mh * 2 + mw;

    for (int bw = par; bw < wm; bw += 2) {
        const uint32_t o = row_byte0 + static_cast<uint32_t>(2 * P * bw + P * mw) * 3u;
        const uint32_t sh = o & 3u;
        uint32_t d[12];
#pragma unroll
        for (int k = 0; k < 12; ++k)
            d[k] = static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b32(rsrc, (o & ~3u) + 4u * k, 0, 0));
        uint32_t bytes[11];   // the patch row's 42 bytes from byte 0
#pragma unroll
        for (int k = 0; k < 11; ++k) bytes[k] = __builtin_amdgcn_alignbyte(d[k + 1], d[k], sh);
        elem_t* dst = static_cast<elem_t*>(out) + (row_base + int64_t(bw) * 4) * kRowLen + (dt * P + y) * P;
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            float v[P];
#pragma unroll
            for (int q = 0; q < P; ++q) {
                const int byte = 3 * q + c;
                v[q] = (float((bytes[byte >> 2] >> (8 * (byte & 3))) & 255u) + z[c]) * a[c];
            }
            elem_t* dc = dst + c * 2 * P * P;
            if constexpr (OUT_BF16 != 0) {
                using f2 = float __attribute__((ext_vector_type(2)));
                using b2 = __bf16 __attribute__((ext_vector_type(2)));
#pragma unroll
                for (int e = 0; e < P / 2; ++e) {
                    const f2 pr = {v[2 * e], v[2 * e + 1]};
                    reinterpret_cast<uint32_t*>(dc)[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(pr, b2));
                }
            } else {
#pragma unroll
                for (int e = 0; e < P / 2; ++e)
                    reinterpret_cast<float2*>(dc)[e] = make_float2(v[2 * e], v[2 * e + 1]);
            }
        }
    }
}

#endif  // VP_PART == 0

// ===========================================================================
// Streaming kernel
// ===========================================================================

constexpr int kPrefetch = 4;           // source rows in flight per lane

using f3 = float __attribute__((ext_vector_type(3)));
using h2 = _Float16 __attribute__((ext_vector_type(2)));

// range - o, or 0 where o > range, for wave-uniform operands, on the
// scalar unit (written out: the compiler forms this saturating difference
// with a vector instruction and a v_readfirstlane, three vector issues per
// source row of the streaming kernels).
__device__ __forceinline__ uint32_t uniform_sat_sub(uint32_t range, uint32_t o) {
    uint32_t r;
    asm("s_sub_u32 %0, %1, %2\n\ts_cselect_b32 %0, 0, %0" : "=s"(r) : "s"(range), "s"(o) : "scc");
    return r;
}

// Orders this wave's LDS accesses before and after it.  LDS operations of
// one wave execute in issue order, so within a wave keeping the compiler from
// moving them across this point is all the synchronisation needed.
__device__ __forceinline__ void wave_lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Workgroup barrier that orders LDS accesses only: global stores and
// prefetch loads still in flight are not waited for.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// One workgroup streams one source frame (or a band of its output rows) top
// to bottom; each of its waves owns one band of up to 64 output columns and
// works alone -- no workgroup barrier anywhere:
//   * y pass, in registers: lane t owns PX consecutive pixels of the band's
//     source span, reads them with one buffer load per row (prefetched four
//     rows ahead), unpacks them once and adds them with wave-uniform scalar
//     weights into M rotating accumulators, one per output row that can
//     still read the row;
//   * when an output row completes, each lane writes its PX pixels to the
//     wave's LDS row (float4 per pixel, 16*PX bytes per lane: no bank
//     conflicts), and the x pass follows at once: lane j = one output column,
//     its KX weights in registers, one ds_read_b128 and three FMAs per tap,
//     then the normalisation FMA and the conversion into the wave's stage;
//   * patch 16: every four output rows the stage holds, for each (patch,
//     channel), the band's part of one 64-value run; it leaves as 16-byte
//     stores, eight lanes per 128-byte run, whole cache lines;
//   * patch 14: a 14-row run (392 bytes in bf16) is not a whole number of
//     cache lines, and the two frames of a pair interleave every 196 values,
//     so stores from one frame alone leave most lines part-written (the L2
//     then fetches them from HBM, and writes them in 32-byte pieces).  The
//     workgroup is therefore four waves: the pair's two frames over two
//     neighbouring bands, which then also read their shared source pixels
//     in step.  They share a stage in output order, [patch][c][frame][14][14]:
//     after every 14th row the four waves write the bands' finished output
//     rows whole (the two patches of a merge window are one contiguous run).
template <int M, int KX, int PX, int OUT_BF16, int P>
__global__ __launch_bounds__(P == 16 ? 64 : 256) __attribute__((amdgpu_waves_per_eu(
    M * PX > 12 || KX >= 20 || 3 * M * PX + KX >= 52 || (OUT_BF16 == 0 && M * PX >= 12) ? 4 : 5)))
void stream_kernel(PlanView plan, int wg0, void* out, Norm norm) {
    static_assert(P == 16 || P == 14, "patch 16 or 14");
    using elem_t = typename std::conditional<OUT_BF16 != 0, uint16_t, float>::type;
    constexpr int kRowPx = 64 * PX;
    constexpr int V = 3 * PX;                      // values per lane per source row
    constexpr int kLoadDwords = PX == 4 ? 4 : 3;   // 3*PX bytes plus up to 3 of misalignment
    constexpr int S = 16 / int(sizeof(elem_t));    // output columns per 16-byte store
    extern __shared__ __align__(16) unsigned char smem[];

    const int lane = static_cast<int>(threadIdx.x) & 63;
    // patch 14: four waves, two neighbouring bands x the pair's two frames;
    // wave wv takes frame wv & 1 of band wv >> 1 of the workgroup's two
    const int wv = P == 16 ? 0 : __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    const int fw = wv & 1;
    // Workgroup -> (unit, column band), from the host's list (which places
    // the bands of one unit on one XCD)
    const uint32_t wg = as_const(plan.wgs)[wg0 + static_cast<int>(blockIdx.x)];
    if (wg == kNoWork) return;
    const int u = static_cast<int>(wg & kWgUnitMask);
    const int wave = static_cast<int>(wg >> kWgBandShift);
    const cptr<StreamUnit> up = as_const(plan.units) + u;
    const int u_item = up->item, u_pf = up->p_flags, i0 = up->i0, i1 = up->i1;
    const int u_p = u_pf & (kUnitBoth - 1);
    const cptr<DevItem> it = as_const(plan.items) + u_item;
    const int w = it->w;
    const int band = it->band;
    // patch 14: the list names the workgroup's pair of bands
    const int j0_wg = P == 16 ? wave * band : 2 * wave * band;   // the workgroup's first column
    const int nbw_wg = min(P == 16 ? band : 2 * band, w - j0_wg);   // and its columns
    const int j0 = P == 16 ? j0_wg : j0_wg + (wv >> 1) * band;  // first output column of this wave
    const int nbw = min(band, w - j0);             // its columns (none: a missing second band)
    const int tt = u_p >> 1;
    const int dt_self = P == 16 ? (u_p & 1) : fw;   // patch 14 units start at the pair's first frame
    // the item's row geometry, held in scalar registers (as constant-memory
    // loads the compiler would re-read them at every store-out)
    int64_t it_row_off = it->row_off;
    int it_hm = it->hm, it_wm = it->wm;
    asm volatile("" : "+s"(it_row_off), "+s"(it_hm), "+s"(it_wm));
    const bool both = (u_pf & kUnitBoth) != 0;

    // patch 16: [row][stage [3][4][64]]; patch 14: [row of each of the four
    // waves][stage [8 patches][1176]]
    float4* row = reinterpret_cast<float4*>(smem + wv * kRowPx * 16);                  // [kRowPx]
    elem_t* stage = reinterpret_cast<elem_t*>(smem + (P == 16 ? 1 : 4) * kRowPx * 16);

    // Patch 14 store-out of patch row pr (output rows 14 pr .. 14 pr + 13):
    // the workgroup's output rows leave the stage whole, in 16-byte pieces
    // shared out over its four waves; consecutive pieces are consecutive in
    // memory within each merge window.
    auto store_rows = [&](int pr) __attribute__((always_inline)) {
        constexpr int kRowElems = 6 * P * P;                           // 1176
        constexpr int VPP = 16 / int(sizeof(elem_t));                  // values per piece
        constexpr int PPR = kRowElems / VPP;                           // pieces per row
        static_assert(kRowElems % VPP == 0, "rows are whole 16-byte pieces");
        const int nq = nbw_wg / 14;
        const int64_t win_row0 = it_row_off + (int64_t(tt) * it_hm + (pr >> 1)) * it_wm * 4 + (pr & 1) * 2;
        using u4v = unsigned __attribute__((ext_vector_type(4)));
        for (int e = static_cast<int>(threadIdx.x); e < nq * PPR; e += 256) {
            const int q = e / PPR;
            const int pc = e - q * PPR;
            const int qa = j0_wg / 14 + q;
            const u4v val = *reinterpret_cast<const u4v*>(stage + q * kRowElems + pc * VPP);
            elem_t* dst = static_cast<elem_t*>(out) + (win_row0 + (qa >> 1) * 4 + (qa & 1)) * kRowElems + pc * VPP;
            __builtin_nontemporal_store(val, reinterpret_cast<u4v*>(dst));
        }
    };
    if (P == 14 && (nbw <= 0 || (both && fw == 1))) {
        // a wave with no frame to stream (the second frame of a pair whose
        // frames are one, or a band past the item's last) reads no table; it
        // keeps step with the other waves' barriers (two per patch row) and
        // stores its share of the rows
        for (int pr = i0 / 14; pr < i1 / 14; ++pr) {
            lds_barrier();
            store_rows(pr);
            lds_barrier();
        }
        return;
    }

    // x pass: output column j0 + lane keeps its KX column weights in registers.
    const cptr<int32_t> tables = as_const(plan.tables);
    const cptr<int32_t> sx_start = tables + it->sx_off;
    const cptr<float> sx_w = (cptr<float>)(sx_start + w);
    const bool xlane = lane < nbw;
    int sj = 0;
    float wx[KX];
    {
        const int jx = xlane ? j0 + lane : w - 1;   // idle lanes read a valid entry, keep zeros
        const cptr<float> src = sx_w + int64_t(jx) * KX;
        if (xlane) sj = sx_start[jx];
#pragma unroll
        for (int k = 0; k < KX; ++k) wx[k] = xlane ? src[k] : 0.f;
    }

    const cptr<int32_t> xs = tables + it->tx_off;   // window starts of the x axis
    const int x0 = xs[j0];                          // first source pixel of the band
    const cptr<int32_t> ys = tables + it->ty_off;
    const cptr<float> slot_w = (cptr<float>)(tables + it->sy_off);             // [H + 6][8]
    const cptr<int32_t> close_row = tables + it->sy_off + (it->H + kSlotMax) * kSlotWords;  // [h]

    // Source frame, read through buffer resources (loads past a resource's
    // range return 0).  Every load is dword-aligned: unaligned per-lane
    // loads cost about a third of the read bandwidth on gfx950.
    const int f = as_const(plan.indices)[it->idx_off + u_p + (P == 16 ? 0 : fw)];
    const uintptr_t fa = reinterpret_cast<uintptr_t>(it->frames + int64_t(f) * it->frame_bytes);
    const uint32_t lead = static_cast<uint32_t>(fa & 3u);
    // Range = the frame rounded up to whole dwords: the range check is per
    // dword, and the dword holding the frame's last byte lies in that byte's
    // (4-byte aligned) page, so it is always readable.
    const uint32_t range = static_cast<uint32_t>((it->frame_bytes + lead + 3) & ~int64_t(3));
    const uint32_t row_bytes = static_cast<uint32_t>(it->W) * 3u;
    // The lane's first byte inside a row, from the dword-aligned frame base.
    // A lane wholly past the row's end reads garbage that no column weight
    // ever touches; it is clamped to the row's end.
    const uint32_t lane_off = lead + min(3u * static_cast<uint32_t>(x0 + PX * lane), row_bytes);
    // v_c = a_c * (R_c + z_c): the x pass starts its sums at z_c, so the
    // normalisation costs one multiply per value
    const float a0 = norm.a[0], a1 = norm.a[1], a2 = norm.a[2];
    const float z0 = norm.z[0], z1 = norm.z[1], z2 = norm.z[2];

    // acc[s][q]: the RGB sums of pixel q of the lane in slot s, as a float3
    // so that each pixel leaves with one 12-byte LDS write straight from its
    // registers.
    f3 acc[M][PX];
#pragma unroll
    for (int s = 0; s < M; ++s)
#pragma unroll
        for (int q = 0; q < PX; ++q) acc[s][q] = f3{0.f, 0.f, 0.f};

    // Output row i accumulates in acc[i % M].  The band starts at the first
    // source row of output row i0; output rows before i0 that are still open
    // there collect partial sums, which are discarded when they close.
    const int y0 = ys[i0];
    const int y1 = close_row[i1 - 1] + 1;   // past the frame: zero-weight rows, loads return 0
    int base = i0;        // next output row to close
    while (base > 0 && close_row[base - 1] >= y0) --base;
    int slot = base % M;
    int next_close = close_row[base];
    int after_close = close_row[base + 1];   // read one ahead (the table ends in two sentinels)

    // Rows are visited in blocks of four starting at a multiple of 4, so
    // that y % 4 = k is known at every step: the lane's byte offset inside
    // row y is then voff[k] (dword aligned) + shf[k] (0..3), with the row
    // block's own offset, a multiple of 4, in the block's buffer resource.
    using load_t = typename std::conditional<kLoadDwords == 4, uint4, uint3>::type;
    // sel[k]: the v_perm selector that moves bytes shift and shift + 1 of
    // the loaded dwords (shift = the lane's byte offset mod 4 in row phase k)
    // into the low bytes of two 16-bit halves and zeroes the high bytes.
    // The x pass reads pixels [0, sx_start[last column] + KX) of the band's
    // source span; a lane whose pixels all lie past that loads nothing: its
    // offset is past every resource's range (such loads return zeros without
    // a memory access), or, in a frame of 2 GiB or more, inside the frame.
    // Neighbouring bands would otherwise fetch the same pixels twice.
    const int span_px = sx_start[j0 + nbw - 1] + KX;
    const bool lane_reads = PX * lane < span_px;
    uint32_t voff[kPrefetch], sel[kPrefetch];
#pragma unroll
    for (int k = 0; k < kPrefetch; ++k) {
        const uint32_t c = lane_off + static_cast<uint32_t>(k) * row_bytes;
        voff[k] = lane_reads ? (c & ~3u) : 0x7FFFFFF0u;
        sel[k] = 0x0C000C00u | (c & 3u) | (((c & 3u) + 1u) << 16);
    }
    // Row yb + k of the block starting at yb: a resource based at the
    // block's first row (a multiple of 4 bytes past the aligned frame base)
    // with the rest of the frame as its range.
    auto load_row = [&](int yb, int k) __attribute__((always_inline)) -> load_t {
        // (the block is wave-uniform; say so, or the descriptor would be built per lane)
        const uint32_t o = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(yb)) * row_bytes;
        const uint32_t n = uniform_sat_sub(range, o);
        const uintptr_t bp = fa - lead + o;
        const uint32_t b_lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(bp));
        const uint32_t b_hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(bp >> 32));
        const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
            reinterpret_cast<void*>((uintptr_t(b_hi) << 32) | b_lo), (short)0, static_cast<int>(n), 0x00020000);
        if constexpr (kLoadDwords == 4) {
            const auto r = __builtin_amdgcn_raw_buffer_load_b128(rb, voff[k], 0, 0);
            return make_uint4(r[0], r[1], r[2], r[3]);
        } else {
            const auto r = __builtin_amdgcn_raw_buffer_load_b96(rb, voff[k], 0, 0);
            return make_uint3(r[0], r[1], r[2]);
        }
    };

    // Patch 14: the lane's column j0 + lane is column lane % 14 of the
    // band's patch lane / 14, at this offset of the stage's patch-row origin.
    const int st14 = ((j0 - j0_wg) / 14 + lane / 14) * (6 * P * P) + lane % 14;

    // Store-out pieces of this lane (patch 16): piece e = lane + 64 r of the
    // band's (patch q, channel c, row ry, piece) runs, as a stage offset
    // (-1: none) and an output offset relative to the merge-window row block.
    constexpr int kPieces = 16 / S;
    constexpr int kPerPatch = 3 * 4 * kPieces;
    constexpr int kStoreIter = (4 * kPerPatch + 63) / 64;
    int st_off[kStoreIter], dst_off[kStoreIter];
    {
        const int n_seg = (nbw >> 4) * kPerPatch;
#pragma unroll
        for (int r = 0; r < kStoreIter; ++r) {
            const int e = lane + 64 * r;
            const int q = e / kPerPatch;
            const int rr = e - q * kPerPatch;
            const int c = rr / (4 * kPieces);
            const int ry = (rr / kPieces) & 3;
            const int piece = rr % kPieces;
            const int qa = (j0 >> 4) + q;
            st_off[r] = e < n_seg ? (c * 4 + ry) * 64 + q * 16 + piece * S : -1;
            dst_off[r] = ((qa >> 1) * 4 + (qa & 1)) * kRow + (c * 2) * 256 + ry * 16 + piece * S;
        }
    }

    // x pass of output row i, normalise, stage; at the end of every group of
    // four rows of a patch (for patch 14 also after its last two): store.
    auto x_pass = [&](int i) __attribute__((always_inline)) {
        const int yy = P == 16 ? (i & 3) : ((i % 14) & 3);
        if (xlane) {
            float r0 = z0, r1 = z1, r2 = z2;
            const float4* src = row + sj;
#pragma unroll
            for (int g = 0; g < KX; g += 4) {
                // four taps at a time (KX mod 4 in a last group): bounds the
                // LDS values held in registers
                __builtin_amdgcn_sched_barrier(0);
                constexpr int kLast = KX % 4 == 0 ? 4 : KX % 4;
                const int n = g + 4 <= KX ? 4 : kLast;
                float4 q[4];
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    if (k < n) q[k] = src[g + k];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    if (k < n) {
                        r0 = fmaf(wx[g + k], q[k].x, r0);
                        r1 = fmaf(wx[g + k], q[k].y, r1);
                        r2 = fmaf(wx[g + k], q[k].z, r2);
                    }
                }
                // the whole 16-byte slots are read (on gfx950 a 16-byte LDS
                // read is cheaper than a 12-byte one); using the fourth words
                // once per group, not per read, lets the reads issue back to
                // back under one wait
                if (n == 4)
                    asm volatile("" : : "v"(q[0].w), "v"(q[1].w), "v"(q[2].w), "v"(q[3].w));
                else if (n == 3)
                    asm volatile("" : : "v"(q[0].w), "v"(q[1].w), "v"(q[2].w));
                else if (n == 2)
                    asm volatile("" : : "v"(q[0].w), "v"(q[1].w));
                else
                    asm volatile("" : : "v"(q[0].w));
            }
            __builtin_amdgcn_sched_barrier(0);
            const float v0 = r0 * a0;
            const float v1 = r1 * a1;
            const float v2 = r2 * a2;
            constexpr int kCh = P == 16 ? 256 : 2 * P * P;   // stage channel stride
            elem_t* st = P == 16 ? stage + yy * 64 + lane : stage + st14 + (i % 14) * 14 + dt_self * (P * P);
            elem_t e0, e1, e2;
            if constexpr (OUT_BF16 != 0) {
                e0 = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v0));
                e1 = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v1));
                e2 = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v2));
            } else {
                e0 = v0;
                e1 = v1;
                e2 = v2;
            }
            st[0] = e0;
            st[kCh] = e1;
            st[2 * kCh] = e2;
            if (P == 14 && both) {   // one frame stands for both halves of the pair
                st[P * P] = e0;
                st[kCh + P * P] = e1;
                st[2 * kCh + P * P] = e2;
            }
        }
        if constexpr (P == 14) {
            if (i % 14 == 13) {
                lds_barrier();
                store_rows(i / 14);
                lds_barrier();
            }
        } else if (yy == 3) {
            wave_lds_fence();
            // rows i-3 .. i: the lane's 16-byte pieces (precomputed below)
            const int yq = (i & 15) >> 2;
            const int bh = i >> 5;
            const int mh = (i >> 4) & 1;
            const int64_t win_row0 = it_row_off + (int64_t(tt) * it_hm + bh) * it_wm * 4 + mh * 2;
            elem_t* const obase = static_cast<elem_t*>(out) + win_row0 * kRow + yq * 64;
#pragma unroll
            for (int r = 0; r < kStoreIter; ++r) {
                if (st_off[r] >= 0) {
                    const uint4 val = *reinterpret_cast<const uint4*>(stage + st_off[r]);
                    elem_t* dst = obase + dst_off[r];
                    // non-temporal: the rows are not read again here
                    using u4v = unsigned __attribute__((ext_vector_type(4)));
                    const u4v vv = {val.x, val.y, val.z, val.w};
                    if (both) {
                        __builtin_nontemporal_store(vv, reinterpret_cast<u4v*>(dst));
                        __builtin_nontemporal_store(vv, reinterpret_cast<u4v*>(dst + 256));
                    } else {
                        __builtin_nontemporal_store(vv, reinterpret_cast<u4v*>(dst + dt_self * 256));
                    }
                }
            }
            wave_lds_fence();
        }
    };

    // The lane's 3*PX source bytes of a row, unpacked two at a time into
    // 16-bit halves with zero high bytes: byte value b reads as the f16
    // number b * 2^-24 (a denormal, exact).  The slot weights carry the
    // factor 2^24, so the mixed-precision FMAs below form w * b exactly, as a
    // float copy of the byte would, without a conversion per value.  Pair p
    // (values 2p, 2p+1) starts at byte shift + 2p, inside dwords p/2 and
    // p/2 + 1: the selector is sel, plus 2 per byte for odd p.
    constexpr int kPairs = (V + 1) / 2;
    auto unpack = [&](load_t cur, uint32_t s0, uint32_t (&hv)[kPairs]) __attribute__((always_inline)) {
        uint32_t d[kLoadDwords];
        d[0] = cur.x;
        d[1] = cur.y;
        d[2] = cur.z;
        if constexpr (kLoadDwords == 4) d[3] = cur.w;
        // (formed here, per row: hoisted out of the row loop, the four odd
        // selectors would hold four more registers)
        uint32_t s1;
        asm volatile("v_add_u32 %0, 0x20002, %1" : "=v"(s1) : "v"(s0));
#pragma unroll
        for (int p = 0; p < kPairs; ++p) {
            const int j = p >> 1;
            const int hi = j + 1 < kLoadDwords ? j + 1 : j;
            hv[p] = __builtin_amdgcn_perm(d[hi], d[j], (p & 1) ? s1 : s0);
        }
    };

    // Source row y (its values in hv) into the slots; then closes the output
    // rows whose close row is y.
    auto process_row = [&](int y, const uint32_t (&hv)[kPairs], const float (&wr)[M]) __attribute__((always_inline)) {
        float v[V];
#pragma unroll
        for (int q = 0; q < V; ++q) {
            const h2 pr = __builtin_bit_cast(h2, hv[q >> 1]);
            v[q] = static_cast<float>((q & 1) ? pr.y : pr.x);   // folds into the FMAs (fma_mix)
        }
        // every slot takes this row with its weight (zero where its output row does not read it)
#pragma unroll
        for (int s = 0; s < M; ++s) {
            const float ws = wr[s];
#pragma unroll
            for (int q = 0; q < PX; ++q) {
                acc[s][q].x = fmaf(ws, v[3 * q], acc[s][q].x);
                acc[s][q].y = fmaf(ws, v[3 * q + 1], acc[s][q].y);
                acc[s][q].z = fmaf(ws, v[3 * q + 2], acc[s][q].z);
            }
        }
        // every output row of the unit that closes on this row (several when
        // the axis is upscaled, or at the bottom border), in order
        while (y == next_close && base < i1) {   // wave-uniform
            const bool keep = base >= i0;
            if (keep) wave_lds_fence();
            // the closing slot goes to the wave's LDS row (kept rows only) and
            // restarts at zero; each case names its registers statically
#pragma unroll
            for (int s = 0; s < M; ++s) {
                if (slot == s) {
                    if (keep) {
#pragma unroll
                        for (int q = 0; q < PX; ++q) *reinterpret_cast<f3*>(row + PX * lane + q) = acc[s][q];
                    }
#pragma unroll
                    for (int q = 0; q < PX; ++q) acc[s][q] = f3{0.f, 0.f, 0.f};
                }
            }
            if (keep) {
                wave_lds_fence();
                x_pass(base);
            }
            ++base;
            slot = slot + 1 == M ? 0 : slot + 1;
            next_close = after_close;
            after_close = close_row[base + 1];
        }
    };

    // Rows are loaded one block (four rows) ahead, unconditionally: a load
    // past the band or the frame is harmless (in-frame data that is never
    // used, or zeros from the range check), and an unconditional load keeps
    // every prefetch register in place.  The first block's loads are issued
    // in row order, as the loop issues them, so that the oldest load is
    // always the next one needed.

    const int yb0 = y0 & ~3;
    load_t pf[kPrefetch];
#pragma unroll
    for (int k = 0; k < kPrefetch; ++k) {
        pf[k] = load_row(yb0, k);
        __builtin_amdgcn_sched_barrier(0);
    }

    for (int yb = yb0; yb < y1; yb += kPrefetch) {
        // the block's slot weights, loaded together ahead of its rows: one
        // wait for scalar loads per block, not per row (a block starts at a
        // row below H and the table has kSlotMax rows past the frame's
        // last, so all four rows are inside it)
        const cptr<float> wblk = slot_w + yb * kSlotWords;
        float wk[kPrefetch][M];
#pragma unroll
        for (int k = 0; k < kPrefetch; ++k)
#pragma unroll
            for (int s = 0; s < M; ++s) wk[k][s] = wblk[k * kSlotWords + s];
#pragma unroll
        for (int k = 0; k < kPrefetch; ++k) {
            const int y = yb + k;
            // unpack first: the next load then reuses the same registers
            uint32_t hv[kPairs];
            unpack(pf[k], sel[k], hv);
            // (keep the unpacking here, ahead of the load that reuses
            // pf[k]'s registers; otherwise it sinks into the conditional use
            // below and pf[k] has to be copied while its load is in flight)
#pragma unroll
            for (int q = 0; q < kPairs; ++q) asm volatile("" : : "v"(hv[q]));
            // (issued at raised wave priority, so that the load leaves ahead
            // of other waves' arithmetic and the memory stream stays full)
            __builtin_amdgcn_s_setprio(2);
            pf[k] = load_row(yb + kPrefetch, k);
            __builtin_amdgcn_s_setprio(0);
            if (y >= y0 && y < y1) process_row(y, hv, wk[k]);
        }
    }
}

template <int M, int KX, int PX>
int launch_stream_shape(const PlanView& plan, const StreamLaunch& L, void* out, int out_dtype,
                        const Norm& norm, hipStream_t stream) {
    const int lds = stream_wave_bytes(PX, KX, out_dtype == 1 ? 2 : 4, L.patch);
    dim3 grid(static_cast<unsigned>(L.count)), block(L.patch == 14 ? 256 : 64);
    if (L.patch == 14) {
        if (out_dtype == 1)
            hipLaunchKernelGGL((stream_kernel<M, KX, PX, 1, 14>), grid, block, lds, stream, plan, L.first, out, norm);
        else
            hipLaunchKernelGGL((stream_kernel<M, KX, PX, 0, 14>), grid, block, lds, stream, plan, L.first, out, norm);
    } else if (out_dtype == 1) {
        hipLaunchKernelGGL((stream_kernel<M, KX, PX, 1, 16>), grid, block, lds, stream, plan, L.first, out, norm);
    } else {
        hipLaunchKernelGGL((stream_kernel<M, KX, PX, 0, 16>), grid, block, lds, stream, plan, L.first, out, norm);
    }
    return static_cast<int>(hipGetLastError());
}


// ===========================================================================
// x-first streaming kernel (patch 16): vertical scales near 1
// ===========================================================================
//
// The streaming kernel above resamples y first and gathers each closed
// output row's x windows from LDS, 16 bytes per tap and lane.  Where the
// vertical scale is near 1 -- upscales, and downscales up to about 1.6x --
// an output row closes on almost every source row, and those gathers bound
// the kernel.  This one resamples x first and keeps LDS for the stage only:
//   * lane j (output column j0 + j) loads its own window of each source row
//     straight from the frame: the dwords holding its 3 KXE bytes (ND of
//     them, dword aligned, four rows ahead, or two for column pairs);
//     neighbouring lanes' windows overlap, and the overlap is served by the
//     L1 cache, not HBM;
//   * with DB > 0 a lane takes two neighbouring columns, j0 + 2j and
//     j0 + 2j + 1 (a wave covers 128): it loads the pair's window, which is
//     the first column's window extended by DB pixels, and the second column
//     gets its KXE weights at their place in it (its window starts 0 to DB
//     pixels after the first's) with zeros elsewhere.  A pair reads about
//     half the bytes that two single columns read, and its tap bytes are
//     extracted once for both columns;
//   * the lane shifts the window to its first byte (v_alignbyte by the
//     window's byte misalignment) and moves the bytes of taps 2m and 2m + 1
//     of each channel (an odd count's last tap alone) into the two 16-bit
//     halves of a register with zero high bytes (one v_perm with a fixed
//     selector): byte value b reads as the f16 denormal b * 2^-24, as in
//     the y-first kernel, so the x sums are mixed-precision FMAs with no
//     conversion (exact products);
//   * the three channel sums go into M rotating accumulator slots with the
//     slot table's wave-uniform weights, which carry the factor 2^24; a slot
//     starts at z_c = -255 mean_c, so a closed slot holds R + z_c;
//   * a closing output row is multiplied by a_c = 1/(255 std_c), converted
//     and staged; every four rows the stage leaves as 16-byte stores, eight
//     lanes per 128-byte run, as in the y-first kernel.
// Window bytes past the end of a row are the next row's (or zeros past the
// frame, from the buffer range check); they meet only zero weights.
template <int M, int KXE, int DB, int OUT_BF16>
__global__ __launch_bounds__(64) void xfirst_kernel(PlanView plan, int wg0, void* out, Norm norm) {
    using elem_t = typename std::conditional<OUT_BF16 != 0, uint16_t, float>::type;
    static_assert(KXE >= 4 && KXE <= 12 && DB >= 0 && DB <= 2, "tap counts from 4 to 12, pair offsets to 2");
    constexpr int CPL = DB > 0 ? 2 : 1;            // output columns per lane
    constexpr int BW = 64 * CPL;                   // output columns per wave
    constexpr int KW = KXE + DB;                   // window taps from the lane's window start
    constexpr int NA = (3 * KW + 3) / 4;           // dwords of the window from its first byte
    constexpr int ND = (3 * KW + 6) / 4;           // dwords loaded: the window at any alignment
    constexpr int S = 16 / int(sizeof(elem_t));    // output columns per 16-byte store
    extern __shared__ __align__(16) unsigned char smem[];
    elem_t* const stage = reinterpret_cast<elem_t*>(smem);   // [3][4][BW]

    const int lane = static_cast<int>(threadIdx.x) & 63;
    const uint32_t wg = as_const(plan.wgs)[wg0 + static_cast<int>(blockIdx.x)];
    if (wg == kNoWork) return;
    const int u = static_cast<int>(wg & kWgUnitMask);
    const int wave = static_cast<int>(wg >> kWgBandShift);
    const cptr<StreamUnit> up = as_const(plan.units) + u;
    const int u_item = up->item, u_pf = up->p_flags, i0 = up->i0, i1 = up->i1;
    const int u_p = u_pf & (kUnitBoth - 1);
    const cptr<DevItem> it = as_const(plan.items) + u_item;
    const int w = it->w;
    const int band = it->band;
    const int j0 = wave * band;                    // first output column of this wave
    const int nbw = min(band, w - j0);             // its columns
    const int tt = u_p >> 1;
    const int dt_self = u_p & 1;
    int64_t it_row_off = it->row_off;
    int it_hm = it->hm, it_wm = it->wm;
    asm volatile("" : "+s"(it_row_off), "+s"(it_hm), "+s"(it_wm));
    const bool both = (u_pf & kUnitBoth) != 0;

    // Column table: window start relative to the band's first source pixel,
    // then KXE weights (zero past the window).  Lanes past the band's last
    // column take its first column's entry (valid reads) with zero weights.
    // A pair's second column (widths are multiples of 32, so it is in the
    // band with the first) takes its weights at its offset in the window.
    const cptr<int32_t> tables = as_const(plan.tables);
    const cptr<int32_t> sx_start = tables + it->sx_off;
    const cptr<float> sx_w = (cptr<float>)(sx_start + w);
    const bool xlane = CPL * lane < nbw;
    const int jx = xlane ? j0 + CPL * lane : j0;
    const int sj = sx_start[jx];
    float wx[KXE];
    {
        const cptr<float> src = sx_w + int64_t(jx) * KXE;
#pragma unroll
        for (int k = 0; k < KXE; ++k) wx[k] = xlane ? src[k] : 0.f;
    }
    float wb[DB > 0 ? KW : 1];
    if constexpr (DB > 0) {
        const int db = sx_start[jx + 1] - sj;     // 0 .. DB
        const cptr<float> src = sx_w + int64_t(jx + 1) * KXE;
        float t[KXE];
#pragma unroll
        for (int k = 0; k < KXE; ++k) t[k] = src[k];
#pragma unroll
        for (int k = 0; k < KW; ++k) {
            float v = 0.f;
#pragma unroll
            for (int d = 0; d <= DB; ++d)
                if (k - d >= 0 && k - d < KXE) v = db == d ? t[k - d] : v;
            wb[k] = xlane ? v : 0.f;
        }
    }
    const cptr<int32_t> xs = tables + it->tx_off;
    const int x0 = xs[j0];                         // first source pixel of the band
    const cptr<int32_t> ys = tables + it->ty_off;
    const cptr<float> slot_w = (cptr<float>)(tables + it->sy_off);
    const cptr<int32_t> close_row = tables + it->sy_off + (it->H + kSlotMax) * kSlotWords;

    // Source frame through buffer resources, as in the y-first kernel: row
    // blocks of four start at a multiple of 4 rows, so each block's offset
    // (a multiple of 4 bytes) goes into its resource, and the lane's window
    // in row phase k sits at the fixed dword offset voff[k], byte sh[k].
    const int f = as_const(plan.indices)[it->idx_off + u_p];
    const uintptr_t fa = reinterpret_cast<uintptr_t>(it->frames + int64_t(f) * it->frame_bytes);
    const uint32_t lead = static_cast<uint32_t>(fa & 3u);
    const uint32_t range = static_cast<uint32_t>((it->frame_bytes + lead + 3) & ~int64_t(3));
    const uint32_t row_bytes = static_cast<uint32_t>(it->W) * 3u;
    // (one offset per 16-byte chunk of the window, so that no row adds them)
    constexpr int NC = (ND + 3) / 4;
    // (column pairs form each row's offsets from c0 as they go; single
    // columns keep the four row phases' offsets)
    constexpr bool kLive = DB > 0;
    const uint32_t c0 = lead + 3u * static_cast<uint32_t>(x0 + sj);
    uint32_t voff[kLive ? 1 : 4][NC], sh[kLive ? 1 : 4];
    if constexpr (!kLive) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t c = c0 + static_cast<uint32_t>(k) * row_bytes;
#pragma unroll
            for (int i = 0; i < NC; ++i) voff[k][i] = (c & ~3u) + 16u * static_cast<uint32_t>(i);
            sh[k] = c & 3u;
        }
    }
    auto phase_off = [&](int k, int i) __attribute__((always_inline)) -> uint32_t {
        if constexpr (kLive)
            return ((c0 + static_cast<uint32_t>(k) * row_bytes) & ~3u) + 16u * static_cast<uint32_t>(i);
        else
            return voff[k][i];
    };
    auto phase_sh = [&](int k) __attribute__((always_inline)) -> uint32_t {
        if constexpr (kLive)
            return (c0 + static_cast<uint32_t>(k) * row_bytes) & 3u;
        else
            return sh[k];
    };
    struct Win {
        uint32_t d[ND];
    };
    auto load_row = [&](int yb, int k) __attribute__((always_inline)) -> Win {
        const uint32_t o = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(yb)) * row_bytes;
        const uint32_t n = uniform_sat_sub(range, o);
        const uintptr_t bp = fa - lead + o;
        const uint32_t b_lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(bp));
        const uint32_t b_hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(bp >> 32));
        const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
            reinterpret_cast<void*>((uintptr_t(b_hi) << 32) | b_lo), (short)0, static_cast<int>(n), 0x00020000);
        Win r;
#pragma unroll
        for (int i = 0; i < ND; i += 4) {
            const uint32_t vo = phase_off(k, i / 4);
            if (ND - i >= 4) {
                const auto v = __builtin_amdgcn_raw_buffer_load_b128(rb, vo, 0, 0);
                r.d[i] = v[0];
                r.d[i + 1] = v[1];
                r.d[i + 2] = v[2];
                r.d[i + 3] = v[3];
            } else if (ND - i == 3) {
                const auto v = __builtin_amdgcn_raw_buffer_load_b96(rb, vo, 0, 0);
                r.d[i] = v[0];
                r.d[i + 1] = v[1];
                r.d[i + 2] = v[2];
            } else if (ND - i == 2) {
                const auto v = __builtin_amdgcn_raw_buffer_load_b64(rb, vo, 0, 0);
                r.d[i] = v[0];
                r.d[i + 1] = v[1];
            } else {
                r.d[i] = __builtin_amdgcn_raw_buffer_load_b32(rb, vo, 0, 0);
            }
        }
        return r;
    };

    const float a0 = norm.a[0], a1 = norm.a[1], a2 = norm.a[2];
    const float z0 = norm.z[0], z1 = norm.z[1], z2 = norm.z[2];
    float acc[M][3 * CPL];   // channels of the lane's first column, then its second's
#pragma unroll
    for (int s = 0; s < M; ++s)
#pragma unroll
        for (int q = 0; q < CPL; ++q) {
            acc[s][3 * q + 0] = z0;
            acc[s][3 * q + 1] = z1;
            acc[s][3 * q + 2] = z2;
        }

    const int y0 = ys[i0];
    const int y1 = close_row[i1 - 1] + 1;
    int base = i0;
    while (base > 0 && close_row[base - 1] >= y0) --base;
    int slot = base % M;
    int next_close = close_row[base];
    int after_close = close_row[base + 1];

    // store-out pieces, as in the y-first kernel (patch 16)
    constexpr int kPieces = 16 / S;
    constexpr int kPerPatch = 3 * 4 * kPieces;
    constexpr int kStoreIter = (BW / 16 * kPerPatch + 63) / 64;
    int st_off[kStoreIter], dst_off[kStoreIter];
    {
        const int n_seg = (nbw >> 4) * kPerPatch;
#pragma unroll
        for (int r = 0; r < kStoreIter; ++r) {
            const int e = lane + 64 * r;
            const int q = e / kPerPatch;
            const int rr = e - q * kPerPatch;
            const int c = rr / (4 * kPieces);
            const int ry = (rr / kPieces) & 3;
            const int piece = rr % kPieces;
            const int qa = (j0 >> 4) + q;
            st_off[r] = e < n_seg ? (c * 4 + ry) * BW + q * 16 + piece * S : -1;
            dst_off[r] = ((qa >> 1) * 4 + (qa & 1)) * kRow + (c * 2) * 256 + ry * 16 + piece * S;
        }
    }
    auto store_out = [&](int i) __attribute__((always_inline)) {   // rows i-3 .. i
        wave_lds_fence();
        const int yq = (i & 15) >> 2;
        const int bh = i >> 5;
        const int mh = (i >> 4) & 1;
        const int64_t win_row0 = it_row_off + (int64_t(tt) * it_hm + bh) * it_wm * 4 + mh * 2;
        elem_t* const obase = static_cast<elem_t*>(out) + win_row0 * kRow + yq * 64;
        using u4v = unsigned __attribute__((ext_vector_type(4)));
#pragma unroll
        for (int r = 0; r < kStoreIter; ++r) {
            if (st_off[r] >= 0) {
                const uint4 val = *reinterpret_cast<const uint4*>(stage + st_off[r]);
                elem_t* dst = obase + dst_off[r];
                const u4v vv = {val.x, val.y, val.z, val.w};
                if (both) {
                    __builtin_nontemporal_store(vv, reinterpret_cast<u4v*>(dst));
                    __builtin_nontemporal_store(vv, reinterpret_cast<u4v*>(dst + 256));
                } else {
                    __builtin_nontemporal_store(vv, reinterpret_cast<u4v*>(dst + dt_self * 256));
                }
            }
        }
        wave_lds_fence();
    };

    // Row y (its window from the first byte: byte t of a[] is window byte t):
    // the window sums, the slots, then the output rows that close on y.
    auto process_row = [&](int y, const uint32_t (&a)[NA], const float (&wr)[M]) __attribute__((always_inline)) {
        float tsum[3 * CPL];
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            float t = 0.f, tb = 0.f;
#pragma unroll
            for (int m = 0; m < (KW + 1) / 2; ++m) {
                // channel c of taps 2m and 2m + 1: window bytes p and p + 3
                // (an odd count's last tap alone, its high half zero)
                constexpr int kZero = 0x0c;   // v_perm selector of a zero byte
                const bool pair = 2 * m + 1 < KW;
                const int p = 6 * m + c;
                const int lo = p >> 2;
                const int hi = lo + 1 < NA ? lo + 1 : lo;   // p + 3 stays in a[lo] when lo is the last
                const uint32_t sel = static_cast<uint32_t>((p & 3) | (kZero << 8) |
                                                           ((pair ? p + 3 - 4 * lo : kZero) << 16) | (kZero << 24));
                const h2 pr = __builtin_bit_cast(h2, __builtin_amdgcn_perm(a[hi], a[lo], sel));
                if (2 * m < KXE) t = fmaf(wx[2 * m], static_cast<float>(pr.x), t);
                if (2 * m + 1 < KXE) t = fmaf(wx[2 * m + 1], static_cast<float>(pr.y), t);
                if constexpr (DB > 0) {
                    tb = fmaf(wb[2 * m], static_cast<float>(pr.x), tb);
                    if (pair) tb = fmaf(wb[2 * m + 1], static_cast<float>(pr.y), tb);
                }
            }
            tsum[c] = t;
            if constexpr (DB > 0) tsum[3 + c] = tb;
        }
#pragma unroll
        for (int s = 0; s < M; ++s) {
            const float ws = wr[s];
#pragma unroll
            for (int q = 0; q < 3 * CPL; ++q) acc[s][q] = fmaf(ws, tsum[q], acc[s][q]);
        }
        while (y == next_close && base < i1) {   // wave-uniform
            const bool keep = base >= i0;
            const int yy = base & 3;
#pragma unroll
            for (int s = 0; s < M; ++s) {
                if (slot == s) {
                    if (keep) {
                        elem_t* st = stage + yy * BW + CPL * lane;
#pragma unroll
                        for (int c = 0; c < 3; ++c) {
                            const float sc = c == 0 ? a0 : (c == 1 ? a1 : a2);
                            const float v = acc[s][c] * sc;
                            if constexpr (DB > 0) {   // the pair's two columns as one store
                                const float vb = acc[s][3 + c] * sc;
                                if constexpr (OUT_BF16 != 0)
                                    *reinterpret_cast<uint32_t*>(st + c * 4 * BW) =
                                        uint32_t(__builtin_bit_cast(uint16_t, static_cast<__bf16>(v))) |
                                        (uint32_t(__builtin_bit_cast(uint16_t, static_cast<__bf16>(vb))) << 16);
                                else
                                    *reinterpret_cast<float2*>(st + c * 4 * BW) = make_float2(v, vb);
                            } else {
                                if constexpr (OUT_BF16 != 0)
                                    st[c * 4 * BW] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));
                                else
                                    st[c * 4 * BW] = v;
                            }
                        }
                    }
#pragma unroll
                    for (int q = 0; q < CPL; ++q) {
                        acc[s][3 * q + 0] = z0;
                        acc[s][3 * q + 1] = z1;
                        acc[s][3 * q + 2] = z2;
                    }
                }
            }
            if (keep && yy == 3) store_out(base);
            ++base;
            slot = slot + 1 == M ? 0 : slot + 1;
            next_close = after_close;
            after_close = close_row[base + 1];
        }
    };

    // Rows in flight per lane: four, or two for column pairs, whose windows
    // are twice as wide (the registers that two more would take cost more
    // occupancy than they hide latency).  Rows go in blocks of four; row k
    // of a block is in buffer k % PF.
    constexpr int PF = DB > 0 ? 2 : kPrefetch;
    static_assert(PF == 2 || PF == 4, "rows in flight divide the block of four");
    const int yb0 = y0 & ~3;
    Win pf[PF];
#pragma unroll
    for (int k = 0; k < PF; ++k) {
        pf[k] = load_row(yb0, k);
        __builtin_amdgcn_sched_barrier(0);
    }
    for (int yb = yb0; yb < y1; yb += 4) {
        const cptr<float> wblk = slot_w + yb * kSlotWords;
        float wk[4][M];
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int s = 0; s < M; ++s) wk[k][s] = wblk[k * kSlotWords + s];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int y = yb + k;
            Win& buf = pf[k % PF];
            // align first: the next load then reuses the buffer's registers
            // instead of copying them while it is in flight
            uint32_t a[NA];
            const uint32_t shk = phase_sh(k);
#pragma unroll
            for (int q = 0; q < NA; ++q)   // (a last dword past ND brings only bytes past the window)
                a[q] = __builtin_amdgcn_alignbyte(buf.d[q + 1 < ND ? q + 1 : q], buf.d[q], shk);
#pragma unroll
            for (int q = 0; q < NA; ++q) asm volatile("" : : "v"(a[q]));
            // (issued at raised wave priority, so that the load leaves ahead
            // of other waves' arithmetic and the memory stream stays full)
            __builtin_amdgcn_s_setprio(2);
            buf = load_row(yb + (k + PF) / 4 * 4, (k + PF) % 4);
            __builtin_amdgcn_s_setprio(0);
            if (y >= y0 && y < y1) process_row(y, a, wk[k]);
        }
    }
}

template <int M, int KXE, int DB>
int launch_xfirst_shape(const PlanView& plan, const StreamLaunch& L, void* out, int out_dtype,
                        const Norm& norm, hipStream_t stream) {
    const int lds = xfirst_wave_bytes(out_dtype == 1 ? 2 : 4, DB > 0 ? 2 : 1);
    dim3 grid(static_cast<unsigned>(L.count)), block(64);
    if (out_dtype == 1)
        hipLaunchKernelGGL((xfirst_kernel<M, KXE, DB, 1>), grid, block, lds, stream, plan, L.first, out, norm);
    else
        hipLaunchKernelGGL((xfirst_kernel<M, KXE, DB, 0>), grid, block, lds, stream, plan, L.first, out, norm);
    return static_cast<int>(hipGetLastError());
}

// ===========================================================================
// uint8 streaming writer
// ===========================================================================

// One single-wave workgroup streams one sampled frame (or a band of its
// output rows) top to bottom for one band of up to 64 output columns, in the
// fixed-point order, horizontal pass first:
//   * each source row arrives as in the float kernel (lane t loads pixels
//     4t .. 4t + 3 of the band's span, four rows ahead); the lane aligns its
//     12 bytes, gathers each channel's four bytes into one dword, offsets
//     them to signed bytes (value - 128) and writes the three dwords to the
//     wave's LDS row, kept as three byte planes;
//   * lane j, output column j0 + j, reads KX / 4 dwords of each plane from
//     its dword-aligned window start and forms the horizontal sum as byte
//     dot products with the three base-256 digits of its weights (held in
//     registers), d2 2^16 + d1 2^8 + d0, from a start value that restores
//     the offset and adds the rounding term; the sum is rounded to a byte;
//   * the bytes are added with wave-uniform weights into M rotating int32
//     accumulators, one per output row open at this row; a closing output
//     row is rounded to bytes into the wave's stage, and every four rows the
//     stage leaves as dword stores (a 64-column band row is 192 bytes: three
//     whole 64-byte sectors).
// The horizontal sum is exact: its true value fits int32 (|q| of a window
// sum to about 2^22, values below 2^8), so the partial sums, which wrap
// modulo 2^32, end on it.
template <int M, int KX>
__global__ __launch_bounds__(64) void resize_stream_kernel(PlanView plan, int wg0, uint8_t* out) {
    constexpr int G = KX / 4;                     // dwords per plane window
    constexpr int kPlane = 64 * kRsPx;            // bytes per plane
    constexpr int kStageRow = 3 * 64;             // stage bytes per output row
    extern __shared__ __align__(16) unsigned char smem[];

    const int lane = threadIdx.x;
    const uint32_t wg = as_const(plan.wgs)[wg0 + static_cast<int>(blockIdx.x)];
    if (wg == kNoWork) return;
    const int u = static_cast<int>(wg & kWgUnitMask);
    const int wave = static_cast<int>(wg >> kWgBandShift);
    const cptr<StreamUnit> up = as_const(plan.units) + u;
    const int u_item = up->item, u_k = up->p_flags, i0 = up->i0, i1 = up->i1;
    const cptr<DevItem> it = as_const(plan.items) + u_item;

    const int w = it->w;
    const int band = it->band;
    const int j0 = wave * band;
    const int nbw = min(band, w - j0);

    uint32_t* plane = reinterpret_cast<uint32_t*>(smem);   // [3][kPlane / 4]
    uint8_t* stage = smem + 3 * kPlane;                     // [4][kStageRow]

    // column j0 + lane: window start (dword), start value, weight digits
    const cptr<int32_t> tables = as_const(plan.tables);
    const cptr<int32_t> cstart = tables + it->sx_off;
    const cptr<int32_t> cterm = cstart + w;
    const cptr<int32_t> cdig = cterm + w;
    const bool xlane = lane < nbw;
    int sw = 0, c0 = 0;
    int32_t dg[3][G];
    {
        const int jx = xlane ? j0 + lane : w - 1;
        const cptr<int32_t> src = cdig + int64_t(jx) * 3 * G;
        if (xlane) {
            sw = cstart[jx];
            c0 = cterm[jx];
        }
#pragma unroll
        for (int d = 0; d < 3; ++d)
#pragma unroll
            for (int g = 0; g < G; ++g) dg[d][g] = xlane ? src[d * G + g] : 0;
    }
    const cptr<int32_t> xs = tables + it->tx_off;
    const int x0 = xs[j0];
    const cptr<int32_t> ys = tables + it->ty_off;
    const cptr<int32_t> slot_q = tables + it->sy_off;                                       // [H + 6][8]
    const cptr<int32_t> close_row = tables + it->sy_off + (it->H + kSlotMax) * kSlotWords;  // [h]

    // the frame through buffer resources, as in the float kernel
    const int f = as_const(plan.indices)[it->idx_off + u_k];
    const uintptr_t fa = reinterpret_cast<uintptr_t>(it->frames + int64_t(f) * it->frame_bytes);
    const uint32_t lead = static_cast<uint32_t>(fa & 3u);
    const uint32_t range = static_cast<uint32_t>((it->frame_bytes + lead + 3) & ~int64_t(3));
    const uint32_t row_bytes = static_cast<uint32_t>(it->W) * 3u;
    const uint32_t lane_off = lead + min(3u * static_cast<uint32_t>(x0 + kRsPx * lane), row_bytes);
    // lanes wholly past the pixels the horizontal pass reads load nothing
    const int span_px = 4 * cstart[j0 + nbw - 1] + KX;
    const bool lane_reads = kRsPx * lane < span_px;
    // voff[k]: the lane's dword-aligned offset in row phase k; sh[k]: its
    // byte offset (v_alignbyte uses the low two bits)
    uint32_t voff[kPrefetch], sh[kPrefetch];
#pragma unroll
    for (int k = 0; k < kPrefetch; ++k) {
        const uint32_t c = lane_off + static_cast<uint32_t>(k) * row_bytes;
        voff[k] = lane_reads ? (c & ~3u) : 0x7FFFFFF0u;
        sh[k] = c & 3u;
    }
    auto load_row = [&](int yb, int k) __attribute__((always_inline)) -> uint4 {
        const uint32_t o = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(yb)) * row_bytes;
        const uint32_t n = uniform_sat_sub(range, o);
        const uintptr_t bp = fa - lead + o;
        const uint32_t b_lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(bp));
        const uint32_t b_hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(bp >> 32));
        const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
            reinterpret_cast<void*>((uintptr_t(b_hi) << 32) | b_lo), (short)0, static_cast<int>(n), 0x00020000);
        const auto r = __builtin_amdgcn_raw_buffer_load_b128(rb, voff[k], 0, 0);
        return make_uint4(r[0], r[1], r[2], r[3]);
    };

    int32_t acc[M][3];
#pragma unroll
    for (int s = 0; s < M; ++s) acc[s][0] = acc[s][1] = acc[s][2] = 0;

    const int y0 = ys[i0];
    const int y1 = close_row[i1 - 1] + 1;
    int base = i0;
    while (base > 0 && close_row[base - 1] >= y0) --base;
    int slot = base % M;
    int next_close = close_row[base];
    int after_close = close_row[base + 1];   // read one ahead (the table ends in two sentinels)

    // rows i - 3 .. i of the band leave the stage as dwords
    // the item's output offset and height, held in scalar registers (as
    // constant-memory loads the compiler would re-read them at every flush)
    int64_t it_row_off = it->row_off;
    int it_h = it->h;
    asm volatile("" : "+s"(it_row_off), "+s"(it_h));
    auto flush = [&](int i) __attribute__((always_inline)) {
        const int nd = 3 * nbw / 4;   // dwords per band row (nbw is a multiple of 4)
        uint8_t* const ob = out + it_row_off + ((int64_t(u_k) * it_h + (i - 3)) * w + j0) * 3;
        for (int e = lane; e < 4 * nd; e += 64) {
            const int r = e / nd;
            const int d = e - r * nd;
            const uint32_t v = *reinterpret_cast<const uint32_t*>(stage + r * kStageRow + 4 * d);
            __builtin_nontemporal_store(v, reinterpret_cast<uint32_t*>(ob + int64_t(r) * w * 3 + 4 * d));
        }
    };

    auto process_row = [&](int y, uint4 cur, uint32_t s8, const int32_t (&wr)[M]) __attribute__((always_inline)) {
        // the lane's 12 bytes from its byte offset: r0 g0 b0 r1 | g1 b1 r2 g2 | b2 r3 g3 b3
        const uint32_t a0 = __builtin_amdgcn_alignbyte(cur.y, cur.x, s8);
        const uint32_t a1 = __builtin_amdgcn_alignbyte(cur.z, cur.y, s8);
        const uint32_t a2 = __builtin_amdgcn_alignbyte(cur.w, cur.z, s8);
        // per channel the four bytes in pixel order, then offset to signed
        const uint32_t rr = __builtin_amdgcn_perm(a2, __builtin_amdgcn_perm(a1, a0, 0x00060300u), 0x05020100u);
        const uint32_t gg = __builtin_amdgcn_perm(a2, __builtin_amdgcn_perm(a1, a0, 0x00070401u), 0x06020100u);
        const uint32_t bb = __builtin_amdgcn_perm(__builtin_amdgcn_perm(a2, a1, 0x07040100u), a0, 0x07060502u);
        plane[lane] = rr ^ 0x80808080u;
        plane[kPlane / 4 + lane] = gg ^ 0x80808080u;
        plane[2 * kPlane / 4 + lane] = bb ^ 0x80808080u;
        wave_lds_fence();
        // horizontal pass, rounded to bytes: digit by digit, each sum
        // starting from the previous one times 2^8 (idle lanes have zero
        // weights and start value, and form 0)
        int32_t h[3];
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            const uint32_t* pw = plane + c * (kPlane / 4) + sw;
            int32_t v[G];
#pragma unroll
            for (int g = 0; g < G; ++g) v[g] = static_cast<int32_t>(pw[g]);
            int32_t sum = 0;
#pragma unroll
            for (int g = 0; g < G; ++g) sum = __builtin_amdgcn_sdot4(dg[2][g], v[g], sum, false);
            sum = static_cast<int32_t>(static_cast<uint32_t>(sum) << 8);
#pragma unroll
            for (int g = 0; g < G; ++g) sum = __builtin_amdgcn_sdot4(dg[1][g], v[g], sum, false);
            sum = static_cast<int32_t>((static_cast<uint32_t>(sum) << 8) + static_cast<uint32_t>(c0));
#pragma unroll
            for (int g = 0; g < G; ++g) sum = __builtin_amdgcn_sdot4(dg[0][g], v[g], sum, false);
            h[c] = min(max(sum >> 22, 0), 255);
        }
        wave_lds_fence();
        // vertical pass: every open slot takes this row with its weight
#pragma unroll
        for (int s = 0; s < M; ++s) {
            const int32_t ws = wr[s];
#pragma unroll
            for (int c = 0; c < 3; ++c) acc[s][c] += __mul24(ws, h[c]);
        }
        while (y == next_close && base < i1) {   // wave-uniform
            const bool keep = base >= i0;
#pragma unroll
            for (int s = 0; s < M; ++s) {
                if (slot == s) {
                    if (keep && xlane) {
                        uint8_t* st = stage + (base & 3) * kStageRow + 3 * lane;
#pragma unroll
                        for (int c = 0; c < 3; ++c)
                            st[c] = static_cast<uint8_t>(min(max((acc[s][c] + (1 << 21)) >> 22, 0), 255));
                    }
                    acc[s][0] = acc[s][1] = acc[s][2] = 0;
                }
            }
            if (keep && (base & 3) == 3) {
                wave_lds_fence();
                flush(base);
                wave_lds_fence();
            }
            ++base;
            slot = slot + 1 == M ? 0 : slot + 1;
            next_close = after_close;
            after_close = close_row[base + 1];
        }
    };

    const int yb0 = y0 & ~3;
    uint4 pf[kPrefetch];
#pragma unroll
    for (int k = 0; k < kPrefetch; ++k) {
        pf[k] = load_row(yb0, k);
        __builtin_amdgcn_sched_barrier(0);
    }
    for (int yb = yb0; yb < y1; yb += kPrefetch) {
        // the block's slot weights, read together (a block starts below H,
        // and the table has kSlotMax rows past the frame's last)
        const cptr<int32_t> wblk = slot_q + yb * kSlotWords;
        int32_t wk[kPrefetch][M];
#pragma unroll
        for (int k = 0; k < kPrefetch; ++k)
#pragma unroll
            for (int s = 0; s < M; ++s) wk[k][s] = wblk[k * kSlotWords + s];
#pragma unroll
        for (int k = 0; k < kPrefetch; ++k) {
            const int y = yb + k;
            const uint4 cur = pf[k];
            pf[k] = load_row(yb + kPrefetch, k);
            if (y >= y0 && y < y1) process_row(y, cur, sh[k], wk[k]);
        }
    }
}

// The uint8 writer's MFMA form, for x axes whose 16-column blocks read at
// most 64 source pixels (downscales up to about 3x).  One single-wave
// workgroup per (frame, band of output rows, band of 64 output columns), as
// above, but source rows go in chunks of 16:
//   * horizontal pass, per block of 16 columns and per channel: lane l loads
//     its own 16 pixels of source row (chunk + l % 16) from the block's
//     window (16 (l / 16) .. +15), de-interleaves them into one channel's
//     signed bytes (value - 128): the A operand of v_mfma_i32_16x16x64_i8
//     (rows x window taps); the B operands are the block's weight digits
//     (taps x columns), held in registers.  Three products, one per digit,
//     from zero, zero and the start value, give the sums exactly (each stays
//     below 2^30); they are combined, rounded to bytes and packed four rows
//     per dword into LDS, [channel][column][16 rows];
//   * vertical pass: lane j reads its column's 16 bytes per channel and
//     adds the chunk's rows into the M rotating slots as before.
template <int M>
__global__ __launch_bounds__(64) void resize_mfma_kernel(PlanView plan, int wg0, uint8_t* out) {
    using v4i = int __attribute__((ext_vector_type(4)));
    constexpr int kStageRow = 3 * 64;
    extern __shared__ __align__(16) unsigned char smem[];

    const int lane = threadIdx.x;
    const uint32_t wg = as_const(plan.wgs)[wg0 + static_cast<int>(blockIdx.x)];
    if (wg == kNoWork) return;
    const int u = static_cast<int>(wg & kWgUnitMask);
    const int wave = static_cast<int>(wg >> kWgBandShift);
    const cptr<StreamUnit> up = as_const(plan.units) + u;
    const int u_item = up->item, u_k = up->p_flags, i0 = up->i0, i1 = up->i1;
    const cptr<DevItem> it = as_const(plan.items) + u_item;

    const int w = it->w;
    const int j0 = wave * 64;
    const int nbw = min(64, w - j0);
    const bool xlane = lane < nbw;

    uint8_t* hbuf = smem;                         // [3][64 columns][16 rows]
    uint8_t* stage = smem + 3 * 64 * 16;          // [4][kStageRow]

    const cptr<int32_t> tables = as_const(plan.tables);
    const cptr<int32_t> band_tab = tables + it->sx_off + wave * kRsMfmaBandWords;
    const cptr<int32_t> cterm = tables + it->sx_off + ((w + 63) / 64) * kRsMfmaBandWords;
    // B operands (weight digits) and start values of the lane's columns
    v4i wt[4][3];
    int32_t cb[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
#pragma unroll
        for (int d = 0; d < 3; ++d) {
            const cptr<int32_t> src = band_tab + 4 + ((b * 3 + d) * 64 + lane) * 4;
            wt[b][d] = v4i{src[0], src[1], src[2], src[3]};
        }
        const int j = j0 + 16 * b + (lane & 15);
        cb[b] = j < w ? cterm[j] : 0;
    }
    const cptr<int32_t> ys = tables + it->ty_off;
    const cptr<int32_t> slot_q = tables + it->sy_off;
    const cptr<int32_t> close_row = tables + it->sy_off + (it->H + kSlotMax) * kSlotWords;

    // the frame through one buffer resource (loads past it return zeros)
    const int f = as_const(plan.indices)[it->idx_off + u_k];
    const uintptr_t fa = reinterpret_cast<uintptr_t>(it->frames + int64_t(f) * it->frame_bytes);
    const uint32_t lead = static_cast<uint32_t>(fa & 3u);
    const uint32_t range = static_cast<uint32_t>((it->frame_bytes + lead + 3) & ~int64_t(3));
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(fa - lead), (short)0, static_cast<int>(range), 0x00020000);
    const uint32_t row_bytes = static_cast<uint32_t>(it->W) * 3u;

    int32_t acc[M][3];
#pragma unroll
    for (int s = 0; s < M; ++s) acc[s][0] = acc[s][1] = acc[s][2] = 0;
    const int y0 = ys[i0];
    const int y1 = close_row[i1 - 1] + 1;
    int base = i0;
    while (base > 0 && close_row[base - 1] >= y0) --base;
    int slot = base % M;
    int next_close = close_row[base];
    int after_close = close_row[base + 1];   // read one ahead (the table ends in two sentinels)

    // the item's output offset and height, held in scalar registers (as
    // constant-memory loads the compiler would re-read them at every flush)
    int64_t it_row_off = it->row_off;
    int it_h = it->h;
    asm volatile("" : "+s"(it_row_off), "+s"(it_h));
    auto flush = [&](int i) __attribute__((always_inline)) {
        const int nd = 3 * nbw / 4;
        uint8_t* const ob = out + it_row_off + ((int64_t(u_k) * it_h + (i - 3)) * w + j0) * 3;
        for (int e = lane; e < 4 * nd; e += 64) {
            const int r = e / nd;
            const int d = e - r * nd;
            const uint32_t v = *reinterpret_cast<const uint32_t*>(stage + r * kStageRow + 4 * d);
            __builtin_nontemporal_store(v, reinterpret_cast<uint32_t*>(ob + int64_t(r) * w * 3 + 4 * d));
        }
    };

    const int g = lane >> 4;          // k group of the lane: window taps 16 g .. 16 g + 15
    for (int yc = y0 & ~15; yc < y1; yc += 16) {
        // ---- horizontal pass of source rows yc .. yc + 15
        const uint32_t rowoff = lead + static_cast<uint32_t>(yc + (lane & 15)) * row_bytes;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const uint32_t o = rowoff + 3u * static_cast<uint32_t>(band_tab[b] + 16 * g);
            const uint32_t oa = o & ~3u;
            const uint32_t sh = o & 3u;
            const auto l0 = __builtin_amdgcn_raw_buffer_load_b128(rsrc, oa, 0, 0);
            const auto l1 = __builtin_amdgcn_raw_buffer_load_b128(rsrc, oa + 16, 0, 0);
            const auto l2 = __builtin_amdgcn_raw_buffer_load_b128(rsrc, oa + 32, 0, 0);
            const uint32_t l3 = __builtin_amdgcn_raw_buffer_load_b32(rsrc, oa + 48, 0, 0);
            const uint32_t raw[13] = {l0[0], l0[1], l0[2], l0[3], l1[0], l1[1], l1[2], l1[3],
                                      l2[0], l2[1], l2[2], l2[3], l3};
            uint32_t a[12];
#pragma unroll
            for (int q = 0; q < 12; ++q) a[q] = __builtin_amdgcn_alignbyte(raw[q + 1], raw[q], sh);
            // channel planes of the lane's 16 pixels, as signed bytes
            v4i pc[3];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t x0w = a[3 * k], x1w = a[3 * k + 1], x2w = a[3 * k + 2];
                pc[0][k] = static_cast<int>(__builtin_amdgcn_perm(x2w, __builtin_amdgcn_perm(x1w, x0w, 0x00060300u), 0x05020100u) ^ 0x80808080u);
                pc[1][k] = static_cast<int>(__builtin_amdgcn_perm(x2w, __builtin_amdgcn_perm(x1w, x0w, 0x00070401u), 0x06020100u) ^ 0x80808080u);
                pc[2][k] = static_cast<int>(__builtin_amdgcn_perm(__builtin_amdgcn_perm(x2w, x1w, 0x07040100u), x0w, 0x07060502u) ^ 0x80808080u);
            }
#pragma unroll
            for (int c = 0; c < 3; ++c) {
                const v4i zero = {0, 0, 0, 0};
                const v4i cs = {cb[b], cb[b], cb[b], cb[b]};
                const v4i s2 = __builtin_amdgcn_mfma_i32_16x16x64_i8(pc[c], wt[b][0], zero, 0, 0, 0);
                const v4i s1 = __builtin_amdgcn_mfma_i32_16x16x64_i8(pc[c], wt[b][1], zero, 0, 0, 0);
                const v4i s0 = __builtin_amdgcn_mfma_i32_16x16x64_i8(pc[c], wt[b][2], cs, 0, 0, 0);
                // D[row 4 g + r][column l % 16]: rows 4g .. 4g + 3 of the lane's column
                uint32_t hb[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const uint32_t sum = (static_cast<uint32_t>(s2[r]) << 16) + (static_cast<uint32_t>(s1[r]) << 8) +
                                         static_cast<uint32_t>(s0[r]);
                    hb[r] = static_cast<uint32_t>(min(max(static_cast<int32_t>(sum) >> 22, 0), 255));
                }
                // packed with v_perm: left to itself the compiler fuses two of
                // the clamps with the packing into a 16-bit v_ashr_pk_u8_i32 and
                // ORs the other two bytes over its undefined upper half
                const uint32_t packed = __builtin_amdgcn_perm(hb[1], hb[0], 0x0C0C0400u) |
                                        __builtin_amdgcn_perm(hb[3], hb[2], 0x04000C0Cu);
                *reinterpret_cast<uint32_t*>(hbuf + c * 1024 + (16 * b + (lane & 15)) * 16 + 4 * g) = packed;
            }
        }
        wave_lds_fence();
        // ---- vertical pass over the chunk's rows
        uint4 hv[3];
#pragma unroll
        for (int c = 0; c < 3; ++c) hv[c] = *reinterpret_cast<const uint4*>(hbuf + c * 1024 + lane * 16);
        wave_lds_fence();
        const cptr<int32_t> wblk = slot_q + yc * kSlotWords;
        int32_t wk[4][M];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int y = yc + r;
            if ((r & 3) == 0 && y < y1) {
                // the next four rows' slot weights, read together (y < y1 <= H,
                // and the table has kSlotMax rows past the frame's last)
#pragma unroll
                for (int k = 0; k < 4; ++k)
#pragma unroll
                    for (int s = 0; s < M; ++s) wk[k][s] = wblk[(r + k) * kSlotWords + s];
            }
            if (y < y0 || y >= y1) continue;   // wave-uniform
            const uint32_t dw = r >> 2;
            const uint32_t sel = 8u * static_cast<uint32_t>(r & 3);
            int32_t h[3];
#pragma unroll
            for (int c = 0; c < 3; ++c) {
                const uint32_t word = dw == 0 ? hv[c].x : dw == 1 ? hv[c].y : dw == 2 ? hv[c].z : hv[c].w;
                h[c] = static_cast<int32_t>(__builtin_amdgcn_ubfe(word, sel, 8));
            }
#pragma unroll
            for (int s = 0; s < M; ++s) {
                const int32_t ws = wk[r & 3][s];
#pragma unroll
                for (int c = 0; c < 3; ++c) acc[s][c] += __mul24(ws, h[c]);
            }
            while (y == next_close && base < i1) {   // wave-uniform
                const bool keep = base >= i0;
#pragma unroll
                for (int s = 0; s < M; ++s) {
                    if (slot == s) {
                        if (keep && xlane) {
                            uint8_t* st = stage + (base & 3) * kStageRow + 3 * lane;
#pragma unroll
                            for (int c = 0; c < 3; ++c)
                                st[c] = static_cast<uint8_t>(min(max((acc[s][c] + (1 << 21)) >> 22, 0), 255));
                        }
                        acc[s][0] = acc[s][1] = acc[s][2] = 0;
                    }
                }
                if (keep && (base & 3) == 3) {
                    wave_lds_fence();
                    flush(base);
                    wave_lds_fence();
                }
                ++base;
                slot = slot + 1 == M ? 0 : slot + 1;
                next_close = after_close;
                after_close = close_row[base + 1];
            }
        }
    }
}

template <int M>
int launch_resize_mfma_shape(const PlanView& plan, const StreamLaunch& L, void* out, hipStream_t stream) {
    hipLaunchKernelGGL((resize_mfma_kernel<M>), dim3(static_cast<unsigned>(L.count)), dim3(64),
                       resize_mfma_bytes(), stream, plan, L.first, static_cast<uint8_t*>(out));
    return static_cast<int>(hipGetLastError());
}

template <int M, int KX>
int launch_resize_stream_shape(const PlanView& plan, const StreamLaunch& L, void* out, hipStream_t stream) {
    hipLaunchKernelGGL((resize_stream_kernel<M, KX>), dim3(static_cast<unsigned>(L.count)), dim3(64),
                       resize_stream_bytes(), stream, plan, L.first, static_cast<uint8_t*>(out));
    return static_cast<int>(hipGetLastError());
}

// One streaming shape of this part: its launch, or -1 if the launch is not
// of this shape or the shape belongs to another part.
template <int MM, int KK, int PP, int ID>
int stream_case(const PlanView& plan, const StreamLaunch& L, void* out, int out_dtype,
                const Norm& norm, hipStream_t stream) {
    if constexpr (ID % VP_PARTS == VP_PART) {
        if (L.m == MM && L.kx == KK && L.px == PP)
            return launch_stream_shape<MM, KK, PP>(plan, L, out, out_dtype, norm, stream);
    }
    return -1;
}

template <int MM, int KK, int DB, int ID>
int xfirst_case(const PlanView& plan, const StreamLaunch& L, void* out, int out_dtype,
                const Norm& norm, hipStream_t stream) {
    if constexpr (ID % VP_PARTS == VP_PART) {
        if (L.m == MM && L.kx == KK && L.px == xfirst_px(DB))
            return launch_xfirst_shape<MM, KK, DB>(plan, L, out, out_dtype, norm, stream);
    }
    return -1;
}

template <int MM, int KK, int ID>
int resize_case(const PlanView& plan, const StreamLaunch& L, void* out, hipStream_t stream) {
    if constexpr (ID % VP_PARTS == VP_PART) {
        if (L.m == MM && L.kx == KK) {
            if constexpr (KK == kRsMfmaWindow)
                return launch_resize_mfma_shape<MM>(plan, L, out, stream);
            else
                return launch_resize_stream_shape<MM, KK>(plan, L, out, stream);
        }
    }
    return -1;
}

}  // namespace

// This part's streaming shapes (-1: the launch's shape is not one of them).
int VP_CAT(launch_stream_part, VP_PART)(const PlanView& plan, const StreamLaunch& L, void* out,
                                        int out_dtype, const Norm& norm, hipStream_t stream) {
#define VP_STREAM_CASE(MM, KK, PP)                                                               \
    if (const int r = stream_case<MM, KK, PP, __COUNTER__>(plan, L, out, out_dtype, norm, stream); \
        r != -1)                                                                                 \
        return r;
#define VP_STREAM_KX(MM, PP) \
    VP_STREAM_CASE(MM, 4, PP) VP_STREAM_CASE(MM, 5, PP) VP_STREAM_CASE(MM, 6, PP) VP_STREAM_CASE(MM, 7, PP) \
    VP_STREAM_CASE(MM, 8, PP) VP_STREAM_CASE(MM, 9, PP) VP_STREAM_CASE(MM, 10, PP) VP_STREAM_CASE(MM, 11, PP) \
    VP_STREAM_CASE(MM, 12, PP) VP_STREAM_CASE(MM, 13, PP) VP_STREAM_CASE(MM, 14, PP) VP_STREAM_CASE(MM, 15, PP) \
    VP_STREAM_CASE(MM, 16, PP)
    VP_STREAM_KX(4, 2) VP_STREAM_KX(5, 2) VP_STREAM_KX(6, 2)
    VP_STREAM_KX(4, 3) VP_STREAM_KX(5, 3)
    VP_STREAM_CASE(7, 4, 2) VP_STREAM_CASE(7, 5, 2) VP_STREAM_CASE(7, 6, 2) VP_STREAM_CASE(7, 7, 2) VP_STREAM_CASE(7, 8, 2)
    VP_STREAM_CASE(8, 4, 2) VP_STREAM_CASE(8, 5, 2) VP_STREAM_CASE(8, 6, 2) VP_STREAM_CASE(8, 7, 2) VP_STREAM_CASE(8, 8, 2)
#define VP_STREAM_LONG(MM, PP) \
    VP_STREAM_CASE(MM, 20, PP) VP_STREAM_CASE(MM, 24, PP) VP_STREAM_CASE(MM, 28, PP) VP_STREAM_CASE(MM, 32, PP)
    VP_STREAM_LONG(4, 2) VP_STREAM_LONG(5, 2) VP_STREAM_LONG(6, 2)
    VP_STREAM_CASE(4, 20, 3) VP_STREAM_CASE(4, 24, 3) VP_STREAM_CASE(5, 20, 3) VP_STREAM_CASE(5, 24, 3)
#undef VP_STREAM_LONG
#undef VP_STREAM_KX
#undef VP_STREAM_CASE
#define VP_XF_CASE(MM, KK, DB)                                                                    \
    if (const int r = xfirst_case<MM, KK, DB, __COUNTER__>(plan, L, out, out_dtype, norm, stream); \
        r != -1)                                                                                 \
        return r;
#define VP_XF_KX(MM) VP_XF_CASE(MM, 4, 0) VP_XF_CASE(MM, 5, 0) VP_XF_CASE(MM, 6, 0) VP_XF_CASE(MM, 7, 0) \
    VP_XF_CASE(MM, 8, 0) VP_XF_CASE(MM, 9, 0) VP_XF_CASE(MM, 10, 0) VP_XF_CASE(MM, 11, 0) VP_XF_CASE(MM, 12, 0)
#define VP_XF_PAIR(MM, DB) VP_XF_CASE(MM, 6, DB) VP_XF_CASE(MM, 7, DB) VP_XF_CASE(MM, 8, DB)
    VP_XF_KX(4) VP_XF_KX(5) VP_XF_KX(6) VP_XF_KX(7) VP_XF_KX(8)
    VP_XF_PAIR(4, 2) VP_XF_PAIR(5, 2) VP_XF_PAIR(6, 2) VP_XF_PAIR(7, 2) VP_XF_PAIR(8, 2)
#undef VP_XF_PAIR
#undef VP_XF_KX
#undef VP_XF_CASE
    return -1;
}

int VP_CAT(launch_resize_stream_part, VP_PART)(const PlanView& plan, const StreamLaunch& L, void* out,
                                               hipStream_t stream) {
#define VP_RS_CASE(MM, KK) \
    if (const int r = resize_case<MM, KK, __COUNTER__>(plan, L, out, stream); r != -1) return r;
#define VP_RS_KX(MM) VP_RS_CASE(MM, 8) VP_RS_CASE(MM, 12) VP_RS_CASE(MM, 16) VP_RS_CASE(MM, 20) \
    VP_RS_CASE(MM, 24) VP_RS_CASE(MM, 28) VP_RS_CASE(MM, 32) VP_RS_CASE(MM, kRsMfmaWindow)
    VP_RS_KX(4) VP_RS_KX(5) VP_RS_KX(6) VP_RS_KX(7) VP_RS_KX(8)
#undef VP_RS_KX
#undef VP_RS_CASE
    return -1;
}

#if VP_PART == 0

// Every part's dispatchers (parts 1 .. VP_PARTS - 1 are other translation units).
#define VP_DECLARE_PART(n)                                                                          \
    int launch_stream_part##n(const PlanView&, const StreamLaunch&, void*, int, const Norm&, hipStream_t); \
    int launch_resize_stream_part##n(const PlanView&, const StreamLaunch&, void*, hipStream_t);
VP_DECLARE_PART(0) VP_DECLARE_PART(1) VP_DECLARE_PART(2) VP_DECLARE_PART(3)
VP_DECLARE_PART(4) VP_DECLARE_PART(5) VP_DECLARE_PART(6) VP_DECLARE_PART(7)
#undef VP_DECLARE_PART

namespace {
using StreamPartFn = int (*)(const PlanView&, const StreamLaunch&, void*, int, const Norm&, hipStream_t);
using ResizePartFn = int (*)(const PlanView&, const StreamLaunch&, void*, hipStream_t);
const StreamPartFn kStreamParts[VP_PARTS] = {
    launch_stream_part0,
#if VP_PARTS > 1
    launch_stream_part1,
#endif
#if VP_PARTS > 2
    launch_stream_part2,
#endif
#if VP_PARTS > 3
    launch_stream_part3,
#endif
#if VP_PARTS > 4
    launch_stream_part4,
#endif
#if VP_PARTS > 5
    launch_stream_part5,
#endif
#if VP_PARTS > 6
    launch_stream_part6,
#endif
#if VP_PARTS > 7
    launch_stream_part7,
#endif
};
const ResizePartFn kResizeParts[VP_PARTS] = {
    launch_resize_stream_part0,
#if VP_PARTS > 1
    launch_resize_stream_part1,
#endif
#if VP_PARTS > 2
    launch_resize_stream_part2,
#endif
#if VP_PARTS > 3
    launch_resize_stream_part3,
#endif
#if VP_PARTS > 4
    launch_resize_stream_part4,
#endif
#if VP_PARTS > 5
    launch_resize_stream_part5,
#endif
#if VP_PARTS > 6
    launch_resize_stream_part6,
#endif
#if VP_PARTS > 7
    launch_resize_stream_part7,
#endif
};
}  // namespace

// The plan memory of vp_preprocess_batch_noalloc: a file-scope device
// array, so that a caller that cannot allocate device memory needs no
// workspace.  Every device the library runs on holds its own copy until the
// process ends.  In host code the array's name is not a device address: the
// address of the current device's copy is looked up with
// hipGetSymbolAddress, once per device, and only that address is used.
__device__ __align__(256) unsigned char scratch[kNoAllocPlanBytes];

int noalloc_plan_memory(void** ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return static_cast<int>(e);
    static std::mutex mu;
    static std::map<int, void*> by_device;
    std::lock_guard<std::mutex> lk(mu);
    auto it = by_device.find(dev);
    if (it == by_device.end()) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return static_cast<int>(e);
        it = by_device.emplace(dev, p).first;
    }
    *ptr = it->second;
    return 0;
}

int launch_positions(const PlanView& plan, int32_t* vit, int32_t* llm, int64_t rows,
                     hipStream_t stream) {
    if (rows <= 0 || (vit == nullptr && llm == nullptr)) return 0;
    const int64_t blocks = std::min<int64_t>((rows + 255) / 256, 65536);
    hipLaunchKernelGGL(positions_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, plan,
                       vit, llm, rows);
    return static_cast<int>(hipGetLastError());
}

int launch_resize(const PlanView& plan, void* out, hipStream_t stream) {
    if (plan.n_tiles <= 0) return 0;
    hipLaunchKernelGGL(resize_u8_kernel, dim3(plan.n_tiles), dim3(kRsThreads), 0, stream, plan,
                       static_cast<uint8_t*>(out));
    return static_cast<int>(hipGetLastError());
}

bool resize_stream_supported(int m, int kx, int px) {
    return m >= 4 && m <= kSlotWords && kx >= 8 && kx <= 32 && kx % 4 == 0 && px == kRsPx;
}

int launch_resize_stream(const PlanView& plan, const StreamLaunch& L, void* out, hipStream_t stream) {
    if (L.count <= 0) return 0;
    if (L.kx == kRsMfmaWindow ? (L.px != kRsPx || L.m < 4 || L.m > kSlotWords)
                              : !resize_stream_supported(L.m, L.kx, L.px))
        return static_cast<int>(hipErrorInvalidConfiguration);
    for (const ResizePartFn part : kResizeParts)
        if (const int r = part(plan, L, out, stream); r != -1) return r;
    return static_cast<int>(hipErrorInvalidConfiguration);
}

int launch_patchify(const PlanView& plan, void* out, int out_dtype, const Norm& norm, int patch,
                    hipStream_t stream) {
    if (plan.n_tiles <= 0) return 0;
    dim3 grid(plan.n_tiles), block(256);
    if (patch == 14) {
        if (out_dtype == 1)
            hipLaunchKernelGGL(patchify14_kernel<1>, grid, block, 0, stream, plan, out, norm);
        else
            hipLaunchKernelGGL(patchify14_kernel<0>, grid, block, 0, stream, plan, out, norm);
    } else if (out_dtype == 1) {
        hipLaunchKernelGGL(patchify_kernel<1>, grid, block, 0, stream, plan, out, norm);
    } else {
        hipLaunchKernelGGL(patchify_kernel<0>, grid, block, 0, stream, plan, out, norm);
    }
    return static_cast<int>(hipGetLastError());
}

int launch_generic(const PlanView& plan, void* out, int out_dtype, const Norm& norm,
                   hipStream_t stream) {
    if (plan.n_tiles <= 0) return 0;
    dim3 grid(plan.n_tiles), block(kGenericThreads);
    if (out_dtype == 1)
        hipLaunchKernelGGL(generic_tile_kernel<1>, grid, block, 0, stream, plan, out, norm);
    else
        hipLaunchKernelGGL(generic_tile_kernel<0>, grid, block, 0, stream, plan, out, norm);
    return static_cast<int>(hipGetLastError());
}

// Compiled shapes: every (M, KX) with 2 pixels per lane, and with 3 pixels
// per lane where the accumulators still fit the registers of a 1024-thread
// block (M <= 5).  KX is any tap count from 4 to 16, and a multiple of 4 beyond.
bool stream_shape_supported(int m, int kx, int px) {
    if (m < 4 || kx < 4 || kx > 32 || (kx > 16 && kx % 4 != 0)) return false;
    if (m > 6)   // 7 or 8 open rows: vertical upscales up to about 2x, whose x axis has short windows too
        return m <= kSlotWords && px == 2 && kx <= 8;
    if (kx <= 16) return px == 2 || (px == 3 && m <= 5);
    // windows of 17 to 32 taps: x downscales of about 3.75x to 7.5x
    return px == 2 || (px == 3 && m <= 5 && kx <= 24);
}

bool xfirst_shape_supported(int m, int kx, int db) {
    return m >= 4 && m <= kSlotWords && kx >= 4 && (db == 0 ? kx <= 12 : db == 2 && kx >= 6 && kx <= 8);
}

int launch_stream(const PlanView& plan, const StreamLaunch& L, void* out, int out_dtype,
                  const Norm& norm, hipStream_t stream) {
    if (L.count <= 0) return 0;
    if (L.px < 0 ? (L.px < xfirst_px(2) || !xfirst_shape_supported(L.m, L.kx, xfirst_db(L.px)) || L.patch != 16)
                 : (!stream_shape_supported(L.m, L.kx, L.px) ||
                    stream_wave_bytes(L.px, L.kx, 4, L.patch) > kStreamLdsBudget))
        return static_cast<int>(hipErrorInvalidConfiguration);
    for (const StreamPartFn part : kStreamParts)
        if (const int r = part(plan, L, out, out_dtype, norm, stream); r != -1) return r;
    return static_cast<int>(hipErrorInvalidValue);
}

#endif  // VP_PART == 0

}  // namespace vp
