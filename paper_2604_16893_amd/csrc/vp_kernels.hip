// vp_kernels.hip -- gfx950 kernels of the preprocessing path.
//
// Two kernels compute the same result (the resampled, normalised,
// merge-window rows of Section 3.1.1 of arXiv 2604.16893, laid out per the
// grid the host reports); the host routes each item to one of them.
//
// Streaming kernel (the fast path; items whose frames are not upscaled
// vertically and whose filters are short enough).  One workgroup streams
// one source frame -- or a band of its output rows -- top to bottom:
//   * y pass first, in registers: each lane owns 12 bytes (4 RGB pixels) of
//     every source row, loads them with one buffer load (prefetched four rows
//     ahead), converts them once, and adds them with wave-uniform scalar
//     weights into M rotating accumulators -- one per output row that can
//     still read the current source row.  The source is read exactly once.
//   * when an output row is complete its accumulator is written to a
//     double-buffered LDS row (one float4 per pixel) and the workgroup
//     barrier hands it to the x pass: one lane per output pixel, its column
//     weights in registers, one ds_read_b128 and three FMAs per tap, then
//     the normalisation FMA and the bf16/f32 conversion into an LDS stage.
//   * every four output rows the stage holds one 64-value run (four patch
//     rows of 16) of every (patch, channel) block; those leave as 16-byte
//     stores that fill whole 128-byte lines.
//
// General kernel (any scale factor): one workgroup per merge window of one
// frame pair; y pass from global memory into an LDS column tile, x pass,
// staging of the four rows in output order, 16-byte stores.  When the
// horizontal window of 32 output columns does not fit the tile, the host
// splits the window into rh x cw sub-tiles.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "vp_plan.h"

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
    __shared__ float stage[kWinElems];     // the unit's four output rows, output order

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

    for (int dt = 0; dt < 2; ++dt) {
        const int f = plan.indices[it.idx_off + 2 * tt + dt];
        const uint8_t* frame = it.frames + int64_t(f) * it.frame_bytes;
        for (int r0 = 0; r0 < kWin; r0 += it.rh) {
            for (int c0 = 0; c0 < kWin; c0 += it.cw) {
                const int i0 = kWin * bh + r0;
                const int j0 = kWin * bw + c0;
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
                    const float v = fmaf(acc, norm.a[c], norm.b[c]);
                    const int il = r0 + r, jl = c0 + cc;
                    const int sub = (il >> 4) * 2 + (jl >> 4);
                    stage[sub * kRow + ((c * 2 + dt) * kPatch + (il & 15)) * kPatch + (jl & 15)] = v;
                }
                __syncthreads();
            }
        }
    }

    const int64_t row0 = it.row_off + ((int64_t(tt) * it.hm + bh) * it.wm + bw) * 4;
    if (OUT_BF16) {
        uint4* dst = reinterpret_cast<uint4*>(static_cast<uint16_t*>(out) + row0 * kRow);
        for (int e = tid; e < kWinElems / 8; e += kGenericThreads) {
            const float* s = stage + e * 8;
            uint4 v;
            v.x = bf16_rne(s[0]) | (bf16_rne(s[1]) << 16);
            v.y = bf16_rne(s[2]) | (bf16_rne(s[3]) << 16);
            v.z = bf16_rne(s[4]) | (bf16_rne(s[5]) << 16);
            v.w = bf16_rne(s[6]) | (bf16_rne(s[7]) << 16);
            dst[e] = v;
        }
    } else {
        float4* dst = reinterpret_cast<float4*>(static_cast<float*>(out) + row0 * kRow);
        for (int e = tid; e < kWinElems / 4; e += kGenericThreads)
            dst[e] = reinterpret_cast<const float4*>(stage)[e];
    }
}

// ===========================================================================
// Streaming kernel
// ===========================================================================

constexpr int kPrefetch = 4;           // source rows in flight per lane
constexpr int kStreamBlock = kStreamMaxThreads;

// Source row y adds to the n open output rows base .. base+n-1, which live in
// acc[0 .. n-1] (acc[0] is always the oldest open row, `base`).
template <int M>
__device__ __forceinline__ void add_row(float (&acc)[M][12], const float (&v)[12], cptr<float> w,
                                        int n) {
#pragma unroll
    for (int m = 0; m < M; ++m) {
        if (m < n) {
            const float wm = w[m];
#pragma unroll
            for (int q = 0; q < 12; ++q) acc[m][q] = fmaf(wm, v[q], acc[m][q]);
        }
    }
}

// Same, for a source row that completes output row `base`: its final value
// goes to `done`, and every other sum moves down one accumulator as it is
// formed (the FMA writes acc[m - 1]), so no register is ever copied.  The
// FMAs are unconditional: the table pads every row with zero weights, so an
// output row that does not read this source row just moves down unchanged
// (output rows not yet started hold zeros; rows past the band hold values
// that are never stored).
template <int M>
__device__ __forceinline__ void add_row_and_close(float (&acc)[M][12], const float (&v)[12],
                                                  cptr<float> w, float (&done)[12]) {
    const float w0 = w[0];
#pragma unroll
    for (int q = 0; q < 12; ++q) done[q] = fmaf(w0, v[q], acc[0][q]);
#pragma unroll
    for (int m = 1; m < M; ++m) {
        const float wm = w[m];
#pragma unroll
        for (int q = 0; q < 12; ++q) acc[m - 1][q] = fmaf(wm, v[q], acc[m][q]);
    }
#pragma unroll
    for (int q = 0; q < 12; ++q) acc[M - 1][q] = 0.f;
}

__device__ __forceinline__ void put_row(const float (&done)[12], float4* dst) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
        dst[q] = make_float4(done[3 * q], done[3 * q + 1], done[3 * q + 2], 0.f);
}

template <int M, int KX, int OUT_BF16>
__global__ __launch_bounds__(kStreamBlock) void stream_kernel(PlanView plan, int unit0, int ring_slots,
                                                              void* out, Norm norm) {
    using elem_t = typename std::conditional<OUT_BF16 != 0, uint16_t, float>::type;
    extern __shared__ __align__(16) unsigned char smem[];

    const cptr<StreamUnit> up = as_const(plan.units) + unit0 + blockIdx.x;
    const int u_item = up->item, u_p = up->p, u_rows = up->rows, u_flags = up->flags;
    const cptr<DevItem> it = as_const(plan.items) + u_item;
    const int t = threadIdx.x;
    const int nt = blockDim.x;
    const int i0 = u_rows & 0xffff;
    const int i1 = u_rows >> 16;
    const int w = it->w;
    const int tlen = it->tlen;
    const int n_strips = it->n_strips;
    const int tt = u_p >> 1;
    const int dt_self = u_p & 1;
    const bool both = (u_flags & 1) != 0;

    float4* ring = reinterpret_cast<float4*>(smem);                               // [slots][tlen]
    elem_t* stage = reinterpret_cast<elem_t*>(smem + size_t(ring_slots) * tlen * 16);  // [w/16][3][4][16]

    // LDS pixels that no lane writes stay zero (they meet zero weights only).
    for (int k = 4 * n_strips + t; k < tlen; k += nt) {
        ring[k] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (ring_slots > 1) ring[tlen + k] = make_float4(0.f, 0.f, 0.f, 0.f);
    }

    // x pass: output pixel j = t keeps its column weights in registers.
    const cptr<int32_t> tables = as_const(plan.tables);
    const cptr<int32_t> sx_start = tables + it->sx_off;
    const cptr<float> sx_w = (cptr<float>)(sx_start + w);
    float wx[KX];
    int sj = 0;
    if (t < w) {
        sj = sx_start[t];
        const cptr<float> src = sx_w + int64_t(t) * KX;
#pragma unroll
        for (int k = 0; k < KX; ++k) wx[k] = src[k];
    } else {
#pragma unroll
        for (int k = 0; k < KX; ++k) wx[k] = 0.f;
    }

    const cptr<int32_t> ys = tables + it->ty_off;
    const cptr<int32_t> scat = tables + it->sy_off;                 // [H + extra][8]
    const cptr<int32_t> close_row = scat + int64_t(it->H + kScatterMax) * kScatterWords;  // [h]

    // Source frame through a buffer resource: loads past the frame return 0.
    const int f = as_const(plan.indices)[it->idx_off + u_p];
    const uintptr_t fa = reinterpret_cast<uintptr_t>(it->frames + int64_t(f) * it->frame_bytes);
    const uint32_t lead = static_cast<uint32_t>(fa & 3u);
    // Range = the frame rounded up to whole dwords: the range check is per
    // dword, and the dword holding the frame's last byte lies in that byte's
    // (4-byte aligned) page, so it is always readable.
    const uint32_t range = static_cast<uint32_t>((it->frame_bytes + lead + 3) & ~int64_t(3));
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<void*>(fa - lead), (short)0, static_cast<int>(range), 0x00020000);
    const uint32_t row_bytes = static_cast<uint32_t>(it->W) * 3u;
    const bool vlane = t < n_strips;
    const uint32_t lane_off = lead + kStripBytes * static_cast<uint32_t>(t);

    const float a0 = norm.a[0], a1 = norm.a[1], a2 = norm.a[2];
    const float b0 = norm.b[0], b1 = norm.b[1], b2 = norm.b[2];

    float acc[M][12];
#pragma unroll
    for (int s = 0; s < M; ++s)
#pragma unroll
        for (int q = 0; q < 12; ++q) acc[s][q] = 0.f;

    int base = i0;        // oldest output row still accumulating, in acc[0]
    const int y0 = ys[i0];
    const int y1 = close_row[i1 - 1] + 1;   // past the frame: zero-weight rows, loads return 0

    auto load_row = [&](int y) __attribute__((always_inline)) -> uint4 {
        const uint32_t off = (lane_off + static_cast<uint32_t>(y) * row_bytes) & ~3u;
        const auto r = __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, 0);
        return make_uint4(r[0], r[1], r[2], r[3]);
    };

    // x pass of output row i, normalise, stage; every 4th row: store.
    auto x_pass = [&](int i) __attribute__((always_inline)) {
        const float4* row = ring + (ring_slots > 1 ? (i & 1) : 0) * tlen;
        const int yy = i & 3;
        for (int j = t; j < w; j += nt) {
            float r0 = 0.f, r1 = 0.f, r2 = 0.f;
            if (j == t) {
                const float4* src = row + sj;
#pragma unroll
                for (int g = 0; g < KX; g += 4) {
                    // four taps at a time: bounds the LDS values held in registers
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int k = g; k < g + 4; ++k) {
                        const float4 q = src[k];
                        r0 = fmaf(wx[k], q.x, r0);
                        r1 = fmaf(wx[k], q.y, r1);
                        r2 = fmaf(wx[k], q.z, r2);
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            } else {   // more outputs than lanes: weights from the table
                const float4* src = row + sx_start[j];
                const cptr<float> wj = sx_w + int64_t(j) * KX;
#pragma unroll
                for (int k = 0; k < KX; ++k) {
                    const float4 q = src[k];
                    const float wk = wj[k];
                    r0 = fmaf(wk, q.x, r0);
                    r1 = fmaf(wk, q.y, r1);
                    r2 = fmaf(wk, q.z, r2);
                }
            }
            const float v0 = fmaf(r0, a0, b0);
            const float v1 = fmaf(r1, a1, b1);
            const float v2 = fmaf(r2, a2, b2);
            const int e = ((j >> 4) * 3 * 4 + yy) * 16 + (j & 15);
            if constexpr (OUT_BF16 != 0) {
                stage[e] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v0));
                stage[e + 64] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v1));
                stage[e + 128] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v2));
            } else {
                stage[e] = v0;
                stage[e + 64] = v1;
                stage[e + 128] = v2;
            }
        }
        if (yy == 3) {
            __syncthreads();
            // rows i-3 .. i hold one 64-value run of every (patch column, channel) block
            constexpr int kChunks = OUT_BF16 ? 8 : 16;   // 16-byte pieces per run
            const int yq = (i & 15) >> 2;
            const int bh = i >> 5;
            const int mh = (i >> 4) & 1;
            const int n_runs = (w >> 4) * 3;
            const int64_t win_row0 = it->row_off + (int64_t(tt) * it->hm + bh) * it->wm * 4 + mh * 2;
            const uint4* st4 = reinterpret_cast<const uint4*>(stage);
            for (int e = t; e < n_runs * kChunks; e += nt) {
                const int run = e / kChunks;
                const int piece = e - run * kChunks;
                const int pj = run / 3;
                const int c = run - pj * 3;
                const int64_t rho = win_row0 + (pj >> 1) * 4 + (pj & 1);
                const uint4 val = st4[e];
                elem_t* dst = static_cast<elem_t*>(out) + rho * kRow + yq * 64;
                if (both) {
                    reinterpret_cast<uint4*>(dst + (c * 2) * 256)[piece] = val;
                    reinterpret_cast<uint4*>(dst + (c * 2 + 1) * 256)[piece] = val;
                } else {
                    reinterpret_cast<uint4*>(dst + (c * 2 + dt_self) * 256)[piece] = val;
                }
            }
        }
    };

    auto process_row = [&](int y, uint4 cur) __attribute__((always_inline)) {
        // base only changes in uniform control flow; say so, so that the
        // table reads below stay scalar loads
        base = __builtin_amdgcn_readfirstlane(base);
        const cptr<int32_t> sr = scat + y * kScatterWords;
        const int first = sr[0];
        const int cnt = sr[1];
        const int skip = base - first;
        const int n = min(cnt, i1 - first) - skip;
        const cptr<float> wr = (cptr<float>)(sr + 2) + skip;
        const bool closes = base < i1 && y == close_row[base];
        if (closes && ring_slots == 1) __syncthreads();   // the previous x pass has read the row
        if (vlane) {
            const uint32_t shift = (lead + static_cast<uint32_t>(y) * row_bytes) & 3u;
            uint32_t d0 = cur.x, d1 = cur.y, d2 = cur.z;
            if (shift != 0) {
                d0 = __builtin_amdgcn_alignbyte(cur.y, cur.x, shift);
                d1 = __builtin_amdgcn_alignbyte(cur.z, cur.y, shift);
                d2 = __builtin_amdgcn_alignbyte(cur.w, cur.z, shift);
            }
            float v[12];
            v[0] = float(d0 & 255u);
            v[1] = float((d0 >> 8) & 255u);
            v[2] = float((d0 >> 16) & 255u);
            v[3] = float(d0 >> 24);
            v[4] = float(d1 & 255u);
            v[5] = float((d1 >> 8) & 255u);
            v[6] = float((d1 >> 16) & 255u);
            v[7] = float(d1 >> 24);
            v[8] = float(d2 & 255u);
            v[9] = float((d2 >> 8) & 255u);
            v[10] = float((d2 >> 16) & 255u);
            v[11] = float(d2 >> 24);
            if (!closes) {
                add_row<M>(acc, v, wr, n);
            } else {
                float done[12];
                add_row_and_close<M>(acc, v, wr, done);
                put_row(done, ring + (ring_slots > 1 ? (base & 1) : 0) * tlen + 4 * t);
            }
        }
        if (closes) {
            __syncthreads();
            x_pass(base);
            ++base;
        }
    };

    // Rows are loaded kPrefetch ahead, unconditionally: a load past the band
    // or the frame is harmless (in-frame data that is never used, or zeros
    // from the buffer's range check), and an unconditional load keeps every
    // prefetch register in place.
    uint4 pf[kPrefetch];
#pragma unroll
    for (int d = 0; d < kPrefetch; ++d) pf[d] = load_row(y0 + d);

    for (int yb = y0; yb < y1; yb += kPrefetch) {
#pragma unroll
        for (int d = 0; d < kPrefetch; ++d) {
            const int y = yb + d;
            if (y < y1) {
                const uint4 cur = pf[d];
                pf[d] = load_row(y + kPrefetch);
                process_row(y, cur);
            }
        }
    }
}

template <int M, int KX>
int launch_stream_shape(const PlanView& plan, const StreamLaunch& L, void* out, int out_dtype,
                        const Norm& norm, hipStream_t stream) {
    const int slots = L.slots;
    const int lds = L.ring_bytes + L.stage_elems * (out_dtype == 1 ? 2 : 4);
    dim3 grid(L.count), block(L.threads);
    if (out_dtype == 1) {
        auto k = stream_kernel<M, KX, 1>;
        if (lds > 65536) (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                                                   hipFuncAttributeMaxDynamicSharedMemorySize, lds);
        hipLaunchKernelGGL(k, grid, block, lds, stream, plan, L.first, slots, out, norm);
    } else {
        auto k = stream_kernel<M, KX, 0>;
        if (lds > 65536) (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                                                   hipFuncAttributeMaxDynamicSharedMemorySize, lds);
        hipLaunchKernelGGL(k, grid, block, lds, stream, plan, L.first, slots, out, norm);
    }
    return static_cast<int>(hipGetLastError());
}

}  // namespace

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

bool stream_shape_supported(int m, int kx) {
    return m >= 4 && m <= 6 && (kx == 4 || kx == 8 || kx == 12 || kx == 16);
}

int launch_stream(const PlanView& plan, const StreamLaunch& L, void* out, int out_dtype,
                  const Norm& norm, hipStream_t stream) {
    if (L.count <= 0) return 0;
    if (L.threads <= 0 || L.threads > kStreamBlock || L.threads % 64 != 0 ||
        (L.slots != 1 && L.slots != 2))
        return static_cast<int>(hipErrorInvalidConfiguration);
#define VP_STREAM_CASE(MM, KK) \
    if (L.m == MM && L.kx == KK) return launch_stream_shape<MM, KK>(plan, L, out, out_dtype, norm, stream);
    VP_STREAM_CASE(4, 4) VP_STREAM_CASE(4, 8) VP_STREAM_CASE(4, 12) VP_STREAM_CASE(4, 16)
    VP_STREAM_CASE(5, 4) VP_STREAM_CASE(5, 8) VP_STREAM_CASE(5, 12) VP_STREAM_CASE(5, 16)
    VP_STREAM_CASE(6, 4) VP_STREAM_CASE(6, 8) VP_STREAM_CASE(6, 12) VP_STREAM_CASE(6, 16)
#undef VP_STREAM_CASE
    return static_cast<int>(hipErrorInvalidValue);
}

}  // namespace vp
