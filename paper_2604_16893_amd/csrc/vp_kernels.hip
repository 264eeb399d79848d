// vp_kernels.hip -- gfx950 kernels of the preprocessing path.
//
// One work unit is one merge window (32 x 32 output pixels) of one frame pair
// of one item: exactly four consecutive output rows of 1536 values
// (Section 3.1.1 of arXiv 2604.16893 requires the same video_grid_thw in
// every stage; the row order is the merge-window order of the grid).  For
// each of the two frames the unit resamples its 32 x 32 pixels with the
// separable antialiased bicubic filter -- first along y into an LDS column
// tile (the u8 source read straight from global memory), then along x out of
// that tile -- normalises with one FMA per value, and stages the result in
// LDS in output order; the four rows then leave with 16-byte stores.
//
// This general kernel handles every scale factor: when the horizontal
// window of 32 output columns does not fit the LDS tile, the unit walks
// its 32 x 32 pixels in sub-tiles of rh rows x cw columns chosen by the host.
#include <hip/hip_runtime.h>

#include "vp_plan.h"

namespace vp {
namespace {

__device__ __forceinline__ uint32_t bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ int find_item(const int32_t* prefix, int n_items, int tile) {
    int lo = 0, hi = n_items;  // prefix[lo] <= tile < prefix[hi]
    while (hi - lo > 1) {
        int mid = (lo + hi) >> 1;
        if (prefix[mid] <= tile) lo = mid; else hi = mid;
    }
    return lo;
}

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

}  // namespace vp
