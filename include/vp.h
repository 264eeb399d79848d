/*
 * vp.h -- C ABI of the MI355X (gfx950) video-frame preprocessing library.
 *
 * The library computes, on one GPU, the per-frame preprocessing of a
 * Qwen-VL-style vision input that EasyVideoR1 (arXiv 2604.16893) caches
 * offline so that it leaves the RL loop (Section 3.1.1, "Efficient RL with
 * Video Caching"): temporal frame-index sampling, smart_resize to multiples
 * of 2P under a per-modality pixel budget (Section 3.1.2, "Independent
 * Resolution Budgets"; Section 4.1, "Training Configuration"), separable
 * antialiased bicubic resampling of decoded uint8 RGB frames, rescale by
 * 1/255 and per-channel mean/std normalisation (Section 1 names sampling,
 * resizing and normalisation as the costly steps), and patchification into
 * merge-window rows of 3 * 2 * P * P values -- P = 16 for Qwen3-VL (1536
 * values), P = 14 for Qwen2-VL and Qwen2.5-VL (1176), the families the
 * paper supports (Section 4.1) -- with the per-item grid (t, h/P, w/P) --
 * the video_grid_thw that every stage must reproduce
 * identically (Section 3.1.1) -- and a row-offset table for ragged mixed
 * image/video batches (Section 3.2.2, "Joint Image-Video Training").
 *
 * Conventions shared by every entry point:
 *  - Return value: a vp_status code; VP_OK (0) on success.  No function
 *    throws, aborts or prints.  Every argument is validated on the host
 *    before anything is enqueued, so on any non-OK status other than
 *    VP_ERR_HIP nothing has been enqueued on the stream and no output
 *    buffer has been written, except that *out_count / *workspace_bytes
 *    style size outputs report the size that would have been needed (strict
 *    failure: never truncate or pad, Section 3.2.2).
 *  - VP_ERR_HIP is the one exception: a HIP runtime call failed after the
 *    checks passed.  Whatever the call had enqueued before that point (the
 *    plan copy into the workspace, earlier kernel launches) stays enqueued
 *    and the stream still orders after it, but the outputs are undefined.
 *    The message names the failing runtime call.
 *  - vp_last_error_message() returns a thread-local, human-readable detail
 *    of the last non-OK status on the calling thread.
 *  - All functions are thread-safe.  Calls that enqueue work on the same
 *    stream execute in stream order.
 *  - "HOST" pointers are ordinary CPU memory, read or written before the
 *    function returns.  "DEVICE" pointers are GPU memory of the current HIP
 *    device, owned by the caller, and must stay valid until the stream has
 *    reached the work the call enqueued.
 */
#ifndef VP_H
#define VP_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define VP_OK 0
#define VP_ERR_NULL 1       /* a required pointer is NULL                         */
#define VP_ERR_ARG 2        /* an argument is out of its documented range         */
#define VP_ERR_ASPECT 3     /* smart_resize: longer/shorter side ratio above 200  */
#define VP_ERR_DIMS 4       /* a size is non-positive or not a multiple of 2P     */
#define VP_ERR_INDEX 5      /* a frame index lies outside [0, n_src)              */
#define VP_ERR_FRAMES 6     /* a frame count is impossible (n < 1, n > N, ...)    */
#define VP_ERR_CAPACITY 7   /* an output or workspace buffer is too small         */
#define VP_ERR_HIP 8        /* a HIP runtime call failed (detail in the message)  */

/* Geometry: patch P = 16 by default (vp_item.patch selects 14), spatial
 * merge 2, temporal patch 2. */
#define VP_PATCH 16
#define VP_PATCH_QWEN2 14
#define VP_MERGE 2
#define VP_TEMPORAL_PATCH 2
#define VP_FACTOR 32        /* VP_PATCH * VP_MERGE (28 for patch 14) */
#define VP_ROW 1536         /* 3 * VP_TEMPORAL_PATCH * VP_PATCH * VP_PATCH (1176 for patch 14) */

/* Frame-index sampling modes. */
#define VP_SAMPLE_UNIFORM 0
#define VP_SAMPLE_FPS 1

/* Output element types. */
#define VP_OUT_F32 0
#define VP_OUT_BF16 1

/*
 * smart_resize (Section 3.1.1: resize under max_pixels; Section 3.1.2:
 * separate image / video budgets; Section 4.1: a per-frame budget).
 *
 * Target size (out_h, out_w), both positive multiples of `factor` (2P: 32
 * for patch 16, 28 for patch 14), for a height x width source under the
 * per-frame budget [min_pixels, max_pixels]:
 *   h = max(F, rhe(H/F)*F), w = max(F, rhe(W/F)*F)   (rhe: round half to even);
 *   if h*w > max_pixels: beta = sqrt(H*W/max_pixels),
 *       h = max(F, floor(H/beta/F)*F), w = max(F, floor(W/beta/F)*F);
 *   else if h*w < min_pixels: beta = sqrt(min_pixels/(H*W)),
 *       h = ceil(H*beta/F)*F, w = ceil(W*beta/F)*F.
 * Every expression is evaluated in IEEE double precision in the written
 * order.  Applying the function to its own output returns the same size
 * whenever that output lies inside the budget (stage consistency).
 * Errors: VP_ERR_NULL (out pointers), VP_ERR_ARG (height, width, factor or
 * max_pixels <= 0, min_pixels < 0 or > max_pixels), VP_ERR_ASPECT
 * (max(H,W)/min(H,W) > 200), VP_ERR_DIMS (result above INT32_MAX).
 */
int32_t vp_smart_resize_dims(int32_t height, int32_t width, int32_t factor,
                             int64_t min_pixels, int64_t max_pixels,
                             int32_t* out_h, int32_t* out_w);

/*
 * Frame-index sampling (Section 3.1.1: cache entries keyed by fps and
 * max_frames; Section 4.1: 2 FPS with at most 128 frames).
 *
 * mode VP_SAMPLE_UNIFORM: n = nframes indices,
 *     idx_i = rhe(i * (N-1) / (n-1)) on the exact rational (idx = {0} for n = 1).
 * mode VP_SAMPLE_FPS: n = N / video_fps * fps (double), clamped to
 *     [ceil_even(min_frames), floor_even(max_frames)] and to N, floored to an
 *     even count; then the uniform indices for that n.  nframes is ignored.
 * out_idx: HOST int32[capacity], receives the n sorted indices in [0, N).
 * out_count: HOST, receives n (also on VP_ERR_CAPACITY, so a caller can size
 * the buffer).
 * Errors: VP_ERR_NULL, VP_ERR_ARG (unknown mode; fps mode with
 * video_fps or fps <= 0, min_frames < 1 or max_frames < min_frames),
 * VP_ERR_FRAMES (N < 1; uniform n < 1 or n > N; fps count < 2),
 * VP_ERR_CAPACITY (capacity < n).
 */
int32_t vp_sample_indices(int32_t total_frames, int32_t mode, int32_t nframes,
                          double video_fps, double fps, int32_t min_frames, int32_t max_frames,
                          int32_t* out_idx, int32_t capacity, int32_t* out_count);

/*
 * Antialiased bicubic filter of one axis resampled from n_in to n_out
 * samples: Keys (1981) cubic convolution with a = -0.5, stretched by
 * sigma = max(n_in/n_out, 1).  Output i is centred at c = (i + 0.5) *
 * n_in/n_out and reads the window [max(0, floor(c - 2 sigma + 0.5)),
 * min(n_in, floor(c + 2 sigma + 0.5))); its weights K((j + 0.5 - c)/sigma)
 * are normalised to sum 1 (truncated and renormalised at the borders).
 *
 * vp_filter_taps: *max_taps = the longest window over all outputs.
 * vp_filter_table: start[n_out], count[n_out] (HOST int32) and
 * weights[n_out][taps] (HOST float, row i zero beyond count[i]); `taps`
 * must be >= vp_filter_taps.  The weights are computed in double precision
 * and rounded once to float.
 * Errors: VP_ERR_NULL, VP_ERR_ARG (n_in or n_out < 1), VP_ERR_CAPACITY
 * (taps too small).
 */
int32_t vp_filter_taps(int32_t n_in, int32_t n_out, int32_t* max_taps);
int32_t vp_filter_table(int32_t n_in, int32_t n_out, int32_t taps,
                        int32_t* start, int32_t* count, float* weights);

/*
 * The same filter in the fixed point of vp_resize_batch: every double
 * weight times 2^22, rounded half away from zero, as int32 (HOST
 * q[n_out][taps], zero beyond count[i]); start and count as above.
 * Errors: as vp_filter_table.
 */
int32_t vp_filter_table_fixed(int32_t n_in, int32_t n_out, int32_t taps,
                              int32_t* start, int32_t* count, int32_t* q);

/*
 * One video or image of a batch.  A video is n_src decoded frames; an image
 * is one frame (n_src = 1, n_idx = 1) that the temporal patch of 2 turns
 * into two identical frames (Section 3.2.2: images and videos share one
 * field schema and one batch).
 */
typedef struct vp_item {
    const uint8_t* frames;   /* DEVICE [n_src][src_h][src_w][3] packed RGB, contiguous   */
    const int32_t* indices;  /* HOST [n_idx] frame indices in [0, n_src), any order;
                                an odd count gets its last index repeated            */
    int32_t n_src;           /* decoded frames available, >= 1                          */
    int32_t src_h, src_w;    /* source size, >= 1                                       */
    int32_t n_idx;           /* sampled frames, >= 1                                    */
    int32_t dst_h, dst_w;    /* target size, positive multiples of 2 * patch
                                (for instance from vp_smart_resize_dims with
                                factor 2 * patch)                                  */
    int32_t patch;           /* patch edge P in pixels: 16 (Qwen3-VL; 0 also means
                                16) or 14 (Qwen2-VL, Qwen2.5-VL).  All items of
                                one call share it; rows hold 3 * 2 * P * P values
                                (1536 or 1176)                                     */
} vp_item;

/*
 * Batch layout (Section 3.1.1: identical video_grid_thw in every stage).
 * With P the items' patch size:
 * grid_thw: HOST int32[n_items][3] = (t, dst_h/P, dst_w/P), t = ceil(n_idx/2).
 * cu_seqlens: HOST int32[n_items + 1], cu[0] = 0, cu[b+1] = cu[b] + t*(h/P)*(w/P);
 *   item b owns output rows [cu[b], cu[b+1]).
 * total_rows: HOST, = cu[n_items].
 * workspace_bytes: HOST, the device workspace vp_preprocess_batch needs.
 * Any of the four output pointers may be NULL when not wanted.
 * The items' frame pointers are not dereferenced.
 * Errors: VP_ERR_NULL (items), VP_ERR_ARG (n_items < 1), VP_ERR_DIMS,
 * VP_ERR_FRAMES, VP_ERR_INDEX (validated as vp_preprocess_batch does),
 * VP_ERR_CAPACITY (more than INT32_MAX rows).
 */
int32_t vp_batch_layout(const vp_item* items, int32_t n_items, int32_t* grid_thw,
                        int32_t* cu_seqlens, int64_t* total_rows, int64_t* workspace_bytes);

/*
 * Diagnostic: the kernel launches that vp_preprocess_batch makes for a
 * batch, without running them (no device memory is touched): which form of
 * the resampling (Section 3.2: resize, normalise and patchify fused into one
 * pass per frame) each group of items takes.  For tests and tuning.
 * launches: HOST int32[capacity][6], or NULL with capacity 0.  Row i:
 *   kind: VP_KERNEL_GENERIC, VP_KERNEL_YFIRST or VP_KERNEL_XFIRST;
 *   M, the accumulator slots (output rows open at one source row; 0 for
 *   the generic kernel);
 *   the column taps of the x windows (0 for the generic kernel);
 *   y-first: source pixels per lane; else 0;
 *   x-first: output columns per lane (1, or 2 for column pairs); else 0;
 *   workgroups (the generic kernel: output tiles).
 *   Rows past `capacity` are not written.
 * n_launches: HOST, receives the number of launches.
 * Errors: as vp_batch_layout; VP_ERR_NULL (n_launches), VP_ERR_ARG
 * (capacity < 0, or launches NULL with capacity > 0).
 */
#define VP_KERNEL_GENERIC 0
#define VP_KERNEL_YFIRST 1
#define VP_KERNEL_XFIRST 2
int32_t vp_batch_kernels(const vp_item* items, int32_t n_items, int32_t* launches,
                         int32_t capacity, int32_t* n_launches);

/*
 * Preprocess a batch on the GPU: for every item, every sampled frame is
 * resampled from (src_h, src_w) to (dst_h, dst_w) with the filter of
 * vp_filter_table along x then y (no clamping, no rounding in between),
 * normalised as v = (R/255 - mean_c)/std_c, padded to an even frame count,
 * and written as merge-window rows of 6*P*P values (P the patch size):
 *   row cu[b] + ((tt*(h/2P) + bh)*(w/2P) + bw)*4 + mh*2 + mw,
 *   column ((c*2 + dt)*P + y)*P + x  holds
 *   v[frame 2*tt + dt][c][P*(2*bh + mh) + y][P*(2*bw + mw) + x].
 *
 * mean, std: HOST float[3] (std > 0, finite).
 * out_dtype: VP_OUT_F32 or VP_OUT_BF16 (round to nearest even).
 * out_rows: DEVICE [out_rows_capacity][6*P*P] of out_dtype, row-major,
 *   16-byte aligned.
 * grid_thw, cu_seqlens: HOST outputs as in vp_batch_layout (may be NULL);
 *   final when the call returns.
 * workspace: DEVICE, >= the workspace_bytes of vp_batch_layout, 256-byte
 *   aligned; the call copies its plan (item table, filter tables, indices)
 *   there on `stream` and the kernels read it.  It may be reused by the
 *   next call on the same stream.
 * stream: the HIP stream all work is enqueued on (0 = the null stream).
 *   When a batch needs kernels of several shapes, the call runs them on up
 *   to three more streams of the device (created once by the library, at
 *   default priority), forked from `stream` and joined back into it with
 *   events: to other work on `stream` the call is one ordered step.
 * out_rows is final when `stream` reaches the end of the enqueued work.
 * Errors: VP_ERR_NULL, VP_ERR_ARG (n_items < 1, bad dtype, std <= 0 or not
 * finite, misaligned pointers, a patch size other than 14 or 16, items with
 * different patch sizes), VP_ERR_DIMS, VP_ERR_FRAMES, VP_ERR_INDEX,
 * VP_ERR_CAPACITY (out_rows_capacity < total rows, workspace too small, a
 * frame of 4 GiB or more, a filter window too long for the kernels),
 * VP_ERR_HIP.
 */
int32_t vp_preprocess_batch(const vp_item* items, int32_t n_items, const float* mean,
                            const float* std, int32_t out_dtype, void* out_rows,
                            int64_t out_rows_capacity, int32_t* grid_thw, int32_t* cu_seqlens,
                            void* workspace, int64_t workspace_bytes, hipStream_t stream);

/*
 * vp_preprocess_batch for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same computation and outputs, with no workspace argument.
 * The plan goes to a fixed array of device memory inside the library,
 * VP_NOALLOC_PLAN_BYTES (16 MiB) per device, held by every device the
 * library runs on until the process ends; it is copied there on `stream`
 * from pageable host memory, and every kernel runs on `stream` itself (no
 * side streams).  The call allocates no device memory, creates no stream or
 * event, and makes no hipMalloc, hipHostMalloc or hipFree call; its first
 * call on a device looks up that device's copy of the array.
 * All calls on one device share the array, which keeps the last call's plan:
 * calls whose work can overlap on one device (different streams, or other
 * threads, without synchronisation between them) race and give undefined
 * output.  Calls on one stream are ordered and safe.
 * Arguments, outputs, ownership and asynchrony otherwise as for
 * vp_preprocess_batch.
 * Errors: as vp_preprocess_batch, with VP_ERR_CAPACITY when the batch's plan
 * (the workspace_bytes of vp_batch_layout) exceeds VP_NOALLOC_PLAN_BYTES;
 * this and every other argument check happens before any HIP call.
 */
#define VP_NOALLOC_PLAN_BYTES (16 * 1024 * 1024)
int32_t vp_preprocess_batch_noalloc(const vp_item* items, int32_t n_items, const float* mean,
                                    const float* std, int32_t out_dtype, void* out_rows,
                                    int64_t out_rows_capacity, int32_t* grid_thw,
                                    int32_t* cu_seqlens, hipStream_t stream);

/*
 * Normalise and patchify frames that are already at the target size: the
 * cached path of Section 3.1.1, where sampling and resizing were done once
 * offline and every RL stage still rescales, normalises and patchifies.
 * Items as for vp_preprocess_batch, with dst_h == src_h and dst_w == src_w
 * (multiples of 2P); `indices` select and order the frames as before, odd
 * counts padded with the last index.  The rows are those vp_preprocess_batch
 * writes for the same items, whose resize is then the identity:
 *   row cu[b] + ((tt*(h/2P) + bh)*(w/2P) + bw)*4 + mh*2 + mw,
 *   column ((c*2 + dt)*P + y)*P + x  holds (F/255 - mean_c)/std_c of
 *   F = frames[indices[2*tt + dt]][P*(2*bh + mh) + y][P*(2*bw + mw) + x][c].
 * Arguments, ownership, asynchrony and stream as for vp_preprocess_batch;
 * the workspace_bytes of vp_batch_layout on the same items suffice.  Each
 * frames pointer must be 4-byte aligned.
 * Errors: as vp_preprocess_batch, plus VP_ERR_DIMS when a target size is not
 * its source size, VP_ERR_ARG when a frames pointer is not 4-byte aligned.
 */
int32_t vp_patchify_batch(const vp_item* items, int32_t n_items, const float* mean,
                          const float* std, int32_t out_dtype, void* out_rows,
                          int64_t out_rows_capacity, int32_t* grid_thw, int32_t* cu_seqlens,
                          void* workspace, int64_t workspace_bytes, hipStream_t stream);

/*
 * Layout of a vp_resize_batch call.
 * frame_off: HOST int64[n_items + 1]: item b's resized frames start at byte
 *   frame_off[b] of the output; frame_off[0] = 0, frame_off[b+1] =
 *   frame_off[b] + n_idx * dst_h * dst_w * 3; frame_off[n_items] is the total.
 * workspace_bytes: HOST, the device workspace vp_resize_batch needs.
 * Either pointer may be NULL.  Frame pointers are not dereferenced.
 * Errors: as vp_batch_layout, plus VP_ERR_CAPACITY when a filter window is
 * too long for the kernel's tiles.
 */
int32_t vp_resize_layout(const vp_item* items, int32_t n_items, int64_t* frame_off,
                         int64_t* workspace_bytes);

/*
 * uint8 cache writer (Section 3.1.1: the offline cache holds frames that are
 * already sampled and resized; as uint8 they take a quarter of the float
 * tensors' space).  For every item, every sampled frame, in index order and
 * without temporal padding, is resampled from (src_h, src_w) to
 * (dst_h, dst_w) in fixed point, so that the bytes are reproducible exactly:
 *   weights q_j = the weights of vp_filter_table computed in double and
 *   scaled by 2^22, rounded half away from zero;
 *   a horizontal pass over every source row, then a vertical pass, each
 *   giving clamp(floor((sum_j q_j * v_j + 2^21) / 2^22), 0, 255).
 * These are the conventions of PIL-style integer resizers for 8-bit images.
 * Item b's frames go to out_frames + frame_off[b] as uint8
 * [n_idx][dst_h][dst_w][3] (see vp_resize_layout).
 * out_frames: DEVICE, >= frame_off[n_items] bytes (out_capacity), 4-byte
 *   aligned.
 * frame_off: HOST output as in vp_resize_layout (may be NULL).
 * workspace, stream, ownership and asynchrony as for vp_preprocess_batch,
 *   with the workspace_bytes of vp_resize_layout.
 * Errors: VP_ERR_NULL, VP_ERR_ARG (n_items < 1, misaligned pointers),
 * VP_ERR_DIMS, VP_ERR_FRAMES, VP_ERR_INDEX, VP_ERR_CAPACITY (output or
 * workspace too small, a filter window too long for the kernel's tiles),
 * VP_ERR_HIP.
 */
int32_t vp_resize_batch(const vp_item* items, int32_t n_items, void* out_frames,
                        int64_t out_capacity, int64_t* frame_off, void* workspace,
                        int64_t workspace_bytes, hipStream_t stream);

/*
 * Position tables of a batch (Section 1: metadata-consistent
 * spatial-temporal positional encoding; Section 3.1.1: the same
 * video_grid_thw in every stage).  Items and their rows as in
 * vp_batch_layout / vp_preprocess_batch (item b owns rows [cu[b], cu[b+1]),
 * row cu[b] + ((tt*(h/2P) + bh)*(w/2P) + bw)*4 + mh*2 + mw):
 *   vit_pos[row] = (tt, 2*bh + mh, 2*bw + mw)  frame pair, patch row, patch column
 *     -- the coordinates of the ViT's 2D rotary embedding;
 *   llm_pos[row/4] = (tt, bh, bw)  one per merge window, the token it becomes
 *     after the 2x2 merge -- the grid coordinates of the LLM's 3-axis M-RoPE
 *     (the model adds its own temporal scaling and text offset);
 *   vit_cu: the ViT's attention segments, one per frame pair of each item:
 *     vit_cu[0] = 0, vit_cu[s+1] = vit_cu[s] + (h/P)*(w/P).
 * vit_pos: DEVICE int32 [rows][3], llm_pos: DEVICE int32 [rows/4][3]; either
 *   may be NULL; rows_capacity = rows the caller's vit_pos holds (llm_pos
 *   holds rows_capacity/4); 4-byte aligned.
 * vit_cu: HOST int32 [vit_cu_capacity] (may be NULL); *n_slices (HOST, may
 *   be NULL) = S, the number of segments.
 * workspace, stream, ownership and asynchrony as for vp_preprocess_batch,
 *   with the workspace_bytes of vp_batch_layout.  The frames pointers are
 *   not dereferenced.
 * Errors: VP_ERR_NULL, VP_ERR_ARG, VP_ERR_DIMS, VP_ERR_FRAMES, VP_ERR_INDEX,
 * VP_ERR_CAPACITY (rows_capacity < rows, vit_cu_capacity < S + 1,
 * workspace too small), VP_ERR_HIP.
 */
int32_t vp_position_ids(const vp_item* items, int32_t n_items, int32_t* vit_pos,
                        int32_t* llm_pos, int64_t rows_capacity, int32_t* vit_cu,
                        int32_t vit_cu_capacity, int32_t* n_slices, void* workspace,
                        int64_t workspace_bytes, hipStream_t stream);

/*
 * Kernel timing hook (measurement only; not a step of the method).  The next
 * vp_preprocess_batch, vp_patchify_batch, vp_resize_batch or vp_position_ids
 * call made on this thread (one that launches kernels) records `start` on
 * its stream immediately before its first kernel
 * launch (after the plan upload) and
 * `stop` immediately after its last launch, then forgets both events, so
 * that hipEventElapsedTime(start, stop) is the device time of that call's
 * kernels alone.  A call that fails before launching records neither.
 * start, stop: events created by the caller (hipEventCreate or equivalent),
 *   still owned by the caller; NULL, NULL cancels a pending request.
 * Errors: VP_ERR_NULL (exactly one of the two is NULL).
 */
int32_t vp_set_kernel_events(hipEvent_t start, hipEvent_t stop);

/* Static name of a status code ("VP_OK", "VP_ERR_ARG", ...). */
const char* vp_status_string(int32_t status);

/* Thread-local detail of the last non-OK status on this thread ("" if none). */
const char* vp_last_error_message(void);

#ifdef __cplusplus
}
#endif

#endif /* VP_H */
