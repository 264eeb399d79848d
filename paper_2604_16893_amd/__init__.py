"""MI355X-native video-frame preprocessing for Qwen-VL-style vision inputs.

Python binding of ``libvp.so`` (C ABI in ``include/vp.h``): the per-frame
preprocessing that EasyVideoR1 (arXiv 2604.16893, Section 3.1.1) caches
offline -- frame-index sampling, smart_resize, antialiased bicubic
resampling, normalisation and merge-window patchification with grid_thw and
cu_seqlens -- runs in hand-written gfx950 HIP kernels.  This module only
marshals arguments: torch provides device memory and the current stream.

Importing never compiles anything; build with
``python -m paper_2604_16893_amd.build``.  Every entry point raises
``VPError`` when the native library is missing -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libvp.so")

VP_OK, VP_ERR_NULL, VP_ERR_ARG, VP_ERR_ASPECT, VP_ERR_DIMS, VP_ERR_INDEX, VP_ERR_FRAMES, \
    VP_ERR_CAPACITY, VP_ERR_HIP = range(9)
VP_SAMPLE_UNIFORM, VP_SAMPLE_FPS = 0, 1
VP_OUT_F32, VP_OUT_BF16 = 0, 1
VP_ROW = 1536
VP_PATCH = 16
VP_NOALLOC_PLAN_BYTES = 16 * 1024 * 1024


def row_width(patch: int = VP_PATCH) -> int:
    """Values per merge-window row: 3 channels x 2 frames x patch x patch
    (1536 for patch 16, 1176 for patch 14)."""
    return 6 * patch * patch
VP_FACTOR = 32

EXPORTED = ("vp_smart_resize_dims", "vp_sample_indices", "vp_filter_taps", "vp_filter_table",
            "vp_filter_table_fixed", "vp_batch_layout", "vp_batch_kernels", "vp_preprocess_batch",
            "vp_preprocess_batch_noalloc", "vp_patchify_batch",
            "vp_resize_layout", "vp_resize_batch", "vp_position_ids", "vp_status_string",
            "vp_last_error_message", "vp_set_kernel_events")


class VPError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


class vp_item(ctypes.Structure):
    _fields_ = [("frames", ctypes.c_void_p),
                ("indices", ctypes.POINTER(ctypes.c_int32)),
                ("n_src", ctypes.c_int32),
                ("src_h", ctypes.c_int32),
                ("src_w", ctypes.c_int32),
                ("n_idx", ctypes.c_int32),
                ("dst_h", ctypes.c_int32),
                ("dst_w", ctypes.c_int32),
                ("patch", ctypes.c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded native library; raises VPError if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise VPError(-1, f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2604_16893_amd.build` (no fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        i32p, i64p, f32p = ctypes.POINTER(i32), ctypes.POINTER(i64), ctypes.POINTER(ctypes.c_float)
        itemp = ctypes.POINTER(vp_item)
        L.vp_smart_resize_dims.argtypes = [i32, i32, i32, i64, i64, i32p, i32p]
        L.vp_sample_indices.argtypes = [i32, i32, i32, f64, f64, i32, i32, i32p, i32, i32p]
        L.vp_filter_taps.argtypes = [i32, i32, i32p]
        L.vp_filter_table.argtypes = [i32, i32, i32, i32p, i32p, f32p]
        L.vp_batch_layout.argtypes = [itemp, i32, i32p, i32p, i64p, i64p]
        L.vp_batch_kernels.argtypes = [itemp, i32, i32p, i32, i32p]
        L.vp_preprocess_batch.argtypes = [itemp, i32, f32p, f32p, i32, ctypes.c_void_p, i64,
                                          i32p, i32p, ctypes.c_void_p, i64, ctypes.c_void_p]
        L.vp_patchify_batch.argtypes = L.vp_preprocess_batch.argtypes
        L.vp_preprocess_batch_noalloc.argtypes = [itemp, i32, f32p, f32p, i32, ctypes.c_void_p, i64,
                                                  i32p, i32p, ctypes.c_void_p]
        L.vp_filter_table_fixed.argtypes = [i32, i32, i32, i32p, i32p, i32p]
        L.vp_position_ids.argtypes = [itemp, i32, ctypes.c_void_p, ctypes.c_void_p, i64, i32p, i32,
                                      i32p, ctypes.c_void_p, i64, ctypes.c_void_p]
        L.vp_resize_layout.argtypes = [itemp, i32, i64p, i64p]
        L.vp_resize_batch.argtypes = [itemp, i32, ctypes.c_void_p, i64, i64p, ctypes.c_void_p, i64,
                                      ctypes.c_void_p]
        L.vp_set_kernel_events.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        L.vp_status_string.argtypes = [i32]
        L.vp_status_string.restype = ctypes.c_char_p
        L.vp_last_error_message.argtypes = []
        L.vp_last_error_message.restype = ctypes.c_char_p
        for name in EXPORTED:
            getattr(L, name).restype = getattr(L, name).restype if name in (
                "vp_status_string", "vp_last_error_message") else i32
        _lib = L
    return _lib


def _check(status: int, what: str):
    if status != VP_OK:
        L = lib()
        raise VPError(status, f"{what}: {L.vp_status_string(status).decode()}: "
                              f"{L.vp_last_error_message().decode()}")


def _ptr(a: np.ndarray, ct):
    return a.ctypes.data_as(ctypes.POINTER(ct))


# --------------------------------------------------------------------------
# Host entry points (same names as the C ABI)
# --------------------------------------------------------------------------

def vp_smart_resize_dims(height: int, width: int, factor: int = VP_FACTOR, min_pixels: int = 0,
                         max_pixels: int = (1 << 62)) -> tuple[int, int]:
    h, w = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().vp_smart_resize_dims(height, width, factor, min_pixels, max_pixels,
                                      ctypes.byref(h), ctypes.byref(w)), "vp_smart_resize_dims")
    return h.value, w.value


def vp_sample_indices(total_frames: int, mode: int = VP_SAMPLE_UNIFORM, nframes: int = 0,
                      video_fps: float = 0.0, fps: float = 0.0, min_frames: int = 1,
                      max_frames: int = 1 << 30) -> np.ndarray:
    cnt = ctypes.c_int32()
    st = lib().vp_sample_indices(total_frames, mode, nframes, video_fps, fps, min_frames,
                                 max_frames, None, 0, ctypes.byref(cnt))
    if st != VP_ERR_CAPACITY:
        _check(st, "vp_sample_indices")
    out = np.zeros(max(cnt.value, 1), np.int32)
    _check(lib().vp_sample_indices(total_frames, mode, nframes, video_fps, fps, min_frames,
                                   max_frames, _ptr(out, ctypes.c_int32), len(out),
                                   ctypes.byref(cnt)), "vp_sample_indices")
    return out[:cnt.value]


def vp_filter_taps(n_in: int, n_out: int) -> int:
    k = ctypes.c_int32()
    _check(lib().vp_filter_taps(n_in, n_out, ctypes.byref(k)), "vp_filter_taps")
    return k.value


def vp_filter_table(n_in: int, n_out: int, taps: Optional[int] = None):
    """(start[n_out], count[n_out], weights[n_out][taps]) of one axis."""
    taps = vp_filter_taps(n_in, n_out) if taps is None else taps
    start = np.zeros(n_out, np.int32)
    count = np.zeros(n_out, np.int32)
    w = np.zeros((n_out, taps), np.float32)
    _check(lib().vp_filter_table(n_in, n_out, taps, _ptr(start, ctypes.c_int32),
                                 _ptr(count, ctypes.c_int32), _ptr(w, ctypes.c_float)),
           "vp_filter_table")
    return start, count, w


def vp_filter_table_fixed(n_in: int, n_out: int, taps: Optional[int] = None):
    """(start int32 [n_out], count int32 [n_out], q int32 [n_out, taps]): the
    filter's weights in units of 2^-22, as the uint8 writer uses them."""
    if taps is None:
        taps = vp_filter_taps(n_in, n_out)
    start = np.zeros(n_out, np.int32)
    count = np.zeros(n_out, np.int32)
    q = np.zeros((n_out, taps), np.int32)
    _check(lib().vp_filter_table_fixed(n_in, n_out, taps, _ptr(start, ctypes.c_int32),
                                       _ptr(count, ctypes.c_int32), _ptr(q, ctypes.c_int32)),
           "vp_filter_table_fixed")
    return start, count, q


# --------------------------------------------------------------------------
# Batches
# --------------------------------------------------------------------------

@dataclasses.dataclass
class Item:
    """One video or image: device frames [n_src, H, W, 3] uint8, sampled
    indices, the target size (multiples of 2 * patch) and the patch size
    (16, or 14 for the Qwen2/2.5-VL geometry; one per call)."""
    frames: object
    indices: Sequence[int]
    dst_h: int
    dst_w: int
    patch: int = VP_PATCH


class _Batch:
    """ctypes view of a list of Items; keeps the host index arrays alive."""

    def __init__(self, items: Sequence):
        self.idx = []
        self.arr = (vp_item * len(items))()
        for k, it in enumerate(items):
            fr = it.frames
            if hasattr(fr, "data_ptr"):
                if fr.dtype.__repr__() != "torch.uint8" or fr.dim() != 4 or fr.shape[3] != 3 \
                        or not fr.is_contiguous():
                    raise VPError(VP_ERR_ARG, f"item {k}: frames must be a contiguous uint8 "
                                              "[n_src, H, W, 3] tensor")
                ptr, (n_src, H, W, _) = fr.data_ptr(), tuple(fr.shape)
            else:   # (device pointer, n_src, H, W) -- layout-only callers
                ptr, n_src, H, W = fr
            idx = np.ascontiguousarray(np.asarray(it.indices, dtype=np.int32).reshape(-1))
            self.idx.append(idx)
            self.arr[k] = vp_item(ptr, _ptr(idx, ctypes.c_int32), n_src, H, W, len(idx),
                                  it.dst_h, it.dst_w, getattr(it, "patch", VP_PATCH))

    def __len__(self):
        return len(self.arr)


def vp_batch_layout(items: Sequence):
    """(grid_thw int32 [B,3], cu_seqlens int32 [B+1], total_rows, workspace_bytes)."""
    b = _Batch(items)
    B = len(b)
    grid = np.zeros((B, 3), np.int32)
    cu = np.zeros(B + 1, np.int32)
    rows, ws = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().vp_batch_layout(b.arr, B, _ptr(grid, ctypes.c_int32), _ptr(cu, ctypes.c_int32),
                                 ctypes.byref(rows), ctypes.byref(ws)), "vp_batch_layout")
    return grid, cu, rows.value, ws.value


VP_KERNEL_GENERIC, VP_KERNEL_YFIRST, VP_KERNEL_XFIRST = 0, 1, 2


def vp_batch_kernels(items: Sequence):
    """The launches vp_preprocess_batch makes for the batch, as int32 rows
    (kind, slots M, column taps, y-first pixels per lane, x-first columns per
    lane, workgroups); no kernel runs."""
    b = _Batch(items)
    n = ctypes.c_int32()
    _check(lib().vp_batch_kernels(b.arr, len(b), None, 0, ctypes.byref(n)), "vp_batch_kernels")
    rows = np.zeros((max(n.value, 1), 6), np.int32)
    _check(lib().vp_batch_kernels(b.arr, len(b), _ptr(rows, ctypes.c_int32), n.value, ctypes.byref(n)),
           "vp_batch_kernels")
    return rows[:n.value]


def _stream_handle(stream) -> int:
    import torch
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def vp_preprocess_batch(items: Sequence, mean, std, out_dtype: int, out_rows, workspace,
                        stream=None):
    """Enqueue the batch on `stream` (torch stream, raw handle, or None for the
    current stream).  out_rows: device tensor [>= rows, 1536] of float32 or
    bfloat16 matching out_dtype; workspace: device uint8 tensor of at least
    the layout's workspace_bytes.  Returns (grid_thw, cu_seqlens)."""
    return _run("vp_preprocess_batch", items, mean, std, out_dtype, out_rows, workspace, stream)


def vp_preprocess_batch_noalloc(items: Sequence, mean, std, out_dtype: int, out_rows, stream=None):
    """As vp_preprocess_batch with no workspace: the plan goes to the library's
    fixed device memory (at most VP_NOALLOC_PLAN_BYTES), and nothing is
    allocated.  Calls whose work can overlap on one device race; calls on one
    stream are ordered.  Returns (grid_thw, cu_seqlens)."""
    import torch
    want = torch.bfloat16 if out_dtype == VP_OUT_BF16 else torch.float32
    width = row_width(getattr(items[0], "patch", VP_PATCH)) if len(items) else VP_ROW
    if out_rows.dtype != want or out_rows.dim() != 2 or out_rows.shape[1] != width \
            or not out_rows.is_contiguous() or not out_rows.is_cuda:
        raise VPError(VP_ERR_ARG, f"out_rows must be a contiguous CUDA [rows, {width}] {want} tensor")
    b = _Batch(items)
    B = len(b)
    m = np.ascontiguousarray(np.asarray(mean, np.float32).reshape(3))
    s = np.ascontiguousarray(np.asarray(std, np.float32).reshape(3))
    grid = np.zeros((B, 3), np.int32)
    cu = np.zeros(B + 1, np.int32)
    _check(lib().vp_preprocess_batch_noalloc(
        b.arr, B, _ptr(m, ctypes.c_float), _ptr(s, ctypes.c_float), out_dtype,
        ctypes.c_void_p(out_rows.data_ptr()), out_rows.shape[0], _ptr(grid, ctypes.c_int32),
        _ptr(cu, ctypes.c_int32), ctypes.c_void_p(_stream_handle(stream))),
        "vp_preprocess_batch_noalloc")
    return grid, cu


def vp_patchify_batch(items: Sequence, mean, std, out_dtype: int, out_rows, workspace,
                      stream=None):
    """As vp_preprocess_batch, for frames already at the target size (every
    item's dst_h, dst_w equal to its frames' H, W): normalise + patchify only."""
    return _run("vp_patchify_batch", items, mean, std, out_dtype, out_rows, workspace, stream)


def _run(name: str, items: Sequence, mean, std, out_dtype: int, out_rows, workspace, stream):
    import torch
    want = torch.bfloat16 if out_dtype == VP_OUT_BF16 else torch.float32
    width = row_width(getattr(items[0], "patch", VP_PATCH)) if len(items) else VP_ROW
    if out_rows.dtype != want or out_rows.dim() != 2 or out_rows.shape[1] != width \
            or not out_rows.is_contiguous() or not out_rows.is_cuda:
        raise VPError(VP_ERR_ARG, f"out_rows must be a contiguous CUDA [rows, {width}] {want} tensor")
    if not workspace.is_cuda or not workspace.is_contiguous():
        raise VPError(VP_ERR_ARG, "workspace must be a contiguous CUDA tensor")
    b = _Batch(items)
    B = len(b)
    m = np.ascontiguousarray(np.asarray(mean, np.float32).reshape(3))
    s = np.ascontiguousarray(np.asarray(std, np.float32).reshape(3))
    grid = np.zeros((B, 3), np.int32)
    cu = np.zeros(B + 1, np.int32)
    _check(getattr(lib(), name)(
        b.arr, B, _ptr(m, ctypes.c_float), _ptr(s, ctypes.c_float), out_dtype,
        ctypes.c_void_p(out_rows.data_ptr()), out_rows.shape[0], _ptr(grid, ctypes.c_int32),
        _ptr(cu, ctypes.c_int32), ctypes.c_void_p(workspace.data_ptr()),
        workspace.numel() * workspace.element_size(), ctypes.c_void_p(_stream_handle(stream))),
        name)
    return grid, cu


def _event_handle(ev) -> int:
    if ev is None:
        return 0
    if isinstance(ev, int):
        return ev
    handle = getattr(ev, "cuda_event", 0)
    if not handle:
        raise VPError(VP_ERR_ARG, "the event has no HIP event yet: record it once first")
    return handle


def vp_set_kernel_events(start, stop):
    """Ask the next vp_preprocess_batch call on this thread to record `start`
    before its first kernel and `stop` after its last one (torch.cuda.Event
    objects that have been recorded at least once, raw hipEvent_t handles, or
    None, None to cancel)."""
    _check(lib().vp_set_kernel_events(ctypes.c_void_p(_event_handle(start)),
                                      ctypes.c_void_p(_event_handle(stop))),
           "vp_set_kernel_events")


def patchify(items: Sequence, mean, std, out_dtype: str = "bf16", stream=None):
    """Allocate the outputs with torch and run vp_patchify_batch (frames
    already at the target size).  Returns (rows, grid_thw, cu_seqlens)."""
    import torch
    code = VP_OUT_BF16 if out_dtype in ("bf16", VP_OUT_BF16) else VP_OUT_F32
    grid, cu, rows, ws = vp_batch_layout(items)
    dev = items[0].frames.device
    out = torch.empty((rows, row_width(getattr(items[0], "patch", VP_PATCH))),
                      dtype=torch.bfloat16 if code == VP_OUT_BF16 else torch.float32,
                      device=dev)
    work = torch.empty(ws, dtype=torch.uint8, device=dev)
    vp_patchify_batch(items, mean, std, code, out, work, stream)
    return out, grid, cu


def vp_resize_layout(items: Sequence):
    """(frame_off int64 [B+1] output byte offsets, workspace_bytes) of the uint8 writer."""
    b = _Batch(items)
    off = np.zeros(len(b) + 1, np.int64)
    ws = ctypes.c_int64()
    _check(lib().vp_resize_layout(b.arr, len(b), _ptr(off, ctypes.c_int64), ctypes.byref(ws)),
           "vp_resize_layout")
    return off, ws.value


def vp_resize_batch(items: Sequence, out_frames, workspace, stream=None):
    """Enqueue the uint8 writer: out_frames is a contiguous CUDA uint8 tensor
    of at least frame_off[-1] bytes; item b's frames [n_idx, dst_h, dst_w, 3]
    start at byte frame_off[b].  Returns frame_off."""
    import torch
    if out_frames.dtype != torch.uint8 or not out_frames.is_contiguous() or not out_frames.is_cuda:
        raise VPError(VP_ERR_ARG, "out_frames must be a contiguous CUDA uint8 tensor")
    if not workspace.is_cuda or not workspace.is_contiguous():
        raise VPError(VP_ERR_ARG, "workspace must be a contiguous CUDA tensor")
    b = _Batch(items)
    off = np.zeros(len(b) + 1, np.int64)
    _check(lib().vp_resize_batch(b.arr, len(b), ctypes.c_void_p(out_frames.data_ptr()),
                                 out_frames.numel(), _ptr(off, ctypes.c_int64),
                                 ctypes.c_void_p(workspace.data_ptr()),
                                 workspace.numel() * workspace.element_size(),
                                 ctypes.c_void_p(_stream_handle(stream))), "vp_resize_batch")
    return off


def vp_position_ids(items: Sequence, vit_pos, llm_pos, workspace, stream=None):
    """Enqueue the position tables: vit_pos int32 CUDA tensor [>= rows, 3] and
    llm_pos int32 CUDA tensor [>= rows/4, 3] (either may be None); workspace
    as for vp_preprocess_batch.  Returns the ViT segments vit_cu (int32
    numpy [S+1]), final on return."""
    import torch
    for name, t in (("vit_pos", vit_pos), ("llm_pos", llm_pos)):
        if t is not None and (t.dtype != torch.int32 or t.dim() != 2 or t.shape[1] != 3
                              or not t.is_contiguous() or not t.is_cuda):
            raise VPError(VP_ERR_ARG, f"{name} must be a contiguous CUDA int32 [n, 3] tensor")
    b = _Batch(items)
    B = len(b)
    cap = sum((len(np.asarray(it.indices).reshape(-1)) + 1) // 2 for it in items) + 1
    cu = np.zeros(cap, np.int32)
    ns = ctypes.c_int32()
    rows_cap = vit_pos.shape[0] if vit_pos is not None else (llm_pos.shape[0] * 4 if llm_pos is not None else 0)
    if vit_pos is not None and llm_pos is not None:
        rows_cap = min(vit_pos.shape[0], llm_pos.shape[0] * 4)
    _check(lib().vp_position_ids(
        b.arr, B, ctypes.c_void_p(vit_pos.data_ptr() if vit_pos is not None else 0),
        ctypes.c_void_p(llm_pos.data_ptr() if llm_pos is not None else 0), rows_cap,
        _ptr(cu, ctypes.c_int32), cap, ctypes.byref(ns), ctypes.c_void_p(workspace.data_ptr()),
        workspace.numel() * workspace.element_size(), ctypes.c_void_p(_stream_handle(stream))),
        "vp_position_ids")
    return cu[:ns.value + 1]


def resize_u8(items: Sequence, stream=None):
    """Allocate with torch and run the uint8 writer.  Returns a list of
    uint8 tensors [n_idx, dst_h, dst_w, 3] (views of one buffer), final when
    the stream is."""
    import torch
    off, ws = vp_resize_layout(items)
    dev = items[0].frames.device
    out = torch.empty(int(off[-1]), dtype=torch.uint8, device=dev)
    work = torch.empty(max(ws, 1), dtype=torch.uint8, device=dev)
    vp_resize_batch(items, out, work, stream)
    return [out[int(off[k]):int(off[k + 1])].view(len(it.indices), it.dst_h, it.dst_w, 3)
            for k, it in enumerate(items)]


def preprocess(items: Sequence, mean, std, out_dtype: str = "bf16", stream=None):
    """Allocate the outputs with torch and run vp_preprocess_batch.

    Returns (rows [total_rows, 1536] on the frames' device, grid_thw int32
    [B, 3], cu_seqlens int32 [B+1]); rows are final when the stream is."""
    import torch
    code = VP_OUT_BF16 if out_dtype in ("bf16", VP_OUT_BF16) else VP_OUT_F32
    grid, cu, rows, ws = vp_batch_layout(items)
    dev = items[0].frames.device
    out = torch.empty((rows, row_width(getattr(items[0], "patch", VP_PATCH))),
                      dtype=torch.bfloat16 if code == VP_OUT_BF16 else torch.float32,
                      device=dev)
    work = torch.empty(ws, dtype=torch.uint8, device=dev)
    vp_preprocess_batch(items, mean, std, code, out, work, stream)
    return out, grid, cu
