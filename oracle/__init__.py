"""TEST INFRASTRUCTURE: ctypes wrapper of the plain fp64 CPU oracle (oracle.c).

The oracle is a slow, obviously-correct definition of the preprocessing path
of EasyVideoR1 (arXiv 2604.16893, Section 3.1.1 "Efficient RL with Video
Caching", Section 3.1.2 "Independent Resolution Budgets", Section 4.1
"Training Configuration"): frame-index sampling, smart_resize, antialiased
bicubic resampling, rescale + normalise, patchify into 1536-wide merge-window
rows, grid_thw and cu_seqlens.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module.  It shares no code with the GPU library
(``paper_2604_16893_amd``) and neither imports the other.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, ERR_NULL, ERR_ARG, ERR_ASPECT, ERR_DIMS, ERR_INDEX, ERR_FRAMES, ERR_CAPACITY = range(8)
ROW = 1536


class OracleError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: oracle status {code}")
        self.code = code


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so with plain gcc (no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math",
             "-ffp-contract=off", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = ctypes.CDLL(_LIB)
        i64, i32p, i64p, f64p = ctypes.c_int64, ctypes.POINTER(ctypes.c_int32), \
            ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_double)
        u8p = ctypes.POINTER(ctypes.c_uint8)
        L.oracle_smart_resize.argtypes = [i64, i64, i64, i64, i64, i64p, i64p]
        L.oracle_sample_uniform.argtypes = [i64, i64, i32p]
        L.oracle_sample_fps.argtypes = [i64, ctypes.c_double, ctypes.c_double, i64, i64,
                                        i32p, i64, i64p]
        L.oracle_keys_cubic.argtypes = [ctypes.c_double]
        L.oracle_keys_cubic.restype = ctypes.c_double
        L.oracle_filter.argtypes = [i64, i64, i64, i64p, i64p, f64p, i64]
        L.oracle_filter_max_taps.argtypes = [i64, i64]
        L.oracle_filter_max_taps.restype = i64
        L.oracle_filter_table.argtypes = [i64, i64, i64p, i64p, f64p, i64]
        L.oracle_resize_frame.argtypes = [u8p, i64, i64, i64, i64, f64p]
        L.oracle_resize_pixel.argtypes = [u8p, i64, i64, i64, i64, i64, i64, i64]
        L.oracle_resize_pixel.restype = ctypes.c_double
        L.oracle_normalize.argtypes = [ctypes.c_double, ctypes.c_double, ctypes.c_double]
        L.oracle_normalize.restype = ctypes.c_double
        L.oracle_item_rows.argtypes = [i64, i64, i64, i64]
        L.oracle_item_rows.restype = i64
        L.oracle_preprocess_item.argtypes = [u8p, i64, i64, i64, i32p, i64, i64, i64, i64,
                                             f64p, f64p, f64p]
        L.oracle_item_row.argtypes = [u8p, i64, i64, i64, i32p, i64, i64, i64, i64,
                                      f64p, f64p, i64, f64p]
        L.oracle_patchify_item.argtypes = [u8p, i64, i64, i64, i32p, i64, i64, f64p, f64p, f64p]
        L.oracle_fixed_weights.argtypes = [i64, i64, i64, i64p, i64p, i32p, i64]
        L.oracle_resize_u8.argtypes = [u8p, i64, i64, i64, i64, u8p]
        L.oracle_resize_u8_item.argtypes = [u8p, i64, i64, i64, i32p, i64, i64, i64, i64, u8p]
        L.oracle_layout.argtypes = [i64, i64p, i64p, i64p, i64, i64p, i64p]
        L.oracle_position_ids.argtypes = [i64, i64p, i64p, i64p, i64, i64p, i64p, i64p, i64p]
        _lib = L
    return _lib


def _p(a: np.ndarray, ct):
    return a.ctypes.data_as(ctypes.POINTER(ct))


def _check(st: int, what: str):
    if st != OK:
        raise OracleError(st, what)


def smart_resize(height: int, width: int, factor: int = 32, min_pixels: int = 0,
                 max_pixels: int = 1 << 62) -> tuple[int, int]:
    h, w = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().oracle_smart_resize(height, width, factor, min_pixels, max_pixels,
                                     ctypes.byref(h), ctypes.byref(w)), "smart_resize")
    return h.value, w.value


def sample_uniform(total: int, n: int) -> np.ndarray:
    out = np.zeros(max(n, 1), np.int32)
    _check(lib().oracle_sample_uniform(total, n, _p(out, ctypes.c_int32)), "sample_uniform")
    return out[:n]


def sample_fps(total: int, video_fps: float, fps: float, min_frames: int = 4,
               max_frames: int = 768) -> np.ndarray:
    cnt = ctypes.c_int64()
    cap = max(total, 1)
    out = np.zeros(cap, np.int32)
    _check(lib().oracle_sample_fps(total, video_fps, fps, min_frames, max_frames,
                                   _p(out, ctypes.c_int32), cap, ctypes.byref(cnt)),
           "sample_fps")
    return out[:cnt.value].copy()


def keys_cubic(x: float) -> float:
    return lib().oracle_keys_cubic(x)


def filter_weights(n_in: int, n_out: int, i: int) -> tuple[int, np.ndarray]:
    """(window start, normalised fp64 weights) of output sample i."""
    cap = 8192
    w = np.zeros(cap, np.float64)
    lo, cnt = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().oracle_filter(n_in, n_out, i, ctypes.byref(lo), ctypes.byref(cnt),
                               _p(w, ctypes.c_double), cap), "filter")
    return lo.value, w[:cnt.value].copy()


def filter_table(n_in: int, n_out: int):
    """(lo[n_out], count[n_out], w[n_out][K]) with K the longest window."""
    k = lib().oracle_filter_max_taps(n_in, n_out)
    if k < 1:
        raise OracleError(ERR_ARG, "filter_max_taps")
    lo = np.zeros(n_out, np.int64)
    cnt = np.zeros(n_out, np.int64)
    w = np.zeros((n_out, k), np.float64)
    _check(lib().oracle_filter_table(n_in, n_out, _p(lo, ctypes.c_int64), _p(cnt, ctypes.c_int64),
                                     _p(w, ctypes.c_double), k), "filter_table")
    return lo, cnt, w


def resize_frame(frame: np.ndarray, h: int, w: int) -> np.ndarray:
    """frame uint8 [H][W][3] -> fp64 [3][h][w] (separable, no clamping)."""
    f = np.ascontiguousarray(frame, dtype=np.uint8)
    H, W, C = f.shape
    assert C == 3
    out = np.zeros((3, h, w), np.float64)
    _check(lib().oracle_resize_frame(_p(f, ctypes.c_uint8), H, W, h, w, _p(out, ctypes.c_double)),
           "resize_frame")
    return out


def resize_pixel(frame: np.ndarray, h: int, w: int, i: int, j: int, c: int) -> float:
    f = np.ascontiguousarray(frame, dtype=np.uint8)
    H, W, _ = f.shape
    return lib().oracle_resize_pixel(_p(f, ctypes.c_uint8), H, W, h, w, i, j, c)


def normalize(r: float, mean: float, std: float) -> float:
    return lib().oracle_normalize(r, mean, std)


def item_rows(n_idx: int, h: int, w: int, patch: int = 16) -> int:
    return lib().oracle_item_rows(n_idx, h, w, patch)


def row_width(patch: int = 16) -> int:
    """Values per merge-window row: 3 channels x 2 frames x patch x patch."""
    return 6 * patch * patch


def _item_args(frames, indices, mean, std):
    f = np.ascontiguousarray(frames, dtype=np.uint8)
    assert f.ndim == 4 and f.shape[3] == 3
    idx = np.ascontiguousarray(indices, dtype=np.int32)
    m = np.ascontiguousarray(np.asarray(mean, dtype=np.float64).reshape(3))
    s = np.ascontiguousarray(np.asarray(std, dtype=np.float64).reshape(3))
    return f, idx, m, s


def preprocess_item(frames: np.ndarray, indices, h: int, w: int, mean, std,
                    patch: int = 16) -> np.ndarray:
    """frames uint8 [N][H][W][3] -> fp64 rows [t*(h/P)*(w/P)][6*P*P]."""
    f, idx, m, s = _item_args(frames, indices, mean, std)
    n_src, H, W, _ = f.shape
    rows = np.zeros((item_rows(len(idx), h, w, patch), row_width(patch)), np.float64)
    _check(lib().oracle_preprocess_item(_p(f, ctypes.c_uint8), n_src, H, W, _p(idx, ctypes.c_int32),
                                        len(idx), h, w, patch, _p(m, ctypes.c_double),
                                        _p(s, ctypes.c_double), _p(rows, ctypes.c_double)),
           "preprocess_item")
    return rows


def patchify_item(frames: np.ndarray, indices, mean, std, patch: int = 16) -> np.ndarray:
    """Normalise + patchify only: frames uint8 [N][h][w][3], already at the
    target size -> fp64 rows [t*(h/P)*(w/P)][6*P*P]."""
    f, idx, m, s = _item_args(frames, indices, mean, std)
    n_src, h, w, _ = f.shape
    rows = np.zeros((item_rows(len(idx), h, w, patch), row_width(patch)), np.float64)
    _check(lib().oracle_patchify_item(_p(f, ctypes.c_uint8), n_src, h, w, _p(idx, ctypes.c_int32),
                                      len(idx), patch, _p(m, ctypes.c_double), _p(s, ctypes.c_double),
                                      _p(rows, ctypes.c_double)), "patchify_item")
    return rows


def fixed_weights(n_in: int, n_out: int, i: int) -> tuple[int, np.ndarray]:
    """(window start, int32 weights in units of 2^-22) of output i."""
    lo, n = ctypes.c_int64(), ctypes.c_int64()
    q = np.zeros(4096, np.int32)
    _check(lib().oracle_fixed_weights(n_in, n_out, i, ctypes.byref(lo), ctypes.byref(n),
                                      _p(q, ctypes.c_int32), 4096), "fixed_weights")
    return lo.value, q[:n.value].copy()


def resize_u8(frame: np.ndarray, h: int, w: int) -> np.ndarray:
    """Fixed-point resample of one uint8 [H][W][3] frame to uint8 [h][w][3]."""
    f = np.ascontiguousarray(frame, dtype=np.uint8)
    H, W, _ = f.shape
    out = np.zeros((h, w, 3), np.uint8)
    _check(lib().oracle_resize_u8(_p(f, ctypes.c_uint8), H, W, h, w, _p(out, ctypes.c_uint8)),
           "resize_u8")
    return out


def resize_u8_item(frames: np.ndarray, indices, h: int, w: int, patch: int = 16) -> np.ndarray:
    """The cache writer for one item: uint8 [n_idx][h][w][3]."""
    f = np.ascontiguousarray(frames, dtype=np.uint8)
    n_src, H, W, _ = f.shape
    idx = np.ascontiguousarray(indices, dtype=np.int32)
    out = np.zeros((len(idx), h, w, 3), np.uint8)
    _check(lib().oracle_resize_u8_item(_p(f, ctypes.c_uint8), n_src, H, W, _p(idx, ctypes.c_int32),
                                       len(idx), h, w, patch, _p(out, ctypes.c_uint8)), "resize_u8_item")
    return out


def item_row(frames: np.ndarray, indices, h: int, w: int, mean, std, rho: int,
             patch: int = 16) -> np.ndarray:
    """One output row by the direct 2D sum (fp64 [6*P*P])."""
    f, idx, m, s = _item_args(frames, indices, mean, std)
    n_src, H, W, _ = f.shape
    row = np.zeros(row_width(patch), np.float64)
    _check(lib().oracle_item_row(_p(f, ctypes.c_uint8), n_src, H, W, _p(idx, ctypes.c_int32),
                                 len(idx), h, w, patch, _p(m, ctypes.c_double), _p(s, ctypes.c_double),
                                 rho, _p(row, ctypes.c_double)), "item_row")
    return row


def layout(n_idx, h, w, patch: int = 16) -> tuple[np.ndarray, np.ndarray]:
    """(grid_thw [B][3], cu_seqlens [B+1]) as int64."""
    n = np.ascontiguousarray(n_idx, dtype=np.int64)
    hh = np.ascontiguousarray(h, dtype=np.int64)
    ww = np.ascontiguousarray(w, dtype=np.int64)
    B = len(n)
    g = np.zeros((B, 3), np.int64)
    cu = np.zeros(B + 1, np.int64)
    _check(lib().oracle_layout(B, _p(n, ctypes.c_int64), _p(hh, ctypes.c_int64),
                               _p(ww, ctypes.c_int64), patch, _p(g, ctypes.c_int64),
                               _p(cu, ctypes.c_int64)), "layout")
    return g, cu


def position_ids(n_idx, h, w, patch: int = 16):
    """(vit_pos int64 [rows][3], llm_pos int64 [rows/4][3], vit_cu int64 [S+1])."""
    n = np.ascontiguousarray(n_idx, dtype=np.int64)
    hh = np.ascontiguousarray(h, dtype=np.int64)
    ww = np.ascontiguousarray(w, dtype=np.int64)
    rows = int(sum(item_rows(int(a), int(b), int(c), patch) for a, b, c in zip(n, hh, ww)))
    slices = int(sum((int(a) + 1) // 2 for a in n))
    vit = np.zeros((rows, 3), np.int64)
    llm = np.zeros((rows // 4, 3), np.int64)
    cu = np.zeros(slices + 1, np.int64)
    ns = ctypes.c_int64()
    _check(lib().oracle_position_ids(len(n), _p(n, ctypes.c_int64), _p(hh, ctypes.c_int64),
                                     _p(ww, ctypes.c_int64), patch, _p(vit, ctypes.c_int64),
                                     _p(llm, ctypes.c_int64), _p(cu, ctypes.c_int64),
                                     ctypes.byref(ns)), "position_ids")
    assert ns.value == slices
    return vit, llm, cu
