"""Seeded synthetic workloads for the preprocessing path (inputs only).

This module holds the five workload configurations and the seeded frame
generators that feed both the GPU library and the CPU oracle.  It contains
none of the preprocessing arithmetic (no sampling, resizing, normalisation or
patchification): every item carries only *parameters* (source shape, sampling
request, pixel budget or explicit target size), and each side computes the
rest itself.

The paper's own workloads -- its ~100K-video RL training set and the
throughput run over videos of up to 256 frames (Section 4.1, Section 4.3) --
are not available; these synthetic items stand in for them, using the
paper's preprocessing parameters (2 fps, <=128 or <=256 frames, per-frame
video budget, separate image budget) as scale references.

All pixel values come from one counter-based generator, the SplitMix64
output function (Steele, Lea and Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014): value_i = mix(seed + (i + 1) * 0x9E3779B97F4A7C15)
with mix(z) = z ^ z>>30, * 0xBF58476D1CE4E5B9, ^ >>27, * 0x94D049BB133111EB,
^ >>31 (all mod 2^64), where i is the byte offset of the pixel channel inside
its item.  The NumPy (host) and torch (device) versions below are
bit-identical, so a device-resident workload can be checked against host
copies of any of its frames.  Distributions use integers only:
  * uniform:   the low byte of value_i;
  * noise(s):  floor((b0 + b1 + b2 + b3 - 510) * s / 148), the sum of the four
               low bytes being approximately normal with sd 147.8;
  * gradient:  32 + floor(160 * (6 x (H-1) + 4 y (W-1)) / (10 (W-1)(H-1)))
               + floor(24 * ((f + 7 c) mod 16) / 15), plus noise(12), clipped;
  * rects:     clip(128 + noise(40)) background under six solid rectangles
               (sides 64..512, random RGB) moving by (vx, vy) in [-8, 8]
               pixels per frame with wrap-around.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB
_M64 = (1 << 64) - 1


def _signed(v: int) -> int:
    return v - (1 << 64) if v >= (1 << 63) else v


# --------------------------------------------------------------------------
# SplitMix64, NumPy (uint64) and torch (int64, two's complement) versions
# --------------------------------------------------------------------------

def splitmix64_np(counter: np.ndarray, seed: int) -> np.ndarray:
    """value_i for the uint64 array of counters i."""
    with np.errstate(over="ignore"):
        z = np.uint64(seed & _M64) + (counter.astype(np.uint64) + np.uint64(1)) * np.uint64(GAMMA)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(MIX1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(MIX2)
        z = z ^ (z >> np.uint64(31))
    return z


def _srl_t(z, k: int):
    return (z >> k) & ((1 << (64 - k)) - 1)


def splitmix64_torch(counter, seed: int):
    """Same as splitmix64_np on an int64 torch tensor (bit pattern of uint64)."""
    z = (counter + 1) * _signed(GAMMA) + _signed(seed & _M64)
    z = (z ^ _srl_t(z, 30)) * _signed(MIX1)
    z = (z ^ _srl_t(z, 27)) * _signed(MIX2)
    return z ^ _srl_t(z, 31)


def _byte_sum4(z):
    return (z & 255) + ((z >> 8) & 255) + ((z >> 16) & 255) + ((z >> 24) & 255)


# --------------------------------------------------------------------------
# Item and workload descriptions
# --------------------------------------------------------------------------

@dataclasses.dataclass
class Item:
    """One video or image: source shape, generator, and preprocessing request.

    sample: {"mode": "uniform", "n": k} or {"mode": "fps", "video_fps": ..,
    "fps": .., "min_frames": .., "max_frames": ..}.
    dims: explicit target (h, w), or None to take smart_resize under
    [min_pixels, max_pixels] with factor 32.
    """
    kind: str
    n_src: int
    H: int
    W: int
    gen: str
    seed: int
    sample: dict
    dims: Optional[tuple] = None
    max_pixels: Optional[int] = None
    min_pixels: int = 0
    rects: Optional[list] = None
    patch: int = 16          # 16, or 14 for the Qwen2/2.5-VL geometry (smart_resize factor 2 * patch)

    @property
    def frame_bytes(self) -> int:
        return self.H * self.W * 3


@dataclasses.dataclass
class Workload:
    name: str
    items: list
    mean: tuple
    std: tuple
    out_dtype: str  # "f32" or "bf16"
    note: str = ""


MEAN_HALF = (0.5, 0.5, 0.5)
STD_HALF = (0.5, 0.5, 0.5)
MEAN_C4 = (0.481, 0.458, 0.408)
STD_C4 = (0.269, 0.261, 0.276)


def _rects(seed: int, H: int, W: int, n: int = 6) -> list:
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        out.append(dict(
            w=int(rng.integers(64, 513)), h=int(rng.integers(64, 513)),
            color=[int(v) for v in rng.integers(0, 256, size=3)],
            x0=int(rng.integers(0, W)), y0=int(rng.integers(0, H)),
            vx=int(rng.integers(-8, 9)), vy=int(rng.integers(-8, 9))))
    return out


def config(k: int) -> Workload:
    """The five workload configurations (0: tiny, 4: rollout-sized batch)."""
    if k == 0:
        return Workload(
            "c0: 1 video, 16x240x320 -> uniform 8 -> 128x160, fp32",
            [Item("video", 16, 240, 320, "uniform", 0, {"mode": "uniform", "n": 8},
                  dims=(128, 160))],
            MEAN_HALF, STD_HALF, "f32")
    if k == 1:
        return Workload(
            "c1: 1 video, 256x480x854 -> fps 8->2 (64) -> smart_resize@230400 (352x640), fp32",
            [Item("video", 256, 480, 854, "gradnoise", 1,
                  {"mode": "fps", "video_fps": 8.0, "fps": 2.0, "min_frames": 4,
                   "max_frames": 128}, max_pixels=230400)],
            MEAN_HALF, STD_HALF, "f32")
    if k == 2:
        return Workload(
            "c2: 1 video, 512x1080x1920 -> uniform 128 -> 448x800, bf16",
            [Item("video", 512, 1080, 1920, "rects", 2, {"mode": "uniform", "n": 128},
                  dims=(448, 800), rects=_rects(2, 1080, 1920))],
            MEAN_HALF, STD_HALF, "bf16")
    if k == 3:
        rng = np.random.default_rng(3)
        items = []
        res = [(360, 640), (480, 854), (720, 1280)]
        for v in range(12):
            H, W = res[int(rng.integers(0, 3))]
            n = 2 * int(rng.integers(16, 129))
            N = int(rng.integers(n, 2 * n + 1))
            items.append(Item("video", N, H, W, "gradnoise", 0,
                              {"mode": "uniform", "n": n}, max_pixels=200704))
        for _ in range(20):
            H = int(rng.integers(256, 1025))
            W = int(rng.integers(256, 1025))
            items.append(Item("image", 1, H, W, "gradnoise", 0,
                              {"mode": "uniform", "n": 1}, max_pixels=1003520,
                              min_pixels=65536))
        order = rng.permutation(len(items))
        items = [items[int(o)] for o in order]
        for b, it in enumerate(items):
            it.seed = 3000 + b
        return Workload(
            "c3: ragged 12 videos (360x640|480x854|720x1280, 32-256 frames, @200704) "
            "+ 20 images (256..1024 square range, @1003520), bf16",
            items, MEAN_C4, STD_C4, "bf16")
    if k == 4:
        items = [Item("video", 256, 720, 1280, "gradnoise", 4000 + v,
                      {"mode": "uniform", "n": 256}, max_pixels=122880)
                 for v in range(64)]
        return Workload(
            "c4: 64 videos x 256 frames 720x1280 -> 256x448 (smart_resize@122880), bf16",
            items, MEAN_C4, STD_C4, "bf16")
    raise ValueError(k)


def patch14_config() -> Workload:
    """Configuration 4's frames in the Qwen2/2.5-VL geometry: patch 14, so
    smart_resize with factor 28 under the same 122,880 px budget gives
    252x448, and rows hold 3 x 2 x 14 x 14 = 1176 values."""
    items = [Item("video", 256, 720, 1280, "gradnoise", 4000 + v, {"mode": "uniform", "n": 256},
                  max_pixels=122880, patch=14)
             for v in range(64)]
    return Workload("q4: 64 videos x 256 frames 720x1280 -> 252x448 (smart_resize factor 28 "
                    "@122880), patch 14, rows of 1176, bf16", items, MEAN_C4, STD_C4, "bf16")


def patchify_config() -> Workload:
    """The cached counterpart of configuration 4: the same 64 x 256 frames,
    already sampled and resized to 256x448 (what an offline cache holds), to
    be normalised and patchified only."""
    items = [Item("video", 256, 256, 448, "gradnoise", 5000 + v, {"mode": "uniform", "n": 256},
                  dims=(256, 448))
             for v in range(64)]
    return Workload("p4: 64 videos x 256 cached frames 256x448, normalise + patchify only, bf16",
                    items, MEAN_C4, STD_C4, "bf16")


# --------------------------------------------------------------------------
# Frame generation
# --------------------------------------------------------------------------

def _gradient_np(f, y, x, c, H, W):
    dy = max(H - 1, 1)
    dx = max(W - 1, 1)
    return (32 + (160 * (6 * x * dy + 4 * y * dx)) // (10 * dx * dy)
            + (24 * ((f + 7 * c) % 16)) // 15)


def frames_np(item: Item, frame_ids=None) -> np.ndarray:
    """Host copy of the requested source frames, uint8 [len(ids)][H][W][3]."""
    ids = list(range(item.n_src)) if frame_ids is None else [int(v) for v in frame_ids]
    H, W = item.H, item.W
    out = np.empty((len(ids), H, W, 3), np.uint8)
    y = np.arange(H, dtype=np.int64).reshape(H, 1, 1)
    x = np.arange(W, dtype=np.int64).reshape(1, W, 1)
    c = np.arange(3, dtype=np.int64).reshape(1, 1, 3)
    local = ((y * W + x) * 3 + c)
    for k, f in enumerate(ids):
        cnt = (local + f * item.frame_bytes).astype(np.uint64)
        z = splitmix64_np(cnt, item.seed)
        if item.gen == "uniform":
            v = (z & np.uint64(255)).astype(np.int64)
        elif item.gen == "gradnoise":
            s = _byte_sum4(z).astype(np.int64)
            v = _gradient_np(f, y, x, c, H, W) + ((s - 510) * 12) // 148
        elif item.gen == "rects":
            s = _byte_sum4(z).astype(np.int64)
            v = np.broadcast_to(128 + ((s - 510) * 40) // 148, (H, W, 3)).copy()
            for r in item.rects:
                inside = ((((x[..., 0] - r["x0"] - r["vx"] * f) % W) < r["w"])
                          & (((y[..., 0] - r["y0"] - r["vy"] * f) % H) < r["h"]))
                v[inside] = np.asarray(r["color"], np.int64)
        else:
            raise ValueError(item.gen)
        out[k] = np.clip(v, 0, 255).astype(np.uint8)
    return out


def frames_torch(item: Item, device, chunk: int = 16, out=None):
    """Device copy of all source frames, uint8 [n_src][H][W][3] (torch)."""
    import torch
    H, W = item.H, item.W
    if out is None:
        out = torch.empty((item.n_src, H, W, 3), dtype=torch.uint8, device=device)
    y = torch.arange(H, dtype=torch.int64, device=device).view(1, H, 1, 1)
    x = torch.arange(W, dtype=torch.int64, device=device).view(1, 1, W, 1)
    c = torch.arange(3, dtype=torch.int64, device=device).view(1, 1, 1, 3)
    local = (y * W + x) * 3 + c
    dy = max(H - 1, 1)
    dx = max(W - 1, 1)
    for f0 in range(0, item.n_src, chunk):
        nf = min(chunk, item.n_src - f0)
        f = torch.arange(f0, f0 + nf, dtype=torch.int64, device=device).view(nf, 1, 1, 1)
        z = splitmix64_torch(local + f * item.frame_bytes, item.seed)
        if item.gen == "uniform":
            v = z & 255
        elif item.gen == "gradnoise":
            s = _byte_sum4(z)
            g = (32 + torch.div(160 * (6 * x * dy + 4 * y * dx), 10 * dx * dy, rounding_mode="floor")
                 + torch.div(24 * torch.remainder(f + 7 * c, 16), 15, rounding_mode="floor"))
            v = g + torch.div((s - 510) * 12, 148, rounding_mode="floor")
        elif item.gen == "rects":
            s = _byte_sum4(z)
            v = (128 + torch.div((s - 510) * 40, 148, rounding_mode="floor")).expand(nf, H, W, 3).clone()
            for r in item.rects:
                inside = ((torch.remainder(x[..., 0] - r["x0"] - r["vx"] * f[..., 0], W) < r["w"])
                          & (torch.remainder(y[..., 0] - r["y0"] - r["vy"] * f[..., 0], H) < r["h"]))
                col = torch.tensor(r["color"], dtype=torch.int64, device=device)
                v = torch.where(inside.unsqueeze(-1), col.view(1, 1, 1, 3), v)
        else:
            raise ValueError(item.gen)
        out[f0:f0 + nf] = torch.clamp(v, 0, 255).to(torch.uint8)
        del z, v
    return out
