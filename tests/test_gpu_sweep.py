"""Seeded random-shape GPU parity sweep through the C ABI against the oracle.

Each case is a small ragged batch of one to three items drawn from one of
eight shape families: downscales up to 6x, near-identity scales, mild
upscales, 2x upscales (eight open output rows), 3x-4x upscales (the general
kernel), extreme aspect ratios up to 200:1 in either direction, and images.
Sizes are odd as often as not, index lists are unsorted with repeats and
odd counts, and the cases alternate fp32 / bf16 output and patch 16 / 14.
Every output element is compared with the oracle; the NaN sentinel rows
past the batch must stay untouched.  The sweep is deterministic (one seed),
and stops at its first mismatch under `pytest -x`.
"""
import sys

import numpy as np
import pytest

import oracle
from oracle import compare
import paper_2604_16893_amd as vp
import workloads

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"
SEED = 2604_16893
KINDS = ("down", "near", "up", "up2", "strong_up", "wide", "tall", "image")
N_CASES = 48


def log(msg):
    print(f"[gpu-sweep] {msg}", flush=True)
    sys.stdout.flush()


def _item(rng, kind, F):
    """(n_src, H, W, indices, h, w) of one item of the given family."""
    if kind in ("wide", "tall"):
        ratio = int(rng.integers(50, 201))
        short, long_ = F, F * max(1, round(ratio))
        s = float(rng.uniform(0.8, 1.6))
        H, W = max(1, round(short * s) + int(rng.integers(-2, 3))), round(long_ * s) + int(rng.integers(-3, 4))
        h, w = short, long_
        if kind == "tall":
            H, W, h, w = W, H, w, h
    else:
        h, w = F * int(rng.integers(1, 9)), F * int(rng.integers(1, 9))
        lo, hi = {"down": (1.05, 6.0), "near": (0.85, 1.15), "up": (0.55, 0.95), "up2": (0.45, 0.55),
                  "strong_up": (0.25, 0.4), "image": (0.4, 3.0)}[kind]
        H = max(1, round(h * float(rng.uniform(lo, hi))) + int(rng.integers(-2, 3)))
        W = max(1, round(w * float(rng.uniform(lo, hi))) + int(rng.integers(-2, 3)))
    if kind == "image":
        return 1, H, W, [0], h, w
    n_src = int(rng.integers(1, 6))
    n_idx = int(rng.integers(1, 6))
    idx = rng.integers(0, n_src, n_idx).tolist()
    return n_src, H, W, idx, h, w


def _case(k):
    rng = np.random.default_rng([SEED, k])
    kind = KINDS[k % len(KINDS)]
    patch = 14 if k % 3 == 2 else 16
    dtype = "bf16" if k % 2 else "f32"
    n_items = int(rng.integers(1, 4))
    specs = [_item(rng, kind if j == 0 else KINDS[int(rng.integers(0, len(KINDS)))], 2 * patch)
             for j in range(n_items)]
    mean = tuple(float(x) for x in rng.uniform(0.3, 0.6, 3))
    std = tuple(float(x) for x in rng.uniform(0.2, 0.35, 3))
    return kind, patch, dtype, specs, mean, std


@pytest.mark.parametrize("k", range(N_CASES), ids=[f"{k}-{KINDS[k % len(KINDS)]}" for k in range(N_CASES)])
def test_random_shapes(k):
    kind, patch, dtype, specs, mean, std = _case(k)
    log(f"case {k} {kind} patch {patch} {dtype}: " +
        ", ".join(f"{n}x{H}x{W}->{h}x{w} idx {idx}" for n, H, W, idx, h, w in specs))
    items, host = [], []
    for j, (n_src, H, W, idx, h, w) in enumerate(specs):
        it = workloads.Item("video", n_src, H, W, "uniform", SEED % 100000 + 97 * k + j,
                            {"mode": "uniform", "n": 1})
        items.append((workloads.frames_torch(it, DEV), np.asarray(idx, np.int32), h, w))
        host.append(workloads.frames_np(it))
    vitems = [vp.Item(f, idx, h, w, patch) for f, idx, h, w in items]
    grid, cu, rows, ws = vp.vp_batch_layout(vitems)
    og, ocu = oracle.layout([len(i[1]) for i in items], [i[2] for i in items], [i[3] for i in items],
                            patch=patch)
    assert grid.tolist() == og.tolist() and cu.tolist() == ocu.tolist()
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    extra = 5
    out = torch.full((rows + extra, vp.row_width(patch)), float("nan"), dtype=tdt, device=DEV)
    work = torch.empty(ws, dtype=torch.uint8, device=DEV)
    vp.vp_preprocess_batch(vitems, mean, std, vp.VP_OUT_BF16 if dtype == "bf16" else vp.VP_OUT_F32,
                           out, work)
    torch.cuda.synchronize()
    assert torch.isnan(out[rows:].float()).all(), "rows past the batch were written"
    for j, (f, idx, h, w) in enumerate(items):
        ref = oracle.preprocess_item(host[j], idx, h, w, mean, std, patch=patch)
        t = out[cu[j]:cu[j + 1]]
        if dtype == "bf16":
            res = compare.check_bf16(t.view(torch.int16).cpu().numpy().view(np.uint16), ref)
        else:
            res = compare.check_f32(t.cpu().numpy(), ref)
        log(f"case {k} item {j}: {res}")
        assert res["ok"], f"case {k} item {j}: {res}"
