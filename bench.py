#!/usr/bin/env python3
"""Throughput of the video-frame preprocessing path on one MI355X.

Workload (default, the rollout-sized batch): 64 videos x 256 decoded frames of
720x1280 uint8 RGB, resident in HBM (45.3 GB), each frame resampled to
256x448 (smart_resize under 122880 px), normalised with per-channel
mean/std (0.481, 0.458, 0.408)/(0.269, 0.261, 0.276) and patchified into
3,670,016 merge-window rows of 1536 bfloat16 values, on one stream.

One step is one pass of the whole path over the batch: per item the target
size (vp_smart_resize_dims) and the frame indices (vp_sample_indices) on the
host, then vp_preprocess_batch (host plan and filter tables, one plan upload,
the resampling/normalise/patchify kernel) on the stream.  W untimed warm-up
steps, then K steps timed with a synchronize on both sides.  Prints one JSON
line on stdout; progress goes to stderr.

value      = sampled source frames per second over the K timed steps.
roofline   = algorithmic HBM bytes of one call (every sampled u8 frame read
             once + every output row written once) / the mean device time of
             the call's kernels, from HIP events that the library records on
             the stream the kernels run on (vp_set_kernel_events).
cpu_baseline = the CPU oracle (double precision, unmodified) on a bounded
             sample of the same workload, on this host's cores.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_sha() -> str:
    h = hashlib.sha256()
    for name in ("vp_kernels.hip", "vp_plan.h"):
        with open(os.path.join(ROOT, "paper_2604_16893_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def counter_traffic(workload_tag: str, sha: str):
    """HBM bytes per call from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"counters_{workload_tag}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("kernel_sha") != sha:
        return None
    return d.get("hbm_bytes_per_call")


def cpu_baseline(wl, frames_dev, planned, patch_only=False, resize_only=False, budget_s=12.0):
    """The oracle, item by item in workload order, until `budget_s` seconds of
    oracle time have been spent (or the workload is done).  Each item's frame
    pairs are copied to the host and spread over a thread pool (ctypes
    releases the GIL); only the oracle calls are timed."""
    import concurrent.futures as cf

    import numpy as np

    import oracle
    oracle.lib()
    cores = min(16, os.cpu_count() or 1)
    frames_count = pairs = items = 0
    spent = 0.0
    with cf.ThreadPoolExecutor(max_workers=cores) as ex:
        for b in range(len(frames_dev)):
            h, w, idx = planned[b]
            padded = list(idx) + ([idx[-1]] if len(idx) % 2 else [])
            host = frames_dev[b].cpu().numpy()
            jobs = [(np.ascontiguousarray(host[[padded[2 * tt], padded[2 * tt + 1]]]), h, w)
                    for tt in range(len(padded) // 2)]
            del host
            t0 = time.perf_counter()
            if resize_only:
                list(ex.map(lambda j: oracle.resize_u8_item(j[0], [0, 1], j[1], j[2]), jobs))
            elif patch_only:
                list(ex.map(lambda j: oracle.patchify_item(j[0], [0, 1], wl.mean, wl.std), jobs))
            else:
                list(ex.map(lambda j: oracle.preprocess_item(j[0], [0, 1], j[1], j[2], wl.mean,
                                                             wl.std, patch=wl.items[0].patch), jobs))
            spent += time.perf_counter() - t0
            frames_count += len(idx)
            pairs += len(jobs)
            items += 1
            if spent >= budget_s:
                break
    return dict(value=round(frames_count / spent, 1), unit="frames/s", cores=cores, kind="oracle",
                sample=f"first {items} of {len(frames_dev)} items of the same workload "
                       f"({frames_count} sampled frames, {pairs} frame pairs), fp64 C oracle, "
                       f"{spent:.1f} s of oracle wall time on {cores} threads")


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", type=int, default=4, choices=range(5),
                    help="workload configuration (4 = 64x256 frames 720x1280, the default)")
    ap.add_argument("--patchify", action="store_true",
                    help="time the normalise+patchify-only entry on the cached counterpart of "
                         "workload 4 (64 x 256 frames already at 256x448) instead")
    ap.add_argument("--resize", action="store_true",
                    help="time the uint8 cache writer (fixed-point resize only) on the workload")
    ap.add_argument("--positions", action="store_true",
                    help="time the position tables (ViT rows, LLM windows) of the workload's rows")
    ap.add_argument("--patch", type=int, default=16, choices=(14, 16),
                    help="14: the Qwen2/2.5-VL geometry on workload 4's frames (252x448, rows of 1176)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run plain 1 GiB device-to-device copies (twice) before the steps, "
                         "to calibrate rocprofv3 FETCH_SIZE / WRITE_SIZE against known bytes")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}): "
              "the path shards by item with no exchange, and this build runs on a single device.",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2604_16893_amd as vp
    import workloads

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    vp.lib()
    dev = torch.device("cuda:0")
    props = torch.cuda.get_device_properties(dev)
    log(f"device {props.name} {getattr(props, 'gcnArchName', '')} CUs={props.multi_processor_count} "
        f"mem={props.total_memory / 2**30:.0f} GiB")

    if args.patch == 14:
        wl = workloads.patch14_config()
    else:
        wl = workloads.patchify_config() if args.patchify else workloads.config(args.workload)
    entry = vp.vp_patchify_batch if args.patchify else vp.vp_preprocess_batch
    log(f"workload {wl.name}")
    t0 = time.perf_counter()
    frames = [workloads.frames_torch(it, dev, chunk=32) for it in wl.items]
    torch.cuda.synchronize()
    log(f"input generated in {time.perf_counter() - t0:.1f} s "
        f"({sum(f.numel() for f in frames) / 1e9:.2f} GB)")

    def plan_items():
        vitems, planned = [], []
        for it, fr in zip(wl.items, frames):
            if it.dims is not None:
                h, w = it.dims
            else:
                h, w = vp.vp_smart_resize_dims(it.H, it.W, 2 * it.patch, it.min_pixels, it.max_pixels)
            s = it.sample
            if s["mode"] == "uniform":
                idx = vp.vp_sample_indices(it.n_src, vp.VP_SAMPLE_UNIFORM, s["n"])
            else:
                idx = vp.vp_sample_indices(it.n_src, vp.VP_SAMPLE_FPS, 0, s["video_fps"], s["fps"],
                                           s["min_frames"], s["max_frames"])
            vitems.append(vp.Item(fr, idx, h, w, it.patch))
            planned.append((h, w, idx))
        return vitems, planned

    vitems, planned = plan_items()
    code = vp.VP_OUT_BF16 if wl.out_dtype == "bf16" else vp.VP_OUT_F32
    if args.resize:
        frame_off, ws_bytes = vp.vp_resize_layout(vitems)
        rows = 0
        out = torch.empty(int(frame_off[-1]), dtype=torch.uint8, device=dev)
    elif args.positions:
        grid, cu, rows, ws_bytes = vp.vp_batch_layout(vitems)
        out = torch.empty((rows, 3), dtype=torch.int32, device=dev)
        out_llm = torch.empty((rows // 4, 3), dtype=torch.int32, device=dev)
    else:
        grid, cu, rows, ws_bytes = vp.vp_batch_layout(vitems)
        out = torch.empty((rows, vp.row_width(wl.items[0].patch)),
                          dtype=torch.bfloat16 if code == vp.VP_OUT_BF16 else torch.float32, device=dev)
    work = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    n_frames = sum(len(p[2]) for p in planned)
    in_bytes = sum(len(p[2]) * it.frame_bytes for p, it in zip(planned, wl.items))
    out_bytes = out.numel() * out.element_size()
    if args.positions:   # no frame is read; both tables are written
        in_bytes = 0
        out_bytes += out_llm.numel() * out_llm.element_size()
    alg_bytes = in_bytes + out_bytes
    log(f"{n_frames} frames, {rows} rows, algorithmic bytes {alg_bytes / 1e9:.3f} GB "
        f"(in {in_bytes / 1e9:.3f}, out {out_bytes / 1e9:.3f})")

    if args.copy_probe:
        src = torch.ones(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
            torch.bitwise_not(src, out=dst)
        torch.cuda.synchronize()
        log("copy probe: 2 x (1 GiB copy_ + 1 GiB bitwise_not), each reads and writes 2^30 bytes")
        del src, dst

    def step():
        items, _ = plan_items()
        if args.resize:
            vp.vp_resize_batch(items, out, work, stream)
        elif args.positions:
            vp.vp_position_ids(items, out, out_llm, work, stream)
        else:
            entry(items, wl.mean, wl.std, code, out, work, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warm-up done ({args.warmup} steps)")

    # Per timed step: events around the whole call (plan + upload + kernels)
    # and, recorded by the library itself, around its kernels alone.
    def pair():
        return torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    call_evs = [pair() for _ in range(args.steps)]
    kern_evs = [pair() for _ in range(args.steps)]
    for a, b in kern_evs:          # HIP events exist once recorded
        a.record(stream)
        b.record(stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        call_evs[k][0].record(stream)
        vp.vp_set_kernel_events(*kern_evs[k])
        step()
        call_evs[k][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    call_ms = [a.elapsed_time(b) for a, b in call_evs]
    kern_ms = [a.elapsed_time(b) for a, b in kern_evs]
    mean_kern_ms = sum(kern_ms) / len(kern_ms)
    ms_per_step = wall * 1e3 / args.steps
    value = n_frames * args.steps / wall
    achieved = alg_bytes / (mean_kern_ms * 1e-3) / 1e9
    log(f"{ms_per_step:.3f} ms/step wall; call {sum(call_ms) / len(call_ms):.3f} ms mean; "
        f"kernels {mean_kern_ms:.3f} ms mean (min {min(kern_ms):.3f}, max {max(kern_ms):.3f}); "
        f"{value:,.0f} frames/s; {achieved:,.0f} GB/s algorithmic "
        f"({achieved / HBM_PEAK_GBPS:.1%} of 8 TB/s)")
    log("kernel ms per step: " + " ".join(f"{t:.3f}" for t in kern_ms))

    tag = "q4" if args.patch == 14 else (
        "p4" if args.patchify else (f"r{args.workload}" if args.resize else
                                    (f"i{args.workload}" if args.positions else f"c{args.workload}")))
    sha = kernel_source_sha()
    traffic = counter_traffic(tag, sha)

    baseline = None
    if not args.no_cpu_baseline and not args.positions:
        log("timing the CPU oracle on a bounded sample")
        baseline = cpu_baseline(wl, frames, planned, patch_only=args.patchify, resize_only=args.resize)
        log(f"cpu baseline {baseline}")

    rec = {
        "metric": "preprocessed frames/s and achieved HBM GB/s (% of MI355X peak) per config",
        "value": round(value, 1),
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i32" if (args.resize or args.positions) else "f32",
        "data": "synthetic (seeded SplitMix64 frames resident in HBM)",
        "config": {
            "workload": wl.name + ("; uint8 cache writer (fixed-point resize only)" if args.resize else
                                   "; position tables only" if args.positions else ""),
            "items": len(wl.items),
            "frames": n_frames,
            "rows": rows,
            "out_dtype": "u8" if args.resize else ("i32" if args.positions else wl.out_dtype),
            "mean": list(wl.mean),
            "std": list(wl.std),
            "algorithmic_bytes": alg_bytes,
            "kernel_sha": sha,
        },
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
            "kernel_ms": round(mean_kern_ms, 4),
        },
        "cpu_baseline": baseline,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
