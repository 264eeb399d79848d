"""Write tests/golden/plan_configs.json from the CPU oracle only.

For each of the five synthetic workloads this records what the oracle derives
from the workload parameters: the per-item target size (smart_resize under
the item's budget, Section 3.1.1 / 3.1.2 / 4.1 of arXiv 2604.16893), the
sampled frame indices (Section 3.1.1 cache key fps / max_frames), the
per-item grid (t, h/16, w/16) and the row-offset table (Section 3.1.1:
identical video_grid_thw in every stage), and the longest filter window of
each axis.  The file is a regression anchor for the oracle and an expected
value for the GPU library's host planning.

Run:  python tests/golden/make_golden.py
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle      # noqa: E402
import workloads   # noqa: E402


def plan(k: int) -> dict:
    wl = workloads.config(k)
    items = []
    for it in wl.items:
        if it.dims is not None:
            h, w = it.dims
        else:
            h, w = oracle.smart_resize(it.H, it.W, 32, it.min_pixels, it.max_pixels)
        s = it.sample
        if s["mode"] == "uniform":
            idx = oracle.sample_uniform(it.n_src, s["n"])
        else:
            idx = oracle.sample_fps(it.n_src, s["video_fps"], s["fps"], s["min_frames"],
                                    s["max_frames"])
        items.append(dict(n_src=it.n_src, H=it.H, W=it.W, h=int(h), w=int(w),
                          indices=[int(v) for v in idx],
                          taps_y=int(oracle.filter_table(it.H, h)[2].shape[1]),
                          taps_x=int(oracle.filter_table(it.W, w)[2].shape[1])))
    g, cu = oracle.layout([len(i["indices"]) for i in items], [i["h"] for i in items],
                          [i["w"] for i in items])
    return dict(name=wl.name, items=items, grid_thw=g.tolist(), cu_seqlens=cu.tolist())


def main():
    oracle.build(force=False)
    out = {"source": "oracle/ via tests/golden/make_golden.py",
           "configs": [plan(k) for k in range(5)]}
    with open(os.path.join(HERE, "plan_configs.json"), "w") as f:
        json.dump(out, f, separators=(",", ":"))
        f.write("\n")


if __name__ == "__main__":
    main()
