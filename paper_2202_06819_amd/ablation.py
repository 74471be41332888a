"""Ablation of the techniques on one MI355X (the study of Sec. 4.4, restated).

For each layer and each tile that has ablation instances, the same schedule
is timed with techniques switched off (``qconv_schedule.ablation``):

    3  baseline: lowered staging (every pixel once per filter tap) and int32
       accumulators through LDS to a separate requantise-and-pack step
    2  + duplicate-aware loading (Sec. 3.1): the input band, staged once
    1  + register-level packing (Sec. 3.2) alone, lowered staging kept
    0  both techniques (the normal kernels)

Accumulated speedup (Fig. 15): 3 -> 2 -> 0.  Marginal speedup of a technique
(Fig. 16): the time with only that technique switched off over the time
with both on.  Every output is checked against the default schedule's.

    python -m paper_2202_06819_amd.ablation --workload table1 --out ablation.jsonl
"""
from __future__ import annotations

import argparse
import json
import os
import sys

ABLATION_TILES = ("wide_b4_w4x1_f1x4_c64", "wide_b4_w8x1_f1x4_c64", "wide_b4_w4x1_f2x4_c64")
MASKS = (3, 2, 1, 0)


def ablate_layer(L, dev, reps: int = 50, rounds: int = 5, log=print) -> list[dict]:
    import torch
    from . import qconv, sweep
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import qconv_inputs as qi
    d = L.desc()
    t = qi.layer_tensors(970, 0, L)
    xp = qconv.pack(torch.from_numpy(t["x"]).to(dev), L.bits, L.x_signed)
    wp = qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
    e = L.epilogue
    kw = dict(requant=True, mult=torch.from_numpy(t["mult"]).to(dev), shift=e.shift, relu=e.relu,
              clamp=(e.lo, e.hi))
    ref = qconv.conv2d(d, xp, wp, tile=qconv.default_tile(d), **kw)
    names = {tt["name"]: tt["id"] for tt in qconv.tiles()}
    rows = []
    for tname in ABLATION_TILES:
        tid = names[tname]
        if qconv.tile_status(d, tid) != 0:
            continue
        wprep = qconv.prepare_filters(d, wp, tid)
        for mask in MASKS:
            sch = {"tile_id": tid, "ablation": mask}
            if qconv.schedule_status(d, sch) != 0:
                continue

            def make(stream=None, sch=sch):
                return qconv.Conv2dCall(d, xp, wprep, schedule=sch, stream=stream, **kw)

            out = make()()
            torch.cuda.synchronize()
            if not torch.equal(out, ref):
                raise RuntimeError(f"{L.name} {tname} ablation {mask}: output differs")
            us = sweep._time(make, reps, rounds)
            rows.append({"layer": L.name, "tile": tname, "ablation": mask, "us": round(us, 3)})
            log(json.dumps(rows[-1]))
    return rows


def summarize(rows: list[dict]) -> list[str]:
    """Accumulated and marginal speedups per (layer, tile) with all four masks."""
    by = {}
    for r in rows:
        by.setdefault((r["layer"], r["tile"]), {})[r["ablation"]] = r["us"]
    out = ["| layer | tile | baseline us | + duplicate-aware | + register packing | marginal: duplicate-aware | "
           "marginal: register packing |", "|---|---|---|---|---|---|---|"]
    for (layer, tile), m in by.items():
        if 0 not in m:
            continue
        base = m.get(3)
        base_s = f"{base:.2f}" if base else "n/a"
        acc1 = f"{base / m[2]:.2f}x ({m[2]:.2f} us)" if base and 2 in m else "n/a"
        acc2 = f"{base / m[0]:.2f}x ({m[0]:.2f} us)" if base else f"({m[0]:.2f} us)"
        dup = f"{m[1] / m[0]:.2f}x" if 1 in m else "n/a (lowered operand exceeds LDS)"
        pack = f"{m[2] / m[0]:.2f}x" if 2 in m else "n/a"
        out.append(f"| `{layer}` | `{tile}` | {base_s} | {acc1} | {acc2} | {dup} | {pack} |")
    return out


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description="technique ablation (see the module docstring)")
    ap.add_argument("--workload", default="table1")
    ap.add_argument("--out", required=True)
    ap.add_argument("--reps", type=int, default=50)
    ap.add_argument("--rounds", type=int, default=5)
    args = ap.parse_args(argv)
    import torch
    from .search import _layers
    dev = torch.device("cuda:0")
    rows = []
    with open(args.out, "a") as fh:
        def log(s):
            print(s, flush=True)
            fh.write(s + "\n")
            fh.flush()
        for L in _layers(args.workload):
            rows += ablate_layer(L, dev, args.reps, args.rounds, log)
    for line in summarize(rows):
        print(line, flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
