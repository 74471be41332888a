"""Ablation of the techniques on one MI355X (the study of Sec. 4.4, restated).

For each layer and each tile that has ablation instances, the same schedule
is timed with techniques switched off (``qconv_schedule.ablation``, a bit
mask of the techniques switched off):

    1  duplicate-aware loading (Sec. 3.1): without it every tile pixel is
       staged once per filter tap, as the lowered matrix
    2  register-level packing (Sec. 3.2): without it the int32 accumulators go
       through LDS to a separate requantise-and-pack step
    4  widening at staging: without it the 4-bit activations stay packed in
       LDS and every fragment is widened inside the MFMA loop

Accumulated speedup (Fig. 15): 7 (all off) -> 6 (+ duplicate-aware) -> 4
(+ register packing) -> 0 (+ widening at staging: the normal kernels).
Marginal speedup of a technique (Fig. 16): the time with only that technique
switched off (mask 1, 2 or 4) over the time with all on.  Every output is
checked against the default schedule's.

    python -m paper_2202_06819_amd.ablation --workload table1 --out ablation.jsonl
"""
from __future__ import annotations

import argparse
import json
import os
import sys

ABLATION_TILES = ("wide_b4_w4x1_f1x4_c64", "wide_b4_w8x1_f1x4_c64", "wide_b4_w4x1_f2x4_c64")
MASKS = (7, 6, 4, 0, 1, 2)
TECHNIQUES = ((1, "duplicate-aware"), (2, "register packing"), (4, "widening at staging"))


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
    """Accumulated and marginal speedups per (layer, tile)."""
    by = {}
    for r in rows:
        by.setdefault((r["layer"], r["tile"]), {})[r["ablation"]] = r["us"]
    out = ["| layer | tile | all off (mask 7) | + duplicate-aware (6) | + register packing (4) | "
           "+ widening at staging (0) | marginal: " + " | marginal: ".join(n for _, n in TECHNIQUES) + " |",
           "|---|---|---|---|---|---|---|---|---|"]

    def cell(m, mask, base):
        if mask not in m:
            return "n/a"
        return f"{m[mask]:.2f} us" + (f" ({base / m[mask]:.2f}x)" if base and mask != 7 else "")

    for (layer, tile), m in by.items():
        if 0 not in m:
            continue
        base = m.get(7)
        acc = " | ".join(cell(m, k, base) for k in (7, 6, 4, 0))
        marg = " | ".join(f"{m[b] / m[0]:.2f}x" if b in m else "n/a" for b, _ in TECHNIQUES)
        out.append(f"| `{layer}` | `{tile}` | {acc} | {marg} |")
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
