"""Tile-configuration sweep: the schedule search space of Sec. 4.1, measured
exhaustively on the GPU (the "Exhaustive" row of Table 1, restated for the
compiled gfx950 tile space).

For each convolution shape and every compiled tile that can run it:
  1. run it and check that its output bytes equal those of a reference tile
     (integer sums have one value, so every tile must agree);
  2. time it with HIP events over back-to-back launches (median of rounds);
  3. append one JSON line to the results file (the run is resumable: pairs
     already in the file are skipped).
The fastest tile per shape goes into the tuned table that qconv2d callers use
when they pass tile -1 through :func:`tuned_tile`.

    python -m paper_2202_06819_amd.sweep --workload 4 --out sweep_w4.jsonl
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys

import torch

from . import qconv

TUNED_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tuned_tiles.json")
INT8_PEAK_TOPS = 5000.0


def shape_key(d: dict, requant: bool = True) -> str:
    nb = int(d.get("nb", 0))
    return ("n{n}_h{h}_w{w}_c{c}_k{k}_r{r}_s{s}_st{stride_h}x{stride_w}_p{pad_h}x{pad_w}_b{bits}_xs{x_signed}"
            "_ws{w_signed}".format(**d) + (f"_nb{nb}" if nb > 1 else "") + ("_rq" if requant else "_raw"))


_tuned_cache = None


def tuned_table() -> dict:
    global _tuned_cache
    if _tuned_cache is None:
        _tuned_cache = json.load(open(TUNED_PATH)) if os.path.exists(TUNED_PATH) else {}
    return _tuned_cache


def tuned_config(d: dict, requant: bool = True) -> tuple[int, int]:
    """(tile id, split-K factor) the sweep found fastest for this shape, else the
    library's built-in tile without a split."""
    entry = tuned_table().get(shape_key(d, requant))
    if isinstance(entry, str):
        entry = {"tile": entry, "splits": 1}
    if entry:
        for t in qconv.tiles():
            if t["name"] == entry["tile"] and qconv.tile_status(d, t["id"]) == 0:
                splits = int(entry.get("splits", 1))
                if splits <= max(1, qconv.max_splits(d, t["id"])):
                    return t["id"], splits
    return qconv.default_tile(d), 1


def tuned_tile(d: dict, requant: bool = True) -> int:
    """The swept best tile id for this shape (the built-in choice when unswept)."""
    return tuned_config(d, requant)[0]


def proj_key(d: dict, requant: bool = True) -> str:
    """Tuned-table key of a 3x3 layer with its 1x1 projection fused in."""
    return shape_key(d, requant) + "_proj"


def tuned_proj_config(d: dict, requant: bool = True) -> tuple[int, int]:
    """(tile id, split-K factor) the sweep found fastest for the 3x3 layer `d`
    with a fused projection (the library's built-in tile without a split when
    unswept)."""
    entry = tuned_table().get(proj_key(d, requant))
    if entry:
        for t in qconv.tiles():
            if t["name"] == entry["tile"] and qconv.proj_tile_status(d, t["id"]) == 0:
                splits = int(entry.get("splits", 1))
                if splits <= max(1, qconv.max_splits(d, t["id"])):
                    return t["id"], splits
    return qconv.proj_default_tile(d), 1


def tuned_proj_tile(d: dict, requant: bool = True) -> int:
    """The swept best tile for the 3x3 layer `d` with a fused projection."""
    return tuned_proj_config(d, requant)[0]


def split_choices(d: dict, tile: int) -> list[int]:
    """Split-K factors worth timing: 1 and the powers of two up to the chunk count."""
    top = max(1, qconv.max_splits(d, tile))
    out, s = [1], 2
    while s <= top:
        out.append(s)
        s *= 2
    return out


def _time(make_call, reps: int, rounds: int) -> float:
    """Median microseconds per launch: a graph of `reps` back-to-back launches
    (calls built by make_call(stream) for the capture stream) replayed `rounds`
    times, timed with HIP events on the replaying stream."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        call = make_call(s)
        call()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for _ in range(reps):
                call()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    res = []
    for _ in range(rounds):
        torch.cuda.synchronize()
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        res.append(e0.elapsed_time(e1) * 1000.0 / reps)
    return statistics.median(res)


def sweep_layer(d: dict, x: torch.Tensor, w: torch.Tensor, mult: torch.Tensor | None, *, shift=20, relu=True,
                clamp=(0, 15), reps=100, rounds=5, done=frozenset(), log=print,
                expected: torch.Tensor | None = None) -> list[dict]:
    """Measure every valid tile on one shape; returns result rows.  Every
    candidate's output must equal `expected` (a caller's reference output, e.g.
    a test's), or else the built-in tile's output from the packed filters."""
    requant = mult is not None
    key = shape_key(d, requant)
    info = qconv.layout(d)
    ops = 2 * info["macs"]
    default = qconv.default_tile(d)
    if expected is None:
        ref_call = qconv.Conv2dCall(d, x, w, requant=requant, mult=mult, shift=shift, relu=relu, clamp=clamp,
                                    tile=default)
        ref = ref_call().clone()   # packed filters, default tile
    else:
        ref = expected.to(x.device)
    rows = []
    for t in qconv.tiles():
        if qconv.tile_status(d, t["id"]) != 0:
            continue
        wprep = qconv.prepare_filters(d, w, t["id"])   # offline filter layout for this tile
        for splits in split_choices(d, t["id"]):
            if (key, t["name"], splits) in done:
                continue
            ws = qconv.make_workspace(d, t["id"], splits, x.device)

            def make(stream=None, tid=t["id"], splits=splits, ws=ws):
                return qconv.Conv2dCall(d, x, wprep, requant=requant, mult=mult, shift=shift, relu=relu,
                                        clamp=clamp, tile=tid, prepared=True, splits=splits, workspace=ws,
                                        stream=stream)

            out = make()()
            torch.cuda.synchronize()
            same = out.shape == ref.shape and bool(torch.equal(out.view(ref.dtype), ref))
            us = _time(make, reps, rounds)
            tops = ops / (us * 1e-6) / 1e12
            row = {"shape": key, "tile": t["name"], "tile_id": t["id"], "splits": splits,
                   "default": t["id"] == default and splits == 1, "us": round(us, 3), "tops": round(tops, 2),
                   "pct_int8_peak": round(100 * tops / INT8_PEAK_TOPS, 3), "identical": same}
            rows.append(row)
            log(json.dumps(row))
            if not same:
                raise RuntimeError(f"tile {t['name']} splits {splits} output differs from the reference on {key}")
    return rows


def sweep_proj_layer(d: dict, x: torch.Tensor, w3: torch.Tensor, w1: torch.Tensor, mult: torch.Tensor | None,
                     mult2: torch.Tensor | None, *, shift=20, shift2=20, relu=True, relu2=False, clamp=(0, 15),
                     reps=100, rounds=5, done=frozenset(), log=print, expected=None) -> list[dict]:
    """Every tile with a projection instance, and each of its split-K factors,
    on a 3x3 layer with its 1x1 projection fused in (packed filters w3 and w1);
    both outputs of each must equal `expected` = (y, y_proj), or else the
    built-in tile's."""
    requant = mult is not None
    key = proj_key(d, requant)
    ops = 2 * qconv.layout(d)["macs"] + 2 * qconv.layout(qconv.proj_desc(d))["macs"]
    default = qconv.proj_default_tile(d)
    kw = dict(requant=True, mult=mult, shift=shift, relu=relu, clamp=clamp,
              proj=dict(mult=mult2, shift=shift2, relu=relu2, clamp=clamp)) if requant else {}

    def make_for(tid, wprep, stream=None, splits=1, ws=None):
        return qconv.ProjConv2dCall(d, x, wprep, tile=tid, stream=stream, splits=splits, workspace=ws, **kw)

    if expected is None:
        y, yp = make_for(default, qconv.prepare_filters_proj(d, w3, w1, default))()
        ref = (y.clone(), yp.clone())
    else:
        ref = tuple(e.to(x.device) for e in expected)
    rows = []
    for t in qconv.tiles():
        if qconv.proj_tile_status(d, t["id"]) != 0:
            continue
        wprep = None
        for splits in split_choices(d, t["id"]):
            if (key, t["name"], splits) in done:
                continue
            if wprep is None:
                wprep = qconv.prepare_filters_proj(d, w3, w1, t["id"])
            nws = qconv.proj_workspace_bytes(d, t["id"], splits)
            ws = torch.zeros(nws, dtype=torch.uint8, device=x.device) if nws else None
            y, yp = make_for(t["id"], wprep, splits=splits, ws=ws)()
            torch.cuda.synchronize()
            same = all(o.shape == r.shape and bool(torch.equal(o.view(r.dtype), r)) for o, r in zip((y, yp), ref))
            us = _time(lambda stream, tid=t["id"], wprep=wprep, splits=splits, ws=ws:
                       make_for(tid, wprep, stream, splits, ws), reps, rounds)
            tops = ops / (us * 1e-6) / 1e12
            row = {"shape": key, "tile": t["name"], "tile_id": t["id"], "splits": splits,
                   "default": t["id"] == default and splits == 1, "us": round(us, 3), "tops": round(tops, 2),
                   "pct_int8_peak": round(100 * tops / INT8_PEAK_TOPS, 3), "identical": same}
            rows.append(row)
            log(json.dumps(row))
            if not same:
                raise RuntimeError(f"tile {t['name']} splits {splits} (fused projection) output differs from the "
                                   f"reference on {key}")
    return rows


def best_per_shape(rows: list[dict]) -> dict:
    best = {}
    for r in rows:
        if r["shape"] not in best or r["us"] < best[r["shape"]]["us"]:
            best[r["shape"]] = r
    return best


def main(argv=None) -> int:
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import qconv_inputs as qi

    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", type=int, action="append", required=True, help="workload id (repeatable)")
    ap.add_argument("--out", required=True, help="JSONL results file (appended; resumable)")
    ap.add_argument("--reps", type=int, default=100)
    ap.add_argument("--rounds", type=int, default=5)
    ap.add_argument("--write-tuned", action="store_true", help="merge the best tiles into tuned_tiles.json")
    ap.add_argument("--proj", action="store_true",
                    help="also sweep the stage entries of workloads 2 and 3 with their projections fused in")
    ap.add_argument("--proj-only", action="store_true", help="sweep only those fused stage entries")
    args = ap.parse_args(argv)

    done = set()
    rows = []
    if os.path.exists(args.out):
        for line in open(args.out):
            if line.strip():
                r = json.loads(line)
                rows.append(r)
                done.add((r["shape"], r["tile"], r.get("splits", 1)))
    dev = torch.device("cuda:0")
    with open(args.out, "a") as fh:
        def log(s):
            print(s, flush=True)
            fh.write(s + "\n")
            fh.flush()
        for cfg in args.workload:
            layers = qi.WORKLOADS[cfg]()
            if cfg in (2, 3):
                layers = qi.distinct(layers)
            for lid, L in enumerate([] if args.proj_only else layers):
                t = qi.layer_tensors(cfg, lid, L)
                x = qconv.pack(torch.from_numpy(t["x"]).to(dev), L.bits, L.x_signed)
                w = qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
                e = L.epilogue
                mult = torch.from_numpy(t["mult"]).to(dev) if e else None
                print(f"# workload {cfg} layer {L.name}", flush=True)
                rows += sweep_layer(L.desc(), x, w, mult, shift=e.shift if e else 20, relu=e.relu if e else False,
                                    clamp=(e.lo, e.hi) if e else (0, 15), reps=args.reps, rounds=args.rounds,
                                    done=frozenset(done), log=log)
            if (args.proj or args.proj_only) and cfg in (2, 3):
                full = qi.WORKLOADS[cfg]()
                names = [L.name for L in full]
                for i, L in enumerate(full):
                    if not (L.name.endswith(".0.conv1") and L.stride == 2):
                        continue
                    j = names.index(L.name.replace("conv1", "downsample"))
                    P = full[j]
                    t, tp = qi.layer_tensors(cfg, i, L), qi.layer_tensors(cfg, j, P)
                    x = qconv.pack(torch.from_numpy(t["x"]).to(dev), L.bits, L.x_signed)
                    w3 = qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
                    w1 = qconv.pack(torch.from_numpy(tp["w"]).to(dev), P.bits, P.w_signed)
                    e, ep = L.epilogue, P.epilogue
                    print(f"# workload {cfg} fused {L.name} + {P.name}", flush=True)
                    rows += sweep_proj_layer(L.desc(), x, w3, w1, torch.from_numpy(t["mult"]).to(dev),
                                             torch.from_numpy(tp["mult"]).to(dev), shift=e.shift, shift2=ep.shift,
                                             relu=e.relu, relu2=ep.relu, clamp=(e.lo, e.hi), reps=args.reps,
                                             rounds=args.rounds, done=frozenset(done), log=log)
    best = best_per_shape(rows)
    for key, r in sorted(best.items()):
        dflt = [x for x in rows if x["shape"] == key and x["default"]]
        speed = f" ({dflt[0]['us'] / r['us']:.2f}x vs default {dflt[0]['tile']})" if dflt else ""
        print(f"best {key}: {r['tile']} splits {r.get('splits', 1)} {r['us']} us {r['tops']} TOP/s{speed}", flush=True)
    if args.write_tuned:
        table = json.load(open(TUNED_PATH)) if os.path.exists(TUNED_PATH) else {}
        table.update({k: {"tile": r["tile"], "splits": r.get("splits", 1)} for k, r in best.items()})
        with open(TUNED_PATH, "w") as fh:
            json.dump(table, fh, indent=1, sort_keys=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
