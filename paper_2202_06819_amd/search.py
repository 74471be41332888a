"""Schedule search with a learned cost model and diversity-aware exploration.

The search of Sec. 3.4, restated for this implementation's schedule space:

* Space: every valid ``qconv_schedule`` of one convolution shape.  Its knobs
  are the compiled tile's own knobs -- kernel variant (the loop order: per-tap
  staging or band staging), waves per workgroup along pixels and channels,
  MFMA fragments per wave along pixels and channels, channel chunk (the
  paper's BLK-ROW/COL-WARPS, WARP-ROW/COL-TILES, CHUNK and REORDER-INNER of
  Sec. 4.1) -- plus the split-K factor and three launch knobs (workgroups per
  CU of a persistent grid, LDS band buffers, XCD-aware block order).  Many
  knobs do nothing for a given shape, so many schedules perform alike: the
  situation Sec. 3.4 describes.
* Cost model: gradient-boosted trees on schedule features, fitted to the
  rank of each measured schedule's speed (only the order matters, as with a
  ranking loss).
* Exploration: simulated annealing on the model's score.  Each round every
  point of the plan mutates one random knob; a mutant replaces its parent if
  it scores higher, or with probability exp(gain / temperature).  The
  temperature starts at 1 and cools by 0.002 per round, for at most 500
  rounds, stopping early when the best unmeasured set has not changed for 50
  rounds.  With ``diversity`` every point yields two mutants and half of all
  mutants are kept by a greedy farthest-point choice in knob space (Hamming
  distance), seeded with the best-scoring mutant; the kept mutants then
  compete with the previous points.
* Measurement: batches of 32 -- the 31 best unmeasured schedules the
  exploration found plus one random unmeasured one (random fill when fewer
  than 31 are new).  The first batch is random.  Every measured schedule's
  output is checked byte for byte against a reference schedule.

    python -m paper_2202_06819_amd.search exhaustive --out table.jsonl     # GPU: time every schedule
    python -m paper_2202_06819_amd.search live --trials 96 --out live.jsonl  # GPU: search on the device
    python -m paper_2202_06819_amd.search replay --table table.jsonl       # CPU: searches against a table
"""
from __future__ import annotations

import argparse
import itertools
import json
import math
import os
import random
import statistics
import sys
from dataclasses import dataclass, field

import numpy as np

TILE_KNOBS = ("variant", "waves_p", "waves_k", "frag_p", "frag_k", "chunk_c")
LAUNCH_KNOBS = ("splits", "wg_per_cu", "band_buffers", "xcd_order")
KNOBS = TILE_KNOBS + LAUNCH_KNOBS
SPLIT_CHOICES = (1, 2, 4, 8, 16)
WG_PER_CU_CHOICES = (0, 1, 2, 3, 4)
BAND_CHOICES = (0, 1, 2)
XCD_CHOICES = (0, 1)


class ScheduleSpace:
    """The valid schedules of one shape, as tuples of knob values (KNOBS order).

    ``configs`` lists them; ``tile_ids`` maps the tile-knob part of a config to
    the compiled tile id; ``extra`` holds per-config derived features."""

    def __init__(self, configs: list[tuple], tile_ids: dict[tuple, int] | None = None,
                 extra: dict[tuple, tuple] | None = None):
        if not configs:
            raise ValueError("empty schedule space")
        self.configs = list(dict.fromkeys(configs))
        self.valid = set(self.configs)
        self.tile_ids = tile_ids or {}
        self.extra = extra or {}
        self.domains = [sorted({c[i] for c in self.configs}) for i in range(len(KNOBS))]

    @classmethod
    def for_shape(cls, d: dict) -> "ScheduleSpace":
        """Enumerate the valid schedules of descriptor `d` through the library's
        host-side checks (no device needed)."""
        from . import qconv
        info = qconv.layout(d)
        configs, tile_ids, extra = [], {}, {}
        for t in qconv.tiles():
            if qconv.tile_status(d, t["id"]) != 0:
                continue
            tk = (t["variant"], t["waves_p"], t["waves_k"], t["frag_p"], t["frag_k"], t["chunk_c"])
            tile_ids[tk] = t["id"]
            chunks = max(1, qconv.max_splits(d, t["id"]))
            ntiles = -(-info["m"] // t["tile_p"]) * -(-d["k"] // t["tile_k"])
            for sp, wg, bb, xo in itertools.product(SPLIT_CHOICES, WG_PER_CU_CHOICES, BAND_CHOICES, XCD_CHOICES):
                if sp > chunks:
                    continue
                sch = {"tile_id": t["id"], "splits": sp, "wg_per_cu": wg, "band_buffers": bb, "xcd_order": xo}
                if qconv.schedule_status(d, sch) != 0:
                    continue
                cfg = tk + (sp, wg, bb, xo)
                configs.append(cfg)
                extra[cfg] = (t["tile_p"], t["tile_k"], t["threads"], math.log2(ntiles * sp), chunks)
        return cls(configs, tile_ids, extra)

    def __len__(self) -> int:
        return len(self.configs)

    def schedule(self, cfg: tuple) -> dict:
        """The qconv_schedule knobs of a config."""
        return {"tile_id": self.tile_ids[cfg[:len(TILE_KNOBS)]], "splits": cfg[6], "wg_per_cu": cfg[7],
                "band_buffers": cfg[8], "xcd_order": cfg[9]}

    def features(self, cfgs: list[tuple]) -> np.ndarray:
        rows = []
        for c in cfgs:
            row = [float(v) for v in c]
            row.append(float(c[3] * c[4]))                       # fragments per wave
            row.append(float(c[1] * c[2]))                       # waves per workgroup
            row.extend(float(v) for v in self.extra.get(c, ()))
            rows.append(row)
        width = max(len(r) for r in rows)
        return np.array([r + [0.0] * (width - len(r)) for r in rows], dtype=np.float64)

    def mutate(self, cfg: tuple, rng: random.Random, attempts: int = 64) -> tuple:
        """Change one random knob to another value of its domain so that the
        result is a valid schedule (the parent itself if none is found)."""
        for _ in range(attempts):
            i = rng.randrange(len(KNOBS))
            choices = [v for v in self.domains[i] if v != cfg[i]]
            if not choices:
                continue
            new = cfg[:i] + (rng.choice(choices),) + cfg[i + 1:]
            if new in self.valid:
                return new
        return cfg

    @staticmethod
    def distance(a: tuple, b: tuple) -> int:
        """Knobs in which two schedules differ."""
        return sum(x != y for x, y in zip(a, b))


class CostModel:
    """Gradient-boosted regression trees fitted to the rank of each measured
    schedule's speed, normalised to [0, 1] (1 = fastest).  Predictions are
    scores: higher means expected faster."""

    def __init__(self, seed: int = 0):
        self.seed = seed
        self.model = None

    def fit(self, X: np.ndarray, us: np.ndarray) -> None:
        from sklearn.ensemble import GradientBoostingRegressor
        order = np.argsort(np.argsort(-np.asarray(us, dtype=np.float64)))   # 0 = slowest
        y = order / max(1, len(us) - 1)
        self.model = GradientBoostingRegressor(n_estimators=80, max_depth=3, learning_rate=0.1, subsample=0.8,
                                               random_state=self.seed)
        self.model.fit(X, y)

    def predict(self, X: np.ndarray) -> np.ndarray:
        if self.model is None:
            return np.zeros(len(X))
        return self.model.predict(X)


def diverse_half(space: ScheduleSpace, cands: list[tuple], scores: np.ndarray, keep: int) -> list[int]:
    """Indices of `keep` candidates chosen for diversity: the best-scoring one
    first, then repeatedly the candidate farthest (in knobs) from everything
    chosen so far, ties going to the higher score."""
    n = len(cands)
    keep = min(keep, n)
    if keep <= 0:
        return []
    first = int(np.argmax(scores))
    chosen = [first]
    mind = np.array([space.distance(cands[first], c) for c in cands], dtype=np.float64)
    mind[first] = -1.0
    while len(chosen) < keep:
        key = mind * 1e6 + np.asarray(scores, dtype=np.float64)
        key[chosen] = -np.inf
        j = int(np.argmax(key))
        chosen.append(j)
        dj = np.array([space.distance(cands[j], c) for c in cands], dtype=np.float64)
        mind = np.minimum(mind, dj)
        mind[chosen] = -1.0
    return chosen


def anneal(space: ScheduleSpace, model: CostModel, measured: set, rng: random.Random, *, want: int,
           plan_size: int = 128, n_iter: int = 500, early_stop: int = 50, temp: float = 1.0, cool: float = 0.002,
           diversity: bool = False, start: list[tuple] | None = None) -> list[tuple]:
    """Simulated annealing on the cost model's score; returns up to `want`
    unmeasured schedules, best predicted first."""
    pool = [c for c in (start or []) if c in space.valid]
    while len(pool) < plan_size:
        pool.append(rng.choice(space.configs))
    points = pool[:plan_size]
    scores = model.predict(space.features(points))
    best: dict[tuple, float] = {}

    def offer(cfgs, sc):
        changed = False
        for c, s in zip(cfgs, sc):
            if c in measured:
                continue
            if c in best:
                continue
            if len(best) < want:
                best[c] = float(s)
                changed = True
            else:
                worst = min(best, key=best.get)
                if s > best[worst]:
                    del best[worst]
                    best[c] = float(s)
                    changed = True
        return changed

    offer(points, scores)
    last_change = 0
    t = temp
    for it in range(n_iter):
        if diversity:
            mutants = [space.mutate(p, rng) for p in points for _ in range(2)]
            msc = model.predict(space.features(mutants))
            sel = diverse_half(space, mutants, msc, len(points))
            rng.shuffle(sel)
            new = [mutants[i] for i in sel]
            new_sc = msc[sel]
        else:
            new = [space.mutate(p, rng) for p in points]
            new_sc = model.predict(space.features(new))
        for i in range(len(points)):
            gain = float(new_sc[i] - scores[i])
            if gain >= 0 or rng.random() < math.exp(gain / max(t, 1e-5)):
                points[i], scores[i] = new[i], new_sc[i]
        if offer(new, new_sc):
            last_change = it
        elif it - last_change >= early_stop:
            break
        t = max(0.0, t - cool)
    return sorted(best, key=best.get, reverse=True)


@dataclass
class Trial:
    index: int
    cfg: tuple
    us: float
    best_us: float


@dataclass
class SearchResult:
    trials: list[Trial] = field(default_factory=list)

    def best(self) -> Trial:
        return min(self.trials, key=lambda t: t.us)

    def best_after(self, n: int) -> float:
        return min(t.us for t in self.trials[:n])


def search(space: ScheduleSpace, measure, *, trials: int, batch: int = 32, diversity: bool = True, seed: int = 0,
           log=None, **anneal_kw) -> SearchResult:
    """Measured batches chosen by the cost model and annealing (see the module
    docstring); `measure(cfg)` returns microseconds (inf for a failed run)."""
    rng = random.Random(seed)
    model = CostModel(seed)
    measured: dict[tuple, float] = {}
    res = SearchResult()
    best_us = math.inf
    total = min(trials, len(space))
    while len(measured) < total:
        room = total - len(measured)
        unmeasured = [c for c in space.configs if c not in measured]
        if not measured:
            cand = rng.sample(unmeasured, min(batch, len(unmeasured)))
        else:
            cfgs = list(measured)
            model.fit(space.features(cfgs), np.array([measured[c] for c in cfgs]))
            top_measured = sorted(cfgs, key=measured.get)[:batch]
            cand = anneal(space, model, set(measured), rng, want=batch - 1, diversity=diversity,
                          start=top_measured, **anneal_kw)
            rest = [c for c in unmeasured if c not in set(cand)]
            if rest:
                cand.append(rng.choice(rest))
            while len(cand) < batch and len(cand) < len(unmeasured):
                c = rng.choice(unmeasured)
                if c not in cand:
                    cand.append(c)
        for cfg in cand[:room]:
            us = float(measure(cfg))
            measured[cfg] = us
            best_us = min(best_us, us)
            res.trials.append(Trial(len(res.trials), cfg, us, best_us))
            if log:
                log(res.trials[-1])
    return res


# ---------------------------------------------------------------------------- device measurement

class LiveMeasure:
    """Times schedules of one layer on the GPU (graph replays, as the sweep
    does) and checks every output against the library's default schedule."""

    def __init__(self, L, dev, reps: int = 50, rounds: int = 5, seed_cfg: int = 900):
        import torch
        from . import qconv
        import qconv_inputs as qi
        self.torch, self.q, self.L, self.dev = torch, qconv, L, dev
        self.reps, self.rounds = reps, rounds
        t = qi.layer_tensors(seed_cfg, 0, L)
        self.xp = qconv.pack(torch.from_numpy(t["x"]).to(dev), L.bits, L.x_signed)
        self.wp = qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
        e = L.epilogue
        self.kw = dict(requant=True, mult=torch.from_numpy(t["mult"]).to(dev), shift=e.shift, relu=e.relu,
                       clamp=(e.lo, e.hi))
        self.ref = qconv.conv2d(L.desc(), self.xp, self.wp, tile=qconv.default_tile(L.desc()), **self.kw)
        torch.cuda.synchronize()
        self.prepared: dict[int, object] = {}
        self.space: ScheduleSpace | None = None

    def __call__(self, cfg: tuple) -> float:
        from . import sweep
        q, torch, d = self.q, self.torch, self.L.desc()
        sch = self.space.schedule(cfg)
        tid = sch["tile_id"]
        if tid not in self.prepared:
            self.prepared[tid] = q.prepare_filters(d, self.wp, tid)
        wprep = self.prepared[tid]
        ws = q.make_workspace(d, tid, sch["splits"], self.dev)

        def make(stream=None):
            return q.Conv2dCall(d, self.xp, wprep, schedule=sch, workspace=ws, stream=stream, **self.kw)

        out = make()()
        torch.cuda.synchronize()
        if not torch.equal(out, self.ref):
            raise RuntimeError(f"schedule {sch} output differs from the default schedule's")
        return sweep._time(make, self.reps, self.rounds)


# ---------------------------------------------------------------------------- command line

def _layers(workload: str):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import qconv_inputs as qi
    if workload == "table1":
        return qi.table1_stages()
    layers = qi.WORKLOADS[int(workload)]()
    if int(workload) in (2, 3):
        layers = qi.distinct(layers)
    return [L for L in layers if L.r == 3 and L.stride == 1]


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description="schedule search (see the module docstring)")
    ap.add_argument("mode", choices=("exhaustive", "live", "replay"))
    ap.add_argument("--workload", default="table1", help="'table1' (Table 1's four 3x3 stages, N=8) or a workload id")
    ap.add_argument("--out", help="JSONL output (exhaustive, live)")
    ap.add_argument("--table", help="JSONL from an exhaustive run (replay)")
    ap.add_argument("--trials", type=int, default=96)
    ap.add_argument("--seeds", type=int, default=20)
    ap.add_argument("--reps", type=int, default=50)
    ap.add_argument("--rounds", type=int, default=5)
    args = ap.parse_args(argv)

    if args.mode == "replay":
        return replay_report(args.table, args.trials, args.seeds)

    import torch
    dev = torch.device("cuda:0")
    with open(args.out, "a") as fh:
        for L in _layers(args.workload):
            space = ScheduleSpace.for_shape(L.desc())
            meas = LiveMeasure(L, dev, args.reps, args.rounds)
            meas.space = space
            print(f"# {L.name}: {len(space)} schedules", flush=True)
            if args.mode == "exhaustive":
                for cfg in space.configs:
                    us = meas(cfg)
                    rec = {"layer": L.name, "cfg": list(cfg), "schedule": space.schedule(cfg), "us": round(us, 4)}
                    fh.write(json.dumps(rec) + "\n")
                    fh.flush()
                best = min((json.loads(l) for l in open(args.out) if json.loads(l)["layer"] == L.name),
                           key=lambda r: r["us"])
                print(f"best {L.name}: {best['schedule']} {best['us']} us", flush=True)
            else:
                for diversity in (False, True):
                    def log(t, diversity=diversity):
                        fh.write(json.dumps({"layer": L.name, "diversity": diversity, "trial": t.index,
                                             "cfg": list(t.cfg), "us": round(t.us, 4),
                                             "best_us": round(t.best_us, 4)}) + "\n")
                        fh.flush()
                    res = search(space, meas, trials=args.trials, diversity=diversity, seed=0, log=log)
                    b = res.best()
                    print(f"search {L.name} diversity={diversity}: best {space.schedule(b.cfg)} {b.us:.3f} us "
                          f"after {args.trials} trials (found at trial {b.index})", flush=True)
    return 0


def replay_report(table: str, trials: int, seeds: int) -> int:
    """Searches against a recorded exhaustive table (each measurement is the
    recorded time), plain and diversity-aware, over several seeds."""
    rows = [json.loads(l) for l in open(table) if l.strip()]
    layers = list(dict.fromkeys(r["layer"] for r in rows))
    for name in layers:
        rec = {tuple(r["cfg"]): r["us"] for r in rows if r["layer"] == name}
        space = ScheduleSpace(list(rec))
        best = min(rec.values())
        print(f"{name}: {len(rec)} schedules, exhaustive best {best:.3f} us")
        for method in ("random", "annealing", "diversity-aware"):
            at = {n: [] for n in (32, 48, 64, 96, 128, 192, 256) if n <= trials}
            hit = []
            for seed in range(seeds):
                if method == "random":
                    order = random.Random(seed).sample(list(rec), min(trials, len(rec)))
                    res = SearchResult()
                    b = math.inf
                    for i, c in enumerate(order):
                        b = min(b, rec[c])
                        res.trials.append(Trial(i, c, rec[c], b))
                else:
                    res = search(space, rec.__getitem__, trials=trials, diversity=method != "annealing", seed=seed)
                for n in at:
                    at[n].append(res.best_after(n) / best)
                first = next((t.index + 1 for t in res.trials if t.us <= best * 1.005), None)
                hit.append(first if first is not None else math.inf)
            summary = ", ".join(f"{n}: {statistics.mean(v):.4f}" for n, v in at.items())
            found = [h for h in hit if h != math.inf]
            print(f"  {method}: mean best/exhaustive after trials {summary}; within 0.5% in "
                  f"{len(found)}/{seeds} seeds, median trial {statistics.median(found) if found else 'n/a'}",
                  flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
