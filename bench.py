#!/usr/bin/env python3
"""Benchmark of the quantised convolution path on one MI355X.

A step is one pass of the whole hot path over one batch: relayout+pack of the
int8 NCHW activations into channel-packed 4-bit NHWC (qconv_pack), then the
implicit-GEMM convolution with the fused requantise/ReLU/clamp/repack
epilogue (qconv2d_prepared).  Filters are packed and laid out for the tile
once beforehand (offline, untimed).

The K timed steps run as replays of a captured HIP graph of G steps (one host
launch per G steps), so the figure is the GPU's time per step, not the host's
kernel-launch rate; the eager time per step (one host launch per kernel) is
reported beside it.

Default workload: N=8, 56x56, C=K=64, 3x3, stride 1, pad 1, 4-bit activations
in [0,15], 4-bit filters in [-8,7], per-channel multipliers in [2^14, 2^15),
shift 20, ReLU, clamp [0,15] -- the stage-2 convolution of the paper's
Table 1 (1,849,688,064 ops).  All inputs are seeded synthetic data, resident
in HBM before timing starts.

Prints ONE JSON line.  `value` = effective TOP/s of the step
(2*N*P*Q*K*C*R*S per step / time per step).
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "effective int4/int8 conv TOPS per layer + % of int8 MFMA peak (1 GPU)"
INT8_PEAK_TOPS = 5000.0      # MI355X dense int8 MFMA, 5.0 POP/s
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, 8 TB/s


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


# measurement aids, not kernels of the path: their sources do not enter the kernel digest
NOT_KERNEL_SOURCES = ("qconv_probe.hip", "qconv_unroll.hip")


def kernel_digest(tile_name: str) -> str:
    """Digest of the kernel sources and the tile: profiler summaries taken for
    another digest describe another kernel and are not reported."""
    h = hashlib.sha256(tile_name.encode())
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2202_06819_amd", "csrc", "*"))):
        if os.path.basename(f) in NOT_KERNEL_SOURCES:
            continue
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def profile_values(kind: str, workload: str, tile_name: str) -> dict | None:
    """The machine-readable lines (`- key: value`) of the committed rocprofv3
    summary profiles/*_<kind>.md of this workload, or None when there is none
    for the current kernel sources and tile."""
    digest = kernel_digest(tile_name)
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", f"*_{kind}.md"))):
        kv = {}
        for line in open(path):
            if line.startswith("- ") and ": " in line:
                k, v = line[2:].split(": ", 1)
                kv[k.strip()] = v.strip().strip("`")
        if kv.get("workload") == workload and kv.get("kernel_digest") == digest:
            kv["file"] = os.path.relpath(path, ROOT)
            return kv
    return None


def measured_traffic(workload: str, tile_name: str):
    """HBM bytes per launch of the conv kernel from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary of this workload (each counter divided by
    what it reads per byte of a plain copy kernel), or None when there is no
    summary for the current kernel sources and tile."""
    kv = profile_values("traffic", workload, tile_name)
    try:
        return int(float(kv["hbm_bytes_per_launch"])) if kv else None
    except (KeyError, ValueError):
        return None


def launch_floor(dev, grids, reps: int = 200) -> list[dict]:
    """Per-launch time of an empty kernel (qconv_probe_launch) over each
    (workgroups, threads, dynamic LDS) grid, back to back in a replayed graph
    (median and min of five replays)."""
    from paper_2202_06819_amd import qconv
    rows = []
    for blocks, threads, lds in grids:
        g, calls = captured(lambda s: [qconv.ProbeLaunchCall(blocks, threads, lds, s)], reps)
        per = sorted(time_graph(g, 1) * 1000.0 / reps for _ in range(5))
        rows.append({"blocks": blocks, "threads": threads, "lds_bytes": lds, "graph_us": round(per[2], 3),
                     "graph_us_min": round(per[0], 3)})
        del g
    return rows


def grid_meeting(dev, blocks_list, rounds: int = 64, reps: int = 50) -> list[dict]:
    """Cost of one device-wide meeting inside a launch (qconv_probe_grid_meet:
    agent-scope release, one atomic arrival, poll until the whole grid is
    there, agent-scope acquire): the per-launch time of a grid meeting `rounds`
    times minus that of the same grid meeting none, over `rounds`, both back to
    back in replayed graphs (median of five replays).  Compare with the launch
    floor: a persistent launch running several layers pays a meeting at each
    layer boundary where launches pay a launch."""
    import torch
    from paper_2202_06819_amd import qconv
    rows = []
    for blocks in blocks_list:
        for two in (False, True):
            state = torch.zeros(qconv.ProbeGridMeetCall.STATE_ELEMS, dtype=torch.int32, device=dev)
            per = {}
            for r in (0, rounds):
                g, calls = captured(lambda s: [qconv.ProbeGridMeetCall(blocks, r, state, two, s)], reps)
                per[r] = sorted(time_graph(g, 1) * 1000.0 / reps for _ in range(5))[2]
                del g
            torch.cuda.synchronize()
            ok = int(state[144].item()) == 0
            rows.append({"blocks": blocks, "threads": 256, "counting": "two-level (per XCD)" if two else "flat",
                         "rounds": rounds, "launch_us_no_meeting": round(per[0], 3), "launch_us": round(per[rounds], 3),
                         "us_per_meeting": round((per[rounds] - per[0]) / rounds, 3) if ok else None,
                         "all_arrived": ok})
    return rows


def copy_calibration(mib: int, reps: int) -> int:
    """A plain one-to-one copy kernel over `mib` MiB of int32 (read once,
    written once): the reference that scales FETCH_SIZE / WRITE_SIZE to bytes."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.arange(n, dtype=torch.int32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(reps):
        torch.bitwise_not(src, out=dst)
    torch.cuda.synchronize()
    ok = bool(torch.equal(torch.bitwise_not(dst), src))
    print(json.dumps({"copy_calibration": {"bytes_read": 4 * n, "bytes_written": 4 * n, "reps": reps,
                                           "kernel": "bitwise_not int32", "verified": ok}}), flush=True)
    return 0 if ok else 1


def time_loop(fn, reps: int) -> float:
    """Average microseconds per call of fn() over reps back-to-back calls, from
    HIP events on the current stream (where the library launches)."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1000.0 / reps


def captured(make_calls, passes: int):
    """A graph holding `passes` back-to-back runs of the calls make_calls(stream)
    returns (built for the capture stream).  Replaying it costs one launch for
    all of them, so its timing is the GPU's and not the host's launch rate."""
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        calls = make_calls(s)
        for c in calls:
            c()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for _ in range(passes):
                for c in calls:
                    c()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    return g, calls


def time_graph(g, replays: int) -> float:
    """Milliseconds for `replays` replays of graph g, from HIP events on the
    stream that launches it."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(replays):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1)


def mfma_probe(dev, blocks: int = 2048, iters: int = 2048, launches: int = 5, shape: int = 0) -> dict:
    """The int8 rate of a kernel that issues nothing but MFMAs (all CUs; with
    the default 2048 workgroups eight waves per SIMD; eight independent chains
    of v_mfma_i32_16x16x64_i8 per wave, or with shape 1 four of
    v_mfma_i32_32x32x32_i8), timed with HIP events; the shader clock it ran
    at from its own counters."""
    import statistics
    import torch
    from paper_2202_06819_amd import qconv
    sink = torch.empty(blocks * 256, dtype=torch.int32, device=dev)
    stamps = torch.zeros(blocks * 4, dtype=torch.int64, device=dev)
    qconv.probe_mfma_i8(blocks, 16, sink, stamps, shape=shape)
    torch.cuda.synchronize()
    best, ops = None, 0
    for _ in range(launches):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        ops = qconv.probe_mfma_i8(blocks, iters, sink, stamps, shape=shape)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    st = stamps.view(blocks, 4).cpu().double()
    ghz = statistics.median(((st[:, 1] - st[:, 0]) / ((st[:, 3] - st[:, 2]) * 10.0)).tolist())
    tops = ops / (best * 1e-3) / 1e12
    nominal = 256 * 4 * 2048 * ghz * 1e9 / 1e12   # 256 CUs x 4 SIMDs x 2048 int8 ops per clock
    return {"tops": round(tops, 1), "clock_ghz": round(ghz, 3), "nominal_tops_at_clock": round(nominal, 1),
            "frac_of_nominal_peak": round(tops / INT8_PEAK_TOPS, 4), "ms": round(best, 4), "ops": ops,
            "blocks": blocks, "iters": iters}


def mfma_shapes(dev) -> list[dict]:
    """The MFMA probe at one and two waves per SIMD (256 and 512 workgroups of
    four waves, the occupancy of the convolution kernels) for both int8
    instruction shapes: what fraction of the matrix cores' rate at the
    measured clock each sustains there."""
    rows = []
    for blocks in (256, 512):
        for shape, name in ((0, "v_mfma_i32_16x16x64_i8"), (1, "v_mfma_i32_32x32x32_i8")):
            r = mfma_probe(dev, blocks=blocks, iters=8192, launches=3, shape=shape)
            rows.append({"instruction": name, "waves_per_simd": blocks // 256, "tops": r["tops"],
                         "clock_ghz": r["clock_ghz"],
                         "frac_of_rate_at_clock": round(r["tops"] / r["nominal_tops_at_clock"], 4)})
    return rows


def layer_bytes(L) -> int:
    """Algorithmic HBM bytes of one layer: the packed input pixels the
    convolution touches once (every pixel for a window wider than the stride,
    only the sampled ones for a 1x1 strided filter), the packed filters once,
    the packed output once and 4 bytes of multiplier per output channel."""
    p = (L.h + 2 * L.pad - L.r) // L.stride + 1
    q = (L.w + 2 * L.pad - L.s) // L.stride + 1
    touched = L.n * p * q if (L.r == 1 and L.s == 1) else L.n * L.h * L.w
    out_bits = L.bits if L.epilogue else 32
    return (touched * L.c * L.bits // 8 + L.k * L.r * L.s * L.c * L.bits // 8 + L.n * p * q * L.k * out_bits // 8
            + (4 * L.k if L.epilogue else 0))


def cold_copies(per_copy_bytes: int, min_bytes: int = 640 << 20) -> int:
    """How many distinct operand copies exceed the L2 caches plus the 256 MB
    Infinity Cache, so a launch that rotates through them reads from HBM."""
    return max(2, -(-min_bytes // max(1, per_copy_bytes)))


def cold_time(calls, rounds: int = 3) -> float:
    """Average microseconds per call when each call of the list works on its
    own copy of the operands (see cold_copies); best of `rounds` passes."""
    def run_all():
        for c in calls:
            c()
    run_all()
    return min(time_loop(run_all, 1) for _ in range(rounds)) / len(calls)


def layer_setup(cfg: int, lid: int, L, dev):
    import torch
    import qconv_inputs as qi
    from paper_2202_06819_amd import qconv
    t = qi.layer_tensors(cfg, lid, L)
    x = torch.from_numpy(t["x"]).to(dev)
    w = torch.from_numpy(t["w"]).to(dev)
    xp = qconv.pack(x, L.bits, L.x_signed)
    wp = qconv.pack(w, L.bits, L.w_signed)
    e = L.epilogue
    mult = torch.from_numpy(t["mult"]).to(dev) if e else None
    return x, xp, wp, mult


def per_layer_table(cfg: int, layers, dev, reps: int) -> list[dict]:
    import torch
    from paper_2202_06819_amd import qconv
    import qconv_inputs as qi
    rows = []
    for lid, L in enumerate(layers):
        from paper_2202_06819_amd import sweep
        x, xp, wp, mult = layer_setup(cfg, lid, L, dev)
        e = L.epilogue
        tile, splits = sweep.tuned_config(L.desc(), e is not None)
        wprep = qconv.prepare_filters(L.desc(), wp, tile)
        ws = qconv.make_workspace(L.desc(), tile, splits, dev)

        def make(stream=None, x_in=xp, out=None):
            return qconv.Conv2dCall(L.desc(), x_in, wprep, requant=e is not None, mult=mult,
                                    shift=e.shift if e else 20, relu=e.relu if e else False,
                                    clamp=(e.lo, e.hi) if e else (0, 15), tile=tile, prepared=True, stream=stream,
                                    splits=splits, workspace=ws, out=out)

        call = make()
        for _ in range(5):
            call()
        eager_us = time_loop(call, reps)
        g, _ = captured(lambda s: [make(s)], reps)
        # per-launch time of each of 5 replays of the reps-launch graph: median and min
        per = sorted(time_graph(g, 1) * 1000.0 / reps for _ in range(5))
        us, us_min = per[2], per[0]
        tops = L.ops / (us * 1e-6) / 1e12
        nbytes = layer_bytes(L)
        row = {"layer": L.name, "tile": qconv.tiles()[call.tile]["name"], "splits": splits, "us": round(us, 3),
               "us_min": round(us_min, 3), "eager_us": round(eager_us, 3),
               "tops": round(tops, 2), "pct_int8_peak": round(100 * tops / INT8_PEAK_TOPS, 2),
               "gops": round(L.ops / 1e9, 4), "alg_bytes": nbytes,
               "gbs": round(nbytes / (us * 1e-6) / 1e9, 1)}
        if L.r == 1 and L.s == 1:
            # HBM-bound layer: also timed cold, each launch on its own copy of x and y
            xb, yb = xp.numel() * xp.element_size(), call.out.numel() * call.out.element_size()
            n_cp = cold_copies(xb + yb)
            big_x = torch.empty((n_cp,) + tuple(xp.shape), dtype=xp.dtype, device=dev)
            big_x.copy_(xp.unsqueeze(0).expand_as(big_x))
            big_y = torch.empty((n_cp,) + tuple(call.out.shape), dtype=call.out.dtype, device=dev)
            cold_us = cold_time([make(x_in=big_x[i], out=big_y[i]) for i in range(n_cp)])
            del big_x, big_y
            row.update({"cold_us": round(cold_us, 3), "cold_gbs": round(nbytes / (cold_us * 1e-6) / 1e9, 1),
                        "cold_copies": n_cp})
        rows.append(row)
        log(f"  {L.name:28s} {us:9.2f} us {tops:8.1f} TOP/s {100 * tops / INT8_PEAK_TOPS:5.1f}%  "
            f"{row['gbs']:7.1f} GB/s  tile {row['tile']} splits {splits}"
            + (f"  cold {row['cold_us']:.2f} us {row['cold_gbs']:.0f} GB/s" if "cold_us" in row else ""))
    return rows


def qi_shape(layers, name: str) -> str:
    """A layer's shape as text: 56x56 64->64 3x3 s1."""
    L = next(L for L in layers if L.name == name)
    return f"{L.h}x{L.w} {L.c}->{L.k} {L.r}x{L.s} s{L.stride}"


def residual_order(layers):
    """The ResNet-18 stack as residual blocks: each block's second 3x3 adds its
    shortcut (the block input, or the stage's 1x1 projection, which is moved
    ahead of it) before ReLU.  Returns (layers in run order, source index,
    shortcut index or None) per layer."""
    order = []
    names = [L.name for L in layers]
    for i, L in enumerate(layers):
        if L.name.endswith("downsample"):
            continue
        order.append(i)
        if L.name.endswith(".0.conv1"):
            ds = L.name.replace("conv1", "downsample")
            if ds in names:
                order.append(names.index(ds))
    pos = {old: new for new, old in enumerate(order)}
    out = []
    for old in order:
        L = layers[old]
        src = -1 if L.src < 0 else pos[L.src]
        short = None
        if L.name.endswith("conv2"):
            ds = L.name.replace("conv2", "downsample")
            if ds in names:
                short = pos[names.index(ds)]
            else:
                block_in = layers[L.src].src     # conv1's input is the block input
                short = -1 if block_in < 0 else pos[block_in]
        out.append((L, src, short, old))
    return out


def chain_time(cfg: int, layers, dev, reps: int, residual: bool = False) -> dict:
    """End-to-end time of a chained network (each output feeds the next layer);
    with `residual`, as residual blocks with a per-channel bias in every layer."""
    import numpy as np
    import torch
    import qconv_inputs as qi
    from paper_2202_06819_amd import nets, qconv
    t0 = qi.layer_tensors(cfg, 0, layers[0])
    x = torch.from_numpy(t0["x"]).to(dev)
    xp = qconv.pack(x, layers[0].bits, layers[0].x_signed)
    specs = []
    plan = residual_order(layers) if residual else [(L, L.src, None, i) for i, L in enumerate(layers)]
    for L, src, short, lid in plan:
        t = qi.layer_tensors(cfg, lid, L)
        wp = qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
        e = L.epilogue
        bias = None
        if residual:
            bias = torch.from_numpy(np.random.default_rng([cfg, lid, 3]).integers(-256, 256, size=L.k)
                                    .astype(np.int32)).to(dev)
        specs.append(nets.LayerSpec(L.desc(), wp, torch.from_numpy(t["mult"]).to(dev), e.shift, e.relu,
                                    (e.lo, e.hi), src=src, bias=bias, residual_src=short,
                                    residual_signed=e.lo < 0))
    out = {"layers": len(layers), "gops": round(sum(L.ops for L in layers) / 1e9, 3)}
    best = None
    # one stream with each stage's projection fused into its strided 3x3 (the
    # chain's default), then unfused on one stream, then the projections on a
    # second stream beside the strided 3x3s
    for kw, tag in ((dict(), ""), (dict(fuse_projections=False), "unfused_"), (dict(branches=True), "branches_")):
        chain = nets.Chain(specs, xp, **kw)
        out[tag + "launches"] = chain.launches
        for _ in range(3):
            chain.forward()
        eager = time_loop(chain.forward, reps)
        out[tag + "eager_us"] = round(eager, 2)
        t = eager
        try:
            chain.capture()
            for _ in range(3):
                chain.replay()
            out[tag + "graph_us"] = round(time_loop(chain.replay, reps), 2)
            t = min(t, out[tag + "graph_us"])
        except Exception as exc:  # graph capture is an extra, report why it is missing
            out[tag + "graph_error"] = str(exc)[:200]
        if not tag:
            best = t
        del chain
    out["tops"] = round(sum(L.ops for L in layers) / (best * 1e-6) / 1e12, 2)
    return out


def proj_table(cfg: int, layers, dev, reps: int) -> list[dict]:
    """Each stage entry of a ResNet-18 stack (strided 3x3 and its 1x1
    projection, which read the same block input) as one fused launch
    (qconv2d_proj, tuned tile), against the two layers' separate launches."""
    import torch
    import qconv_inputs as qi
    from paper_2202_06819_amd import qconv, sweep
    names = [L.name for L in layers]
    rows = []
    for i, L in enumerate(layers):
        if not (L.name.endswith(".0.conv1") and L.stride == 2):
            continue
        j = names.index(L.name.replace("conv1", "downsample"))
        P = layers[j]
        t, tp = qi.layer_tensors(cfg, i, L), qi.layer_tensors(cfg, j, P)
        xp = qconv.pack(torch.from_numpy(t["x"]).to(dev), L.bits, L.x_signed)
        w3 = qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
        w1 = qconv.pack(torch.from_numpy(tp["w"]).to(dev), P.bits, P.w_signed)
        m3, m1 = torch.from_numpy(t["mult"]).to(dev), torch.from_numpy(tp["mult"]).to(dev)
        e, ep = L.epilogue, P.epilogue
        tile, psplits = sweep.tuned_proj_config(L.desc())
        wprep = qconv.prepare_filters_proj(L.desc(), w3, w1, tile)
        nws = qconv.proj_workspace_bytes(L.desc(), tile, psplits)
        pws = torch.zeros(nws, dtype=torch.uint8, device=dev) if nws else None

        def make(stream=None):
            return qconv.ProjConv2dCall(L.desc(), xp, wprep, tile=tile, requant=True, mult=m3, shift=e.shift,
                                        relu=e.relu, clamp=(e.lo, e.hi),
                                        proj=dict(mult=m1, shift=ep.shift, relu=ep.relu, clamp=(ep.lo, ep.hi)),
                                        splits=psplits, workspace=pws, stream=stream)

        g, _ = captured(lambda s: [make(s)], reps)
        per = sorted(time_graph(g, 1) * 1000.0 / reps for _ in range(5))
        sep = []
        for lay, tt, wpk, mm in ((L, t, w3, m3), (P, tp, w1, m1)):
            tl, sp = sweep.tuned_config(lay.desc())
            wpr = qconv.prepare_filters(lay.desc(), wpk, tl)
            ws = qconv.make_workspace(lay.desc(), tl, sp, dev)
            ee = lay.epilogue

            def mk(stream=None, lay=lay, wpr=wpr, tl=tl, sp=sp, ws=ws, mm=mm, ee=ee):
                return qconv.Conv2dCall(lay.desc(), xp, wpr, requant=True, mult=mm, shift=ee.shift, relu=ee.relu,
                                        clamp=(ee.lo, ee.hi), tile=tl, prepared=True, splits=sp, workspace=ws,
                                        stream=stream)
            gs, _ = captured(lambda s, mk=mk: [mk(s)], reps)
            sep.append(sorted(time_graph(gs, 1) * 1000.0 / reps for _ in range(5))[2])
        ops = L.ops + P.ops
        rows.append({"layers": f"{L.name} + {P.name}", "tile": qconv.tiles()[tile]["name"], "splits": psplits,
                     "fused_us": round(per[2], 3), "separate_us": round(sum(sep), 3),
                     "conv3x3_us": round(sep[0], 3), "proj_us": round(sep[1], 3),
                     "gops": round(ops / 1e9, 4), "tops": round(ops / (per[2] * 1e-6) / 1e12, 2)})
        log(f"  fused {L.name} + {P.name}: {per[2]:.2f} us vs {sum(sep):.2f} us as two launches "
            f"(tile {rows[-1]['tile']} splits {psplits})")
    return rows


def bottleneck_stack_time(dev, reps: int) -> dict:
    """The ResNet-50 bottleneck stack of workload 4 with its block counts
    (3, 4, 6, 3 blocks at 56, 28, 14, 7): per stage, the blocks chained (1x1
    reduce, 3x3, 1x1 expand, the expand's output feeding the next block's
    reduce), each stage timed end to end eager and as a graph replay.  The
    stages' first blocks keep the repeated blocks' shapes (no strided entry
    block, no projection shortcut, no residual add): a bottleneck stack, not a
    full ResNet-50."""
    import torch
    import qconv_inputs as qi
    from paper_2202_06819_amd import nets, qconv
    layers = qi.WORKLOADS[4]()
    stages, total_eager, total_graph, total_ops = [], 0.0, 0.0, 0
    for st in range(4):
        red, mid, exp = layers[3 * st: 3 * st + 3]
        blocks = qi.BOTTLENECK_REPEATS[red.h]
        t0 = qi.layer_tensors(4, 3 * st, red)
        xp = qconv.pack(torch.from_numpy(t0["x"]).to(dev), red.bits, red.x_signed)
        specs = []
        for b in range(blocks):
            for j, L in enumerate((red, mid, exp)):
                t = t0 if j == 0 else qi.layer_tensors(4, 3 * st + j, L)
                e = L.epilogue
                src = len(specs) - 1
                specs.append(nets.LayerSpec(L.desc(), qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed),
                                            torch.from_numpy(t["mult"]).to(dev), e.shift, e.relu, (e.lo, e.hi),
                                            src=src))
        chain = nets.Chain(specs, xp)
        for _ in range(3):
            chain.forward()
        eager = time_loop(chain.forward, reps)
        chain.capture()
        for _ in range(3):
            chain.replay()
        graph = time_loop(chain.replay, reps)
        ops = blocks * (red.ops + mid.ops + exp.ops)
        stages.append({"stage": f"{red.h}x{red.h}", "blocks": blocks, "layers": 3 * blocks,
                       "gops": round(ops / 1e9, 3), "eager_us": round(eager, 2), "graph_us": round(graph, 2),
                       "tops": round(ops / (min(eager, graph) * 1e-6) / 1e12, 1)})
        total_eager += eager
        total_graph += graph
        total_ops += ops
        del chain
    best = min(total_eager, total_graph)
    return {"stack": "ResNet-50 bottleneck blocks 3/4/6/3, N=64, 4-bit, stride 1 (not a full ResNet-50)",
            "layers": sum(s["layers"] for s in stages), "gops": round(total_ops / 1e9, 2),
            "eager_us": round(total_eager, 1), "graph_us": round(total_graph, 1),
            "tops": round(total_ops / (best * 1e-6) / 1e12, 1), "stages": stages}


def stem_time(dev, n: int, reps: int) -> dict:
    """The 3-channel 7x7 stride-2 stem (8-bit, 224x224 -> 112x112 x 64) run
    patch-unrolled, in both foldings (row pairs and columns into 64 channels,
    a 4x1 convolution; every tap into 192 channels, a 1x1 convolution): the
    input unroll and the convolution are timed (the filter unroll is offline);
    each convolution takes the fastest tile of a short sweep."""
    import torch
    import qconv_inputs as qi
    from paper_2202_06819_amd import qconv
    L = qi.Layer("stem", n, 224, 224, 3, 64, 7, 7, 2, 3, bits=8, x_signed=True, w_signed=True, x_range=qi.S8,
                 w_range=qi.S8, epilogue=qi.Epilogue(relu=True, lo=-128, hi=127))
    t = qi.layer_tensors(6, 0, L)
    x = torch.from_numpy(t["x"]).to(dev)
    mult = torch.from_numpy(t["mult"]).to(dev)
    folds = {}
    for fold, c_out in (("rows", 64), ("all", 192)):
        plan = qconv.few_channel_plan(L.desc(), c_out, fold)
        d = plan["desc"]
        wu = qconv.unroll(torch.from_numpy(t["w"]).to(dev), c_out, **plan["w"])
        xu = qconv.unroll(x, c_out, **plan["x"])
        best = None
        for tt in qconv.tiles():
            if qconv.tile_status(d, tt["id"]) != 0:
                continue
            wp = qconv.prepare_filters(d, wu, tt["id"]) if tt["variant"] == 2 else wu

            def make(stream=None, tid=tt["id"], wp=wp, prep=tt["variant"] == 2, d=d, xu=xu):
                return qconv.Conv2dCall(d, xu, wp, requant=True, mult=mult, shift=20, relu=True, clamp=(-128, 127),
                                        tile=tid, prepared=prep, stream=stream)

            g, _ = captured(lambda st: [make(st)], 20)
            us = time_graph(g, 3) * 1000.0 / 60
            if best is None or us < best[0]:
                best = (us, tt["name"], make)
        g, _ = captured(lambda st: [best[2](st)], reps)
        conv_us = time_graph(g, 3) * 1000.0 / (3 * reps)

        def make_unroll(stream=None, xu=xu, plan=plan, c_out=c_out):
            return lambda: qconv.unroll(x, c_out, out=xu, stream=stream, **plan["x"])

        g, _ = captured(lambda st: [make_unroll(st)], reps)
        unroll_us = time_graph(g, 3) * 1000.0 / (3 * reps)
        folds[fold] = {"c_out": c_out, "conv": f"{d['r']}x1 over {c_out} channels", "tile": best[1],
                       "unroll_us": round(unroll_us, 3), "conv_us": round(conv_us, 3),
                       "unrolled_mb": round(xu.numel() / 1e6, 2),
                       "tops": round(L.ops / ((unroll_us + conv_us) * 1e-6) / 1e12, 2)}
    pick = max(folds, key=lambda f: folds[f]["tops"])
    return {"layer": "stem 7x7/2 3->64 224x224, 8-bit, patch-unrolled", "n": n, "gops": round(L.ops / 1e9, 4),
            "best_fold": pick, "tops": folds[pick]["tops"], "folds": folds}


def layout_table(dev, reps: int) -> list[dict]:
    """The batch-interleaved layout (NHWCnc, nb images per pixel) against the
    plain one on the stride-1 3x3 layers: per layer the plain layout's tuned
    schedule, and for each nb the fastest tile of a short sweep; plus the
    pack kernel of the layer's input in each layout."""
    import torch
    import qconv_inputs as qi
    from paper_2202_06819_amd import qconv, sweep
    layers = [qi.WORKLOADS[1]()[0]] + [L for L in qi.distinct(qi.WORKLOADS[2]()) if L.r == 3 and L.stride == 1]
    rows = []
    for lid, L in enumerate(layers):
        e = L.epilogue
        t = qi.layer_tensors(40, lid, L)
        x = torch.from_numpy(t["x"]).to(dev)
        wp = qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
        mult = torch.from_numpy(t["mult"]).to(dev)
        row = {"layer": L.name, "n": L.n, "h": L.h, "c": L.c, "k": L.k, "gops": round(L.ops / 1e9, 4)}
        ref = None
        for nb in (1, 2, 4, 8, 16):
            if L.n % nb:
                continue
            d = dict(L.desc(), nb=nb)
            xp = qconv.pack(x, L.bits, L.x_signed, nb=nb)
            if nb == 1:
                cands = [sweep.tuned_config(d)]
            else:
                cands = [(tt["id"], sp) for tt in qconv.tiles() if qconv.tile_status(d, tt["id"]) == 0
                         for sp in sweep.split_choices(d, tt["id"])]
            if not cands:   # no tile stages the band of rows this wide
                row[f"nb{nb}"] = None
                continue
            best = None
            for tid, splits in cands:
                wprep = qconv.prepare_filters(d, wp, tid)
                ws = qconv.make_workspace(d, tid, splits, dev)

                def make(stream=None, tid=tid, splits=splits, wprep=wprep, ws=ws, d=d, xp=xp):
                    return qconv.Conv2dCall(d, xp, wprep, requant=True, mult=mult, shift=e.shift, relu=e.relu,
                                            clamp=(e.lo, e.hi), tile=tid, prepared=True, stream=stream,
                                            splits=splits, workspace=ws)

                out = make()()
                torch.cuda.synchronize()
                flat = out.reshape(-1, *out.shape[-1:]) if nb == 1 else \
                    out.permute(0, 3, 1, 2, 4).reshape(-1, out.shape[-1])
                if ref is None:
                    ref = flat.clone()
                elif not torch.equal(flat, ref):
                    raise RuntimeError(f"{L.name} nb={nb} tile {tid}: output differs from the plain layout")
                g, _ = captured(lambda st: [make(st)], 20 if len(cands) > 1 else reps)
                us = time_graph(g, 3) * 1000.0 / (60 if len(cands) > 1 else 3 * reps)
                if best is None or us < best[0]:
                    best = (us, tid, make, splits)
            if len(cands) > 1:
                g, _ = captured(lambda st: [best[2](st)], reps)
                best = (time_graph(g, 3) * 1000.0 / (3 * reps),) + best[1:]

            def make_pack(stream=None, nb=nb, xp=xp):
                return lambda: qconv.pack(x, L.bits, L.x_signed, out=xp, stream=stream, nb=nb)

            g, _ = captured(lambda st: [make_pack(st)], reps)
            pack_us = time_graph(g, 3) * 1000.0 / (3 * reps)
            row[f"nb{nb}"] = {"tile": qconv.tiles()[best[1]]["name"], "splits": best[3], "us": round(best[0], 3),
                              "tops": round(L.ops / (best[0] * 1e-6) / 1e12, 1), "pack_us": round(pack_us, 3)}
        rows.append(row)
        log(f"  {L.name:24s} " + "  ".join(f"{k}: {v['us']:.2f} us (pack {v['pack_us']:.2f})" if v else f"{k}: n/a"
                                            for k, v in row.items() if k.startswith("nb")))
    return rows


def batch_table(dev, reps: int, batches=(16, 32, 64, 128, 256)) -> list[dict]:
    """The four 4-bit 3x3 stride-1 layers of the ResNet-18 stack (fused
    epilogue) at growing batch: the fastest (tile, split) of a short sweep per
    batch, its time and fraction of the int8 MFMA peak.  Shows how much of a
    launch is fixed cost (launch, prologue, epilogue) at batch 16."""
    import torch
    from paper_2202_06819_amd import qconv, sweep
    import qconv_inputs as qi
    shapes = [L for L in qi.distinct(qi.WORKLOADS[2]()) if L.r == 3 and L.stride == 1]
    rows = []
    for lid, L0 in enumerate(shapes):
        e = L0.epilogue
        for n in batches:
            L = qi.Layer(L0.name, n, L0.h, L0.w, L0.c, L0.k, 3, 3, 1, 1)
            t = qi.layer_tensors(41, lid, L)
            d = L.desc()
            xp = qconv.pack(torch.from_numpy(t["x"]).to(dev), L.bits, L.x_signed)
            wp = qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
            mult = torch.from_numpy(t["mult"]).to(dev)
            ref, best = None, None
            for tt in qconv.tiles():
                if qconv.tile_status(d, tt["id"]) != 0 or not tt["name"].startswith("wide"):
                    continue
                wprep = qconv.prepare_filters(d, wp, tt["id"])
                for splits in sweep.split_choices(d, tt["id"]):
                    ws = qconv.make_workspace(d, tt["id"], splits, dev)

                    def make(stream=None, tid=tt["id"], splits=splits, wprep=wprep, ws=ws):
                        return qconv.Conv2dCall(d, xp, wprep, requant=True, mult=mult, shift=e.shift, relu=e.relu,
                                                clamp=(e.lo, e.hi), tile=tid, prepared=True, stream=stream,
                                                splits=splits, workspace=ws)

                    out = make()()
                    torch.cuda.synchronize()
                    if ref is None:
                        ref = out.clone()
                    elif not torch.equal(out, ref):
                        raise RuntimeError(f"{L.name} n={n} tile {tt['name']} splits {splits}: output differs")
                    g, _ = captured(lambda st: [make(st)], 20)
                    us = time_graph(g, 3) * 1000.0 / 60
                    if best is None or us < best[0]:
                        best = (us, tt["name"], splits, make)
            g, _ = captured(lambda st: [best[3](st)], reps)
            us = time_graph(g, 3) * 1000.0 / (3 * reps)
            tops = L.ops / (us * 1e-6) / 1e12
            row = {"layer": L.name, "n": n, "gops": round(L.ops / 1e9, 3), "tile": best[1], "splits": best[2],
                   "us": round(us, 3), "tops": round(tops, 1), "pct_int8_peak": round(100 * tops / INT8_PEAK_TOPS, 2)}
            rows.append(row)
            log(f"  {L.name:24s} N={n:3d} {us:8.2f} us {tops:7.1f} TOP/s {row['pct_int8_peak']:5.1f}%  "
                f"tile {best[1]} splits {best[2]}")
            del xp, wp, ref
    return rows


def fused_step_time(L, x, xp_ref, wp, mult, y_ref, dev, reps: int, tile_name: str):
    """The benchmark step as one launch: qconv2d_packing, the pack fused into
    the convolution, writing the packed input too.  Every tile with the fused
    instance is timed (reported as a table) and checked against the two-launch
    step's output and packed input; the step runs `tile_name` (the layer's
    tuned tile) when it has the instance, so that the choice does not depend on
    a short timing, else the fastest."""
    import torch
    from paper_2202_06819_amd import qconv
    e = L.epilogue
    d = L.desc()
    best = None
    chosen = None
    sweep_rows = []
    for t in qconv.tiles():
        if t["variant"] != 2 or qconv.tile_status(d, t["id"]) != 0:
            continue
        wprep = qconv.prepare_filters(d, wp, t["id"])

        def make(stream=None, tid=t["id"], wprep=wprep):
            return qconv.PackingConv2dCall(d, x, wprep, tile=tid, mult=mult, shift=e.shift, relu=e.relu,
                                           clamp=(e.lo, e.hi), x_packed=True, stream=stream)

        call = make()
        y = call()
        torch.cuda.synchronize()
        if not (torch.equal(y, y_ref) and torch.equal(call.x_packed, xp_ref)):
            raise RuntimeError(f"fused pack + conv on {t['name']} differs from the two-launch step")
        g, _ = captured(lambda st: [make(st)], 20)
        us = time_graph(g, 3) * 1000.0 / 60
        sweep_rows.append({"tile": t["name"], "us": round(us, 3)})
        if best is None or us < best[0]:
            best = (us, t["name"], make)
        if t["name"] == tile_name:
            chosen = (us, t["name"], make)
    if chosen is None:
        chosen = best
    g, _ = captured(lambda st: [chosen[2](st)], reps)
    us = time_graph(g, 5) * 1000.0 / (5 * reps)
    return {"us": round(us, 3), "tops": round(L.ops / (us * 1e-6) / 1e12, 2), "tile": chosen[1],
            "entry": "qconv2d_packing", "packed_copy": True, "tiles": sweep_rows}, chosen[2]


def cpu_baseline(L, seconds: float, threads: int | None = None) -> dict:
    """The oracle, as it stands, on the host cores: pack + conv + requant + repack
    of the same layer, repeated for about `seconds` (all cores by default)."""
    import oracle
    import qconv_inputs as qi
    t = qi.layer_tensors(1, 0, L)
    threads = threads or oracle.max_threads()
    e = L.epilogue
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.qconv_layer(t["x"], t["w"], bits=L.bits, x_signed=L.x_signed, w_signed=L.w_signed,
                           stride=(L.stride, L.stride), pad=(L.pad, L.pad), mult=t["mult"], shift=e.shift,
                           relu=e.relu, lo=e.lo, hi=e.hi, threads=threads)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    return {"value": round(L.ops * reps / el / 1e12, 6), "unit": "TOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} full passes of the benchmark layer ({L.name}: relayout+pack, direct conv, "
                      f"requant, repack) in {el:.1f} s on {threads} OpenMP thread{'s' if threads > 1 else ''}"}


def cpu_network_times(cfgs, single_thread_cfgs) -> dict:
    """The oracle, as it stands, over every layer of whole workloads (each
    layer once: relayout+pack, direct conv, requant, repack), per layer and
    per network in seconds, on all host threads and, for `single_thread_cfgs`,
    on one thread.  A reported baseline for the per-network GPU times."""
    import oracle
    import qconv_inputs as qi
    out = {}
    for cfg in cfgs:
        layers = qi.WORKLOADS[cfg]()
        modes = [oracle.max_threads()] + ([1] if cfg in single_thread_cfgs else [])
        entry = {"layers": len(layers), "gops": round(sum(L.ops for L in layers) / 1e9, 3)}
        for th in modes:
            per, total = [], 0.0
            for lid, L in enumerate(layers):
                t = qi.layer_tensors(cfg, lid, L)
                e = L.epilogue
                t0 = time.perf_counter()
                oracle.qconv_layer(t["x"], t["w"], bits=L.bits, x_signed=L.x_signed, w_signed=L.w_signed,
                                   stride=(L.stride, L.stride), pad=(L.pad, L.pad), mult=t["mult"], shift=e.shift,
                                   relu=e.relu, lo=e.lo, hi=e.hi, threads=th)
                el = time.perf_counter() - t0
                per.append({"layer": L.name, "s": round(el, 4)})
                total += el
            key = "all_threads" if th > 1 else "one_thread"
            entry[key] = {"threads": th, "network_s": round(total, 3),
                          "tops": round(sum(L.ops for L in layers) / total / 1e12, 5), "per_layer": per}
            log(f"  oracle, workload {cfg}, {th} thread{'s' if th > 1 else ''}: {total:.2f} s")
        out[f"workload{cfg}"] = entry
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--layer-reps", type=int, default=200, help="repetitions per layer in the per-layer tables")
    ap.add_argument("--tables", default="2,3,4",
                    help="comma list of workloads with per-layer tables (2,3,4) or 'none'")
    ap.add_argument("--launch-floor", action="store_true",
                    help="also time the empty-kernel launch probe over a range of grid shapes")
    ap.add_argument("--layout-table", action="store_true",
                    help="also time the batch-interleaved layout against the plain one")
    ap.add_argument("--batch-table", action="store_true",
                    help="also time the 4-bit 3x3 stride-1 ResNet-18 layers at batch 16..256 (best tile each)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--cpu-networks", action="store_true",
                    help="also time the oracle over every layer of workloads 2 and 4 (per layer and per network)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--tile", type=int, default=-1)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain copy kernel over MIB MiB (counter calibration) and exit")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the quantised convolution path has no multi-GPU mode "
              f"(--gpus {args.gpus} requested).", file=sys.stderr)
        return 2

    if args.copy_calibration:
        return copy_calibration(args.copy_calibration, max(1, min(args.steps, 50)))

    import torch
    import qconv_inputs as qi
    from paper_2202_06819_amd import build as hip_build
    from paper_2202_06819_amd import qconv, sweep

    hip_build.ensure_built()   # rebuilds when the library is missing or older than its sources
    dev = torch.device("cuda:0")
    L = qi.workload1()[0]
    e = L.epilogue
    x, xp, wp, mult = layer_setup(1, 0, L, dev)
    tile = sweep.tuned_tile(L.desc()) if args.tile == -1 else args.tile
    wprep = qconv.prepare_filters(L.desc(), wp, tile)     # offline, like packing the filters
    y = torch.empty(qconv.packed_shape(L.n, L.p, L.q, L.k, L.bits), dtype=qconv.packed_dtype(L.bits), device=dev)

    def make_pack(stream=None):
        return qconv.PackCall(x, L.bits, L.x_signed, out=xp, stream=stream)

    def make_conv(stream=None):
        return qconv.Conv2dCall(L.desc(), xp, wprep, requant=True, mult=mult, shift=e.shift, relu=e.relu,
                                clamp=(e.lo, e.hi), tile=tile, prepared=True, out=y, stream=stream)

    pack, conv = make_pack(), make_conv()

    def step():
        pack()
        conv()

    tile_name = qconv.tiles()[conv.tile]["name"]
    log(f"workload {L.name}: {L.ops / 1e9:.4f} GOP per step, tile {tile_name}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ref_out = y.clone()

    # eager: one host launch per kernel (bounded by the host's launch rate)
    eager_ms = time_loop(step, args.steps) / 1000.0

    # timed region: the K steps as replays of a captured graph of G steps
    G = max(d for d in range(1, min(args.steps, 100) + 1) if args.steps % d == 0)
    g_step, _ = captured(lambda s: [make_pack(s), make_conv(s)], G)
    for _ in range(max(1, args.warmup // G)):
        g_step.replay()
    torch.cuda.synchronize()
    y.zero_()
    t_wall = time.perf_counter()
    ms_total = time_graph(g_step, args.steps // G)
    t_wall = time.perf_counter() - t_wall
    if not torch.equal(y, ref_out):
        raise RuntimeError("graph replay output differs from the eager output")
    ms_per_step = ms_total / args.steps
    value = L.ops / (ms_per_step * 1e-3) / 1e12
    log(f"step: {ms_per_step * 1000:.2f} us ({value:.1f} TOP/s) from {args.steps // G} replays of a {G}-step graph, "
        f"wall {t_wall:.3f} s; eager {eager_ms * 1000:.2f} us per step")

    # per-kernel averages in the same launch configuration: graphs of back-to-back
    # launches of one kernel, HIP events on the launching stream
    reps = 200
    g_conv, _ = captured(lambda s: [make_conv(s)], reps)
    g_pack, _ = captured(lambda s: [make_pack(s)], reps)
    conv_us = time_graph(g_conv, 5) * 1000.0 / (5 * reps)
    pack_us = time_graph(g_pack, 5) * 1000.0 / (5 * reps)
    conv_tops = L.ops / (conv_us * 1e-6) / 1e12
    pack_bytes = L.n * L.c * L.h * L.w + L.n * L.h * L.w * L.c // 2
    conv_bytes = layer_bytes(L)
    pack_gbs = pack_bytes / (pack_us * 1e-6) / 1e9
    log(f"conv kernel {conv_us:.2f} us = {conv_tops:.1f} TOP/s ({100 * conv_tops / INT8_PEAK_TOPS:.1f}% of int8 peak); "
        f"pack kernel {pack_us:.2f} us = {pack_gbs:.0f} GB/s")
    # the pack kernel cold: every launch on its own copy, so its bytes come from HBM
    n_cp = cold_copies(x.numel() + xp.numel() * xp.element_size())
    big_x = torch.empty((n_cp,) + tuple(x.shape), dtype=x.dtype, device=dev)
    big_x.copy_(x.unsqueeze(0).expand_as(big_x))
    big_p = torch.empty((n_cp,) + tuple(xp.shape), dtype=xp.dtype, device=dev)
    pack_cold_us = cold_time([qconv.PackCall(big_x[i], L.bits, L.x_signed, out=big_p[i]) for i in range(n_cp)])
    del big_x, big_p
    fused, fused_make = fused_step_time(L, x, xp, wp, mult, ref_out, dev, reps, tile_name)
    log(f"the step as one launch (pack fused into the conv, packed copy written): {fused['us']:.2f} us = "
        f"{fused['tops']:.1f} TOP/s, tile {fused['tile']}")
    # the same timed region for the one-launch form of the step
    g_one, one_calls = captured(lambda s: [fused_make(s)], G)
    for _ in range(max(1, args.warmup // G)):
        g_one.replay()
    torch.cuda.synchronize()
    one_calls[0].out.zero_()
    one_calls[0].x_packed.zero_()
    t_wall_one = time.perf_counter()
    ms_total_one = time_graph(g_one, args.steps // G)
    t_wall_one = time.perf_counter() - t_wall_one
    if not (torch.equal(one_calls[0].out, ref_out) and torch.equal(one_calls[0].x_packed, xp)):
        raise RuntimeError("the one-launch step's graph replay differs from the two-launch step's output")
    ms_per_step_one = ms_total_one / args.steps
    log(f"one-launch step: {ms_per_step_one * 1000:.2f} us ({L.ops / (ms_per_step_one * 1e-3) / 1e12:.1f} TOP/s) "
        f"from {args.steps // G} replays of a {G}-step graph, wall {t_wall_one:.3f} s")
    one_form = ms_per_step_one < ms_per_step   # the step's faster form is the one reported
    forms = {"two_launches": {"ms_per_step": round(ms_per_step, 6), "tile": tile_name,
                              "value": round(value, 3)},
             "one_launch": {"ms_per_step": round(ms_per_step_one, 6), "tile": fused["tile"],
                            "value": round(L.ops / (ms_per_step_one * 1e-3) / 1e12, 3)}}
    probe = mfma_probe(dev)
    shapes = mfma_shapes(dev)
    log("MFMA rate at 1 and 2 waves per SIMD (fraction of the matrix cores' rate at the measured clock): "
        + ", ".join(f"{r['instruction'][7:]} x{r['waves_per_simd']} {r['frac_of_rate_at_clock']:.3f}" for r in shapes))
    log(f"pack kernel cold ({n_cp} copies): {pack_cold_us:.2f} us = {pack_bytes / (pack_cold_us * 1e-6) / 1e9:.0f} GB/s; "
        f"MFMA-only probe {probe['tops']:.0f} TOP/s at {probe['clock_ghz']:.2f} GHz")

    workload = (f"conv2d n{L.n} {L.h}x{L.w} {L.c}->{L.k} {L.r}x{L.s} stride {L.stride} pad {L.pad}, "
                f"{L.bits}-bit, fused requant+repack")
    workload_one = workload + ", pack fused in (int8 NCHW input, packed copy written)"
    traffic = measured_traffic(workload, tile_name)
    stats = profile_values("kernel_stats", workload, tile_name)
    traffic_one = measured_traffic(workload_one, fused["tile"] + ":fused")
    stats_one = profile_values("kernel_stats", workload_one, fused["tile"] + ":fused")
    conv()
    geo = qconv.last_launch()
    torch.cuda.synchronize()
    floor = launch_floor(dev, [(geo["grid"], geo["threads"], 0)])[0]
    meeting = grid_meeting(dev, [geo["grid"], 256])
    log(f"launch floor {floor['graph_us']} us; device-wide meeting inside a launch: "
        + ", ".join(f"{m['blocks']} workgroups {m['counting']} {m['us_per_meeting']} us" for m in meeting))
    conv_roofline = {"bound": "mfma", "achieved": round(conv_tops, 3), "peak": INT8_PEAK_TOPS, "unit": "TOP/s",
                     "frac": round(conv_tops / INT8_PEAK_TOPS, 5), "traffic": traffic,
                     "kernel": "conv_wide" if tile_name.startswith("wide") else "conv_staged",
                     "avg_us": round(conv_us, 3), "algorithmic_ops_per_launch": L.ops,
                     "algorithmic_bytes_per_launch": conv_bytes, "kernel_digest": kernel_digest(tile_name),
                     "frac_of_mfma_probe": round(conv_tops / probe["tops"], 5)}
    if stats:
        # the committed kernel-trace summary of this kernel (same sources and tile): its
        # average over the dispatches that started back to back (< 1 us after the
        # previous one ended, as in the timed graph), and over all of them (the
        # tracer's own gaps between dispatches slow the kernel that follows)
        pavg = float(stats["conv_avg_ns_back_to_back"]) / 1000.0
        conv_roofline.update({"profile_avg_us": round(pavg, 3),
                              "profile_frac": round(L.ops / (pavg * 1e-6) / 1e12 / INT8_PEAK_TOPS, 5),
                              "profile_avg_us_all_dispatches": round(float(stats["conv_avg_ns"]) / 1000.0, 3),
                              "profile": stats["file"]})
    # the one-launch kernel reads the int8 input and writes its packed copy too
    one_bytes = conv_bytes + L.n * L.c * L.h * L.w
    one_tops = L.ops / (fused["us"] * 1e-6) / 1e12
    one_roofline = {"bound": "mfma", "achieved": round(one_tops, 3), "peak": INT8_PEAK_TOPS, "unit": "TOP/s",
                    "frac": round(one_tops / INT8_PEAK_TOPS, 5), "traffic": traffic_one,
                    "kernel": "conv_wide (int8 NCHW input: the pack fused in)", "avg_us": fused["us"],
                    "algorithmic_ops_per_launch": L.ops, "algorithmic_bytes_per_launch": one_bytes,
                    "kernel_digest": kernel_digest(fused["tile"] + ":fused"),
                    "frac_of_mfma_probe": round(one_tops / probe["tops"], 5),
                    "hbm_frac": round(one_bytes / (fused["us"] * 1e-6) / 1e9 / HBM_PEAK_GBS, 5)}
    if stats_one:
        pavg = float(stats_one["conv_avg_ns_back_to_back"]) / 1000.0
        one_roofline.update({"profile_avg_us": round(pavg, 3),
                             "profile_frac": round(L.ops / (pavg * 1e-6) / 1e12 / INT8_PEAK_TOPS, 5),
                             "profile_avg_us_all_dispatches": round(float(stats_one["conv_avg_ns"]) / 1000.0, 3),
                             "profile": stats_one["file"]})
    result = {
        "metric": METRIC,
        "value": round(L.ops / (ms_per_step_one * 1e-3) / 1e12 if one_form else value, 3),
        "unit": "TOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step_one if one_form else ms_per_step, 6),
        "eager_ms_per_step": round(eager_ms, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int4",
        "data": "synthetic",
        "config": {"workload": workload,
                   "step": ("qconv2d_packing: int8 NCHW activations packed while the convolution stages them, "
                            "packed copy written (one launch)") if one_form else
                           "qconv_pack (int8 NCHW -> packed 4-bit NHWC) + qconv2d (two launches)",
                   "n": L.n, "h": L.h, "w": L.w, "c": L.c, "k": L.k, "r": L.r, "s": L.s, "stride": L.stride,
                   "pad": L.pad, "bits": L.bits, "ops_per_step": L.ops,
                   "tile": fused["tile"] if one_form else tile_name, "step_forms": forms},
        "roofline": one_roofline if one_form else conv_roofline,
        "roofline_packed_input_conv": conv_roofline,
        "kernels": {"conv_us": round(conv_us, 3), "pack_us": round(pack_us, 3),
                    "pack_gbs": round(pack_gbs, 1), "pack_frac_hbm": round(pack_gbs / HBM_PEAK_GBS, 4),
                    "pack_algorithmic_bytes": pack_bytes, "pack_cold_us": round(pack_cold_us, 3),
                    "pack_cold_gbs": round(pack_bytes / (pack_cold_us * 1e-6) / 1e9, 1), "pack_cold_copies": n_cp,
                    "fused_step": fused},
        "mfma_probe": probe,
        "mfma_shapes": shapes,
        "launch_floor": {"grid": floor, "note": "empty kernel over the conv kernel's grid (qconv_probe_launch)",
                         "grid_meeting": meeting,
                         "grid_meeting_note": "one device-wide meeting inside a launch (qconv_probe_grid_meet): what "
                                              "a persistent multi-layer launch pays per layer boundary"},
        "build": {"source_digest": hip_build.source_digest(), "library_digest": qconv.build_digest()},
    }

    tables = [] if args.tables == "none" else [int(v) for v in args.tables.split(",") if v]
    for cfg in tables:
        layers = qi.WORKLOADS[cfg]()
        log(f"workload {cfg}: per-layer ({len(qi.distinct(layers)) if cfg in (2, 3) else len(layers)} layers)")
        rows = per_layer_table(cfg, qi.distinct(layers) if cfg in (2, 3) else layers, dev, args.layer_reps)
        entry = {"per_layer": rows}
        if cfg in (2, 3):
            entry["proj_fused"] = proj_table(cfg, layers, dev, args.layer_reps)
            entry["chain"] = chain_time(cfg, layers, dev, max(20, args.layer_reps // 4))
            log(f"  chained network: {entry['chain']}")
            entry["chain_residual"] = chain_time(cfg, layers, dev, max(20, args.layer_reps // 4), residual=True)
            log(f"  as residual blocks with biases: {entry['chain_residual']}")
        if cfg == 3:
            entry["stem"] = stem_time(dev, 16, max(20, args.layer_reps // 4))
            log(f"  stem: {entry['stem']}")
        if cfg == 4:
            entry["bottleneck_stack"] = bottleneck_stack_time(dev, max(10, args.layer_reps // 10))
            log(f"  bottleneck stack: {entry['bottleneck_stack']}")
        result[f"workload{cfg}"] = entry
        if cfg == 2:
            # the stated goal: the batch-16 4-bit 3x3 stride-1 layers at >= 50 % of the int8 peak
            tgt = [r for r in rows if "3x3" in qi_shape(layers, r["layer"]) and "s1" in qi_shape(layers, r["layer"])]
            result["target"] = {
                "what": "ResNet-18 4-bit 3x3 stride-1 layers at N=16, % of the 5.0 POP/s dense int8 peak",
                "goal_pct": 50.0,
                "layers": [{"layer": r["layer"], "shape": qi_shape(layers, r["layer"]), "us": r["us"],
                            "tops": r["tops"], "pct_int8_peak": r["pct_int8_peak"]} for r in tgt],
                "met": all(r["pct_int8_peak"] >= 50.0 for r in tgt) if tgt else False,
            }
            if "chain" in entry:
                result["target"]["chain_graph_us"] = entry["chain"].get("graph_us")

    if args.launch_floor:
        log("launch floor: empty kernel, back to back in a replayed graph")
        result["launch_floor"]["sweep"] = launch_floor(dev, [(b, t, l) for b in (196, 256, 512, 1024, 2048)
                                                             for t in (256, 512) for l in (0, 48 << 10)])

    if args.layout_table:
        log("layouts: plain NHWC vs batch-interleaved (nb images per pixel)")
        result["layouts"] = layout_table(dev, max(20, args.layer_reps // 4))

    if args.batch_table:
        log("batch scaling: 4-bit 3x3 stride-1 ResNet-18 layers, best tile per batch")
        result["batch_scaling"] = batch_table(dev, max(20, args.layer_reps // 4))

    if not args.no_cpu:
        log(f"cpu baseline: oracle for ~{args.cpu_seconds:.0f} s ...")
        result["cpu_baseline"] = cpu_baseline(L, args.cpu_seconds)
        one = cpu_baseline(L, max(1.0, args.cpu_seconds / 3), threads=1)
        result["cpu_baseline"]["single_core"] = {"value": one["value"], "unit": one["unit"], "sample": one["sample"]}
        log(f"  {result['cpu_baseline']}")
        if args.cpu_networks:
            result["cpu_baseline"]["networks"] = cpu_network_times((2, 4), single_thread_cfgs=(2,))
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
