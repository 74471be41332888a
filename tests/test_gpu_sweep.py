"""The tile sweep harness (the exhaustive schedule measurement) run on small
shapes with the oracle's output as the reference: every (tile, split)
candidate it times must reproduce the oracle's bytes, and the table it
returns names every valid candidate once.  Also the sweep of the fused
projection layers."""
import numpy as np
import pytest

import oracle
import qconv_inputs as qi
from _util import announce, oracle_threads, stress_shift

pytestmark = pytest.mark.gpu

SHAPES = [
    qi.Layer("sw4_2x14x14_128to64_3x3", 2, 14, 14, 128, 64, 3, 3, 1, 1, w_range=(-7, 7)),
    qi.Layer("sw8_1x9x9_64to128_1x1_s2", 1, 9, 9, 64, 128, 1, 1, 2, 0, bits=8, x_signed=True, w_signed=True,
             x_range=qi.S8, w_range=qi.S8, epilogue=None),
]


@pytest.mark.parametrize("lid", range(len(SHAPES)), ids=[L.name for L in SHAPES])
def test_sweep_candidates_match_the_oracle(lid):
    import torch
    from paper_2202_06819_amd import qconv, sweep
    L = SHAPES[lid]
    dev = torch.device("cuda:0")
    t = qi.layer_tensors(90, lid, L)
    d = L.desc()
    requant = L.epilogue is not None
    sh = stress_shift(L, L.x_range, L.w_range) if requant else 20
    kw = dict(mult=t["mult"], shift=sh, relu=True, lo=0, hi=15) if requant else {}
    ref = oracle.qconv_layer(t["x"], t["w"], bits=L.bits, x_signed=L.x_signed, w_signed=L.w_signed,
                             stride=(L.stride, L.stride), pad=(L.pad, L.pad), threads=oracle_threads(), **kw)
    want = ref["y_packed"] if requant else ref["acc"]
    x = qconv.pack(torch.from_numpy(t["x"]).to(dev), L.bits, L.x_signed)
    w = qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
    mult = torch.from_numpy(t["mult"]).to(dev) if requant else None
    expected = torch.from_numpy(np.ascontiguousarray(want).view(np.int32 if L.bits == 4 or not requant else np.int8))
    announce(f"sweep {L.name} against the oracle")
    rows = sweep.sweep_layer(d, x, w, mult, shift=sh, relu=True, clamp=(0, 15), reps=3, rounds=1,
                             expected=expected, log=lambda s: None)
    want_rows = {(tt["name"], sp) for tt in qconv.tiles() if qconv.tile_status(d, tt["id"]) == 0
                 for sp in sweep.split_choices(d, tt["id"])}
    assert {(r["tile"], r["splits"]) for r in rows} == want_rows and len(rows) == len(want_rows)
    assert all(r["identical"] for r in rows)
    assert any(r["splits"] > 1 for r in rows) == any(sp > 1 for _, sp in want_rows)
    best = sweep.best_per_shape(rows)[sweep.shape_key(d, requant)]
    assert best["us"] == min(r["us"] for r in rows)


def test_proj_sweep_candidates_match_the_oracle():
    import torch
    from paper_2202_06819_amd import qconv, sweep
    L = qi.Layer("swp4_2x10x10_64to64_s2", 2, 10, 10, 64, 64, 3, 3, 2, 1, w_range=(-7, 7))
    dev = torch.device("cuda:0")
    t = qi.layer_tensors(91, 0, L)
    w1 = qi.draw_int8(np.random.default_rng([91, 0, 5]), (L.k, L.c, 1, 1), -7, 7)
    mult2 = np.random.default_rng([91, 0, 6]).integers(1 << 14, 1 << 15, size=L.k).astype(np.int32)
    sh = stress_shift(L, L.x_range, L.w_range)
    kw = dict(bits=4, x_signed=False, w_signed=True, stride=(2, 2), threads=oracle_threads())
    r3 = oracle.qconv_layer(t["x"], t["w"], pad=(1, 1), mult=t["mult"], shift=sh, relu=True, lo=0, hi=15, **kw)
    r1 = oracle.qconv_layer(t["x"], w1, pad=(0, 0), mult=mult2, shift=sh - 2, relu=False, lo=0, hi=15, **kw)
    x = qconv.pack(torch.from_numpy(t["x"]).to(dev), 4, False)
    w3p = qconv.pack(torch.from_numpy(t["w"]).to(dev), 4, True)
    w1p = qconv.pack(torch.from_numpy(w1).to(dev), 4, True)
    expected = (torch.from_numpy(r3["y_packed"].view(np.int32)), torch.from_numpy(r1["y_packed"].view(np.int32)))
    announce(f"proj sweep {L.name} against the oracle")
    rows = sweep.sweep_proj_layer(L.desc(), x, w3p, w1p, torch.from_numpy(t["mult"]).to(dev),
                                  torch.from_numpy(mult2).to(dev), shift=sh, shift2=sh - 2, relu=True, relu2=False,
                                  clamp=(0, 15), reps=3, rounds=1, expected=expected, log=lambda s: None)
    want = {tt["name"] for tt in qconv.tiles() if qconv.proj_tile_status(L.desc(), tt["id"]) == 0}
    assert {r["tile"] for r in rows} == want and len(rows) == len(want) >= 2
    assert all(r["identical"] for r in rows)
