"""A 1x1 projection fused into a 3x3 launch (qconv2d_proj) against the oracle,
element by element: both outputs -- the 3x3 layer's and the projection's --
as raw int32 accumulators and requantised (each with its own multipliers,
shift, clamp and optional bias), on every tile that has a projection
instance, without and with split-K (each split call made twice on one
workspace), on small ragged shapes (odd sizes, several channel chunks, 4-bit
and 8-bit, stride 2 and 1) and on the three stage entries of the ResNet-18
stacks at full size in the configuration the chain runs."""
import numpy as np
import pytest

import oracle
import qconv_inputs as qi
from _util import announce, assert_same, oracle_threads, stress_shift

pytestmark = pytest.mark.gpu


def _layer(name, n, h, w, c, k, stride, bits):
    if bits == 4:
        return qi.Layer(name, n, h, w, c, k, 3, 3, stride, 1, w_range=(-7, 7))
    return qi.Layer(name, n, h, w, c, k, 3, 3, stride, 1, bits=8, x_signed=True, w_signed=True, x_range=qi.S8,
                    w_range=qi.S8, epilogue=qi.Epilogue(relu=False, lo=-128, hi=127))


SMALL = [
    _layer("p4_2x9x9_64to64_s2", 2, 9, 9, 64, 64, 2, 4),
    _layer("p4_1x15x13_128to128_s2", 1, 15, 13, 128, 128, 2, 4),
    _layer("p4_3x10x10_64to128_s1", 3, 10, 10, 64, 128, 1, 4),
    _layer("p4_2x14x14_256to64_s2", 2, 14, 14, 256, 64, 2, 4),
    _layer("p8_2x11x11_64to64_s2", 2, 11, 11, 64, 64, 2, 8),
    _layer("p8_1x14x14_256to128_s2", 1, 14, 14, 256, 128, 2, 8),
]


def _tensors(wid, lid, L):
    """x, the 3x3 filters, the projection's 1x1 filters, both multiplier sets and biases."""
    t = qi.layer_tensors(wid, lid, L)
    g = np.random.default_rng([wid, lid, 5])
    t["w1"] = qi.draw_int8(g, (L.k, L.c, 1, 1), *L.w_range)
    lo, hi = qi.MULT
    t["mult2"] = np.random.default_rng([wid, lid, 6]).integers(lo, hi, size=L.k).astype(np.int32)
    t["bias"] = np.random.default_rng([wid, lid, 7]).integers(-2000, 2000, size=L.k).astype(np.int32)
    t["bias2"] = np.random.default_rng([wid, lid, 8]).integers(-2000, 2000, size=L.k).astype(np.int32)
    return t


def _refs(L, t, shift, shift2, bias):
    kw = dict(bits=L.bits, x_signed=L.x_signed, w_signed=L.w_signed, threads=oracle_threads())
    e = L.epilogue
    r3 = oracle.qconv_layer(t["x"], t["w"], stride=(L.stride, L.stride), pad=(1, 1), mult=t["mult"], shift=shift,
                            relu=e.relu, lo=e.lo, hi=e.hi, bias=t["bias"] if bias else None, **kw)
    r1 = oracle.qconv_layer(t["x"], t["w1"], stride=(L.stride, L.stride), pad=(0, 0), mult=t["mult2"], shift=shift2,
                            relu=False, lo=e.lo, hi=e.hi, bias=t["bias2"] if bias else None, **kw)
    return r3, r1


def _check_layer(L, t, tile, shifts, label, splits=(1,)):
    import torch
    from paper_2202_06819_amd import qconv
    dev = torch.device("cuda:0")
    d = L.desc()
    e = L.epilogue
    xp = qconv.pack(torch.from_numpy(t["x"]).to(dev), L.bits, L.x_signed)
    w3 = qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
    w1 = qconv.pack(torch.from_numpy(t["w1"]).to(dev), L.bits, L.w_signed)
    wprep = qconv.prepare_filters_proj(d, w3, w1, tile)
    dv = {k: torch.from_numpy(t[k]).to(dev) for k in ("mult", "mult2", "bias", "bias2")}
    refs = {}

    def ref(shift, shift2, bias):
        if (shift, shift2, bias) not in refs:
            refs[(shift, shift2, bias)] = _refs(L, t, shift, shift2, bias)
        return refs[(shift, shift2, bias)]

    for sp in splits:
        nws = qconv.proj_workspace_bytes(d, tile, sp)
        ws = torch.zeros(nws, dtype=torch.uint8, device=dev) if nws else None
        rounds = 2 if sp > 1 else 1   # a split call leaves its workspace ready for the next
        announce(f"proj {label} {L.name} tile {tile} splits {sp} raw")
        call = qconv.ProjConv2dCall(d, xp, wprep, tile=tile, splits=sp, workspace=ws)
        r3, r1 = ref(shifts[0][0], shifts[0][1], False)
        for rnd in range(rounds):
            y, yp = call()
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), r3["acc"], f"{L.name} tile {tile} splits {sp} ({rnd}): 3x3 accumulators")
            assert_same(yp.cpu().numpy(), r1["acc"], f"{L.name} tile {tile} splits {sp} ({rnd}): projection "
                                                     f"accumulators")
        for shift, shift2 in shifts:
            for bias in (False, True):
                announce(f"proj {label} {L.name} tile {tile} splits {sp} shifts {shift}/{shift2} bias {bias}")
                call = qconv.ProjConv2dCall(d, xp, wprep, tile=tile, requant=True, mult=dv["mult"], shift=shift,
                                            relu=e.relu, clamp=(e.lo, e.hi), bias=dv["bias"] if bias else None,
                                            proj=dict(mult=dv["mult2"], shift=shift2, relu=False, clamp=(e.lo, e.hi),
                                                      bias=dv["bias2"] if bias else None), splits=sp, workspace=ws)
                r3, r1 = ref(shift, shift2, bias)
                for rnd in range(rounds):
                    y, yp = call()
                    torch.cuda.synchronize()
                    what = f"{L.name} tile {tile} splits {sp} ({rnd}) shift {shift}/{shift2} bias {bias}"
                    assert_same(y.cpu().numpy(), r3["y_packed"], f"{what}: 3x3")
                    assert_same(yp.cpu().numpy(), r1["y_packed"], f"{what}: proj")


@pytest.mark.parametrize("lid", range(len(SMALL)))
def test_proj_every_tile_small(lid):
    from paper_2202_06819_amd import qconv
    L = SMALL[lid]
    t = _tensors(80, lid, L)
    s3 = stress_shift(L, L.x_range, L.w_range)
    s1 = stress_shift(qi.Layer("p", L.n, L.h, L.w, L.c, L.k, 1, 1, bits=L.bits), L.x_range, L.w_range)
    tiles = [tt["id"] for tt in qconv.tiles() if qconv.proj_tile_status(L.desc(), tt["id"]) == 0]
    assert tiles, f"no projection tile fits {L.name}"
    for tile in tiles:
        chunks = qconv.max_splits(L.desc(), tile)
        _check_layer(L, t, tile, [(s3, s1)], "small", splits=sorted({1, 2, chunks} & set(range(1, chunks + 1))))


@pytest.mark.parametrize("first", [0, 20, 40])
def test_proj_random_shapes(first):
    """Random shapes (batch 1-12, 2-40 pixels a side, stride 1 or 2, 32-320
    input and 8-320 output channels, 4-bit and 8-bit) on every tile with a
    projection instance, without a split and with a random one."""
    from paper_2202_06819_amd import qconv
    ran = 0
    for seed in range(first, first + 20):
        g = np.random.default_rng([5151, seed])
        bits = 8 if seed % 3 == 2 else 4
        stride = int(g.choice([1, 2, 2]))
        n, h, w = int(g.integers(1, 13)), int(g.integers(2, 41)), int(g.integers(2, 41))
        c, k = 32 * int(g.integers(1, 11)), 8 * int(g.integers(1, 41))
        L = _layer(f"pr{seed}", n, h, w, c, k, stride, bits)
        tiles = [tt["id"] for tt in qconv.tiles() if qconv.proj_tile_status(L.desc(), tt["id"]) == 0]
        assert tiles, f"no projection tile fits {L.desc()}"
        t = _tensors(5151, seed, L)
        s3 = stress_shift(L, L.x_range, L.w_range)
        s1 = stress_shift(qi.Layer("p", L.n, L.h, L.w, L.c, L.k, 1, 1, bits=L.bits), L.x_range, L.w_range)
        for tile in tiles:
            chunks = qconv.max_splits(L.desc(), tile)
            splits = sorted({1} | ({int(g.integers(2, chunks + 1))} if chunks >= 2 else set()))
            _check_layer(L, t, tile, [(s3, s1)], "random", splits=splits)
            ran += 1
    assert ran > 0


def _stage_entries(cfg):
    """(3x3 stride-2 layer, its 1x1 projection, their workload layer ids) of a ResNet-18 stack."""
    layers = qi.WORKLOADS[cfg]()
    names = [L.name for L in layers]
    out = []
    for i, L in enumerate(layers):
        if L.name.endswith(".0.conv1") and L.stride == 2:
            j = names.index(L.name.replace("conv1", "downsample"))
            out.append((L, layers[j], i, j))
    return out


@pytest.mark.parametrize("cfg", [2, 3])
def test_proj_stage_entries_full_size(cfg):
    """The stage entries of the ResNet-18 stacks at N=16 with their own seeded
    inputs (the 3x3 layer's x, filters and multipliers; the projection's
    filters and multipliers), the tuned tile, the literal epilogues and ones
    that spread outputs over the clamp range."""
    from paper_2202_06819_amd import qconv, sweep
    for L, P, i, j in _stage_entries(cfg):
        t = qi.layer_tensors(cfg, i, L)
        tp = qi.layer_tensors(cfg, j, P)
        t["w1"], t["mult2"] = tp["w"], tp["mult"]
        g = np.random.default_rng([cfg, i, 9])
        t["bias"] = g.integers(-256, 256, size=L.k).astype(np.int32)
        t["bias2"] = g.integers(-256, 256, size=L.k).astype(np.int32)
        tile, splits = sweep.tuned_proj_config(L.desc())
        e = L.epilogue
        shifts = [(e.shift, P.epilogue.shift),
                  (stress_shift(L, L.x_range, L.w_range), stress_shift(P, P.x_range, P.w_range))]
        other = 2 if splits == 1 and qconv.max_splits(L.desc(), tile) >= 2 else 1
        _check_layer(L, t, tile, shifts, f"workload {cfg}", splits=sorted({splits, other}))


def test_proj_rejects_what_it_does_not_run():
    import torch
    from paper_2202_06819_amd import qconv
    L = SMALL[0]
    d = L.desc()
    assert qconv.proj_tile_status(dict(d, pad_h=0, pad_w=0), qconv.proj_default_tile(d)) == qconv.EUNSUPPORTED
    assert qconv.proj_tile_status(dict(d, r=1, s=1, pad_h=0, pad_w=0), 0) == qconv.EUNSUPPORTED
    no_proj = [tt["id"] for tt in qconv.tiles() if tt["bits"] == 4 and tt["variant"] == 2
               and qconv.tile_status(d, tt["id"]) == 0 and qconv.proj_tile_status(d, tt["id"]) != 0]
    assert no_proj, "every fitting tile has a projection instance"
    torch.cuda.synchronize()
