"""GPU parity: the HIP path (qconv_pack + qconv2d through the C ABI) against the
CPU oracle, bit for bit, on seeded inputs.

Integer sums have exactly one value, so every tile, every shape and every
run must reproduce the oracle's bytes: packed inputs, raw int32 accumulators
and requantised packed outputs.
"""
import numpy as np
import pytest

import oracle
import qconv_inputs as qi
from _util import announce, assert_same, gpu_layer, oracle_threads, ref_layer, stress_shift, unroll_def

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


def _qconv():
    from paper_2202_06819_amd import qconv
    return qconv


def _valid_tiles(L):
    q = _qconv()
    return [t["id"] for t in q.tiles() if q.tile_status(L.desc(), t["id"]) == 0]


# ----------------------------------------------------------------- qconv_pack

PACK_CASES = [
    # n, c, h, w, bits, signed, value range
    (8, 64, 56, 56, 4, False, (-128, 127)),
    (1, 8, 5, 7, 4, False, (-20, 30)),
    (2, 72, 3, 11, 4, True, (-128, 127)),
    (3, 136, 9, 9, 4, True, (-9, 9)),
    (64, 64, 3, 3, 4, True, (-8, 7)),           # filters K x C x R x S
    (4, 64, 28, 28, 4, False, (0, 15)),         # every value in range (no clamping needed)
    (2, 32, 14, 14, 4, True, (-8, 7)),
    (2, 32, 14, 14, 4, True, (-9, 8)),          # just outside both ends
    (2, 64, 56, 56, 8, True, (-128, 127)),
    (1, 20, 7, 5, 8, True, (-128, 127)),
    (2, 100, 1, 1, 8, True, (-128, 127)),
]


@pytest.mark.parametrize("case", PACK_CASES, ids=lambda c: "n%d_c%d_%dx%d_b%d_%s" % (c[:5] + ("s" if c[5] else "u",)))
def test_pack_matches_oracle(case):
    torch, q = _torch(), _qconv()
    n, c, h, w, bits, signed, (lo, hi) = case
    src = np.random.default_rng([7, n, c, h, w, bits]).integers(lo, hi + 1, size=(n, c, h, w)).astype(np.int8)
    ref = oracle.relayout_pack(src, bits, signed)
    announce(f"qconv_pack {case}")
    got = q.pack(torch.from_numpy(src).cuda(), bits, signed)
    torch.cuda.synchronize()
    assert_same(got.cpu().numpy(), ref, "pack")


def test_pack_zero_size_is_noop():
    torch, q = _torch(), _qconv()
    src = torch.empty((0, 64, 4, 4), dtype=torch.int8, device="cuda")
    out = q.pack(src, 4, False)
    torch.cuda.synchronize()
    assert out.numel() == 0


# ----------------------------------------------------------------- configs 0 and 1 at full size

def test_config0_raw_every_tile():
    L = qi.workload0()[0]
    t = qi.layer_tensors(0, 0, L)
    ref = ref_layer(L, t, requant=False)
    for tid in _valid_tiles(L):
        announce(f"workload0 raw tile {tid}")
        got = gpu_layer(L, t, requant=False, tile=tid)
        assert_same(got["x_packed"], ref["x_packed"], "x packed")
        assert_same(got["w_packed"], ref["w_packed"], "w packed")
        assert_same(got["y"], ref["acc"], f"raw acc tile {tid}")
        announce(f"workload0 raw tile {tid} prepared filters")
        assert_same(gpu_layer(L, t, requant=False, tile=tid, prepared=True)["y"], ref["acc"], f"prepared tile {tid}")


def test_config1_requant_every_tile():
    L = qi.workload1()[0]
    t = qi.layer_tensors(1, 0, L)
    ref = ref_layer(L, t, requant=True)
    for tid in _valid_tiles(L):
        announce(f"workload1 requant tile {tid}")
        got = gpu_layer(L, t, requant=True, tile=tid)
        assert_same(got["y"], ref["y_packed"], f"requant tile {tid}")
        announce(f"workload1 requant tile {tid} prepared filters")
        got = gpu_layer(L, t, requant=True, tile=tid, prepared=True)
        assert_same(got["y"], ref["y_packed"], f"requant tile {tid} prepared")


@pytest.mark.parametrize("shape", [
    # name, n, h, c, k, r, stride, pad -- the strided and 1x1 layers of the ResNet stacks
    ("ds1x1_s2_64to128", 2, 56, 64, 128, 1, 2, 0),
    ("conv3x3_s2_64to128", 2, 56, 64, 128, 3, 2, 1),
    ("conv1x1_s1_256to64", 2, 28, 256, 64, 1, 1, 0),
    ("conv3x3_s1_512to512", 2, 7, 512, 512, 3, 1, 1),
], ids=lambda v: v[0])
def test_resnet_shapes_every_tile_prepared(shape):
    """Every tile that runs the shape, from packed and from prepared filters
    (prepared 3x3 and 1x1 layers run the fixed-size kernel instances)."""
    name, n, h, c, k, r, stride, pad = shape
    L = qi.Layer(name, n, h, h, c, k, r, r, stride, pad, w_range=(-7, 7))
    t = qi.layer_tensors(500, r * 10 + stride, L)
    sh = stress_shift(L, L.x_range, L.w_range)
    ref = ref_layer(L, t, requant=True, shift=sh)
    ref_raw = ref_layer(L, t, requant=False)
    for tid in _valid_tiles(L):
        announce(f"{name} tile {tid} prepared requant shift={sh}")
        assert_same(gpu_layer(L, t, requant=True, tile=tid, shift=sh, prepared=True)["y"], ref["y_packed"],
                    f"{name} tile {tid} prepared")
        announce(f"{name} tile {tid} prepared raw")
        assert_same(gpu_layer(L, t, requant=False, tile=tid, prepared=True)["y"], ref_raw["acc"],
                    f"{name} tile {tid} prepared raw")


@pytest.mark.parametrize("shape", [
    # name, n, h, c, k, r, stride, pad -- enough output tiles that workgroups walk several
    # of them (persistent plans, with one or two LDS band buffers)
    ("n32_56_64to64_3x3", 32, 56, 64, 64, 3, 1, 1),
    ("n64_56_64to256_1x1", 64, 56, 64, 256, 1, 1, 0),
    ("n64_28_128to128_3x3", 64, 28, 128, 128, 3, 1, 1),
], ids=lambda v: v[0])
def test_persistent_plans_every_wide_tile(shape):
    """Large batches, where each workgroup stages several output tiles in turn."""
    q = _qconv()
    name, n, h, c, k, r, stride, pad = shape
    L = qi.Layer(name, n, h, h, c, k, r, r, stride, pad, w_range=(-7, 7))
    t = qi.layer_tensors(600, c + k + r, L)
    sh = stress_shift(L, L.x_range, L.w_range)
    ref = ref_layer(L, t, requant=True, shift=sh)
    ref_raw = ref_layer(L, t, requant=False)
    wide = [tt["id"] for tt in q.tiles() if tt["variant"] == 2 and q.tile_status(L.desc(), tt["id"]) == 0]
    assert wide
    for tid in wide:
        announce(f"{name} tile {tid} prepared requant shift={sh}")
        assert_same(gpu_layer(L, t, requant=True, tile=tid, shift=sh, prepared=True)["y"], ref["y_packed"],
                    f"{name} tile {tid} prepared")
    announce(f"{name} tile {wide[0]} prepared raw")
    assert_same(gpu_layer(L, t, requant=False, tile=wide[0], prepared=True)["y"], ref_raw["acc"],
                f"{name} tile {wide[0]} prepared raw")


def test_config1_raw_default_tile():
    L = qi.workload1()[0]
    t = qi.layer_tensors(1, 0, L)
    ref = ref_layer(L, t, requant=False)
    announce("workload1 raw default tile")
    assert_same(gpu_layer(L, t, requant=False)["y"], ref["acc"], "raw acc")


# ----------------------------------------------------------------- ragged random shapes

def _random_layer(seed: int) -> qi.Layer:
    g = np.random.default_rng([99, seed])
    bits = 8 if seed % 4 == 3 else 4
    r = int(g.choice([1, 2, 3, 5, 7]))
    s = int(g.choice([1, 3, r]))
    stride = int(g.choice([1, 1, 2, 3]))
    pad = int(g.integers(0, (max(r, s) // 2) + 2))
    h = int(g.integers(max(1, r - 2 * pad), 24))
    w = int(g.integers(max(1, s - 2 * pad), 24))
    if bits == 4:
        c = 8 * int(g.integers(1, 26))
        k = 8 * int(g.integers(1, 18))
        xs = bool(seed % 5 == 1)
        ws = not (seed % 7 == 2)
        xr = qi.S4 if xs else qi.U4
        wr = qi.S4 if ws else qi.U4
        epi = qi.Epilogue(relu=bool(seed % 2), lo=-8 if seed % 3 == 0 else 0, hi=7 if seed % 3 == 0 else 15)
        return qi.Layer(f"rand{seed}", int(g.integers(1, 4)), h, w, c, k, r, s, stride, pad, 4, xs, ws, xr, wr, epi)
    c = 4 * int(g.integers(1, 50))
    k = 4 * int(g.integers(1, 34))
    epi = qi.Epilogue(relu=bool(seed % 2), lo=-128, hi=127)
    return qi.Layer(f"rand{seed}", int(g.integers(1, 4)), h, w, c, k, r, s, stride, pad, 8, True, True, qi.S8, qi.S8,
                    epi)


@pytest.mark.parametrize("seed", range(32))
def test_random_shape(seed):
    L = _random_layer(seed)
    if L.h + 2 * L.pad < L.r or L.w + 2 * L.pad < L.s:
        pytest.skip("window larger than padded input")
    t = qi.layer_tensors(100, seed, L)
    sh = stress_shift(L, L.x_range, L.w_range)
    ref_raw = ref_layer(L, t, requant=False)
    ref_req = ref_layer(L, t, requant=True, shift=sh)
    tiles = _valid_tiles(L)
    assert tiles, "no tile fits"
    pick = [-1, tiles[seed % len(tiles)], tiles[-1]]
    for tid in pick:
        announce(f"random seed={seed} {L} tile={tid} raw")
        assert_same(gpu_layer(L, t, requant=False, tile=tid)["y"], ref_raw["acc"], f"raw tile {tid}")
        announce(f"random seed={seed} tile={tid} requant shift={sh}")
        assert_same(gpu_layer(L, t, requant=True, tile=tid, shift=sh)["y"], ref_req["y_packed"], f"requant tile {tid}")
        announce(f"random seed={seed} tile={tid} requant shift={sh} prepared filters")
        assert_same(gpu_layer(L, t, requant=True, tile=tid, shift=sh, prepared=True)["y"], ref_req["y_packed"],
                    f"requant tile {tid} prepared")


# ----------------------------------------------------------------- epilogue stress

@pytest.mark.parametrize("bits", [4, 8])
def test_epilogue_spread_and_ties(bits):
    """Zero-mean filters and a shift that spreads outputs over the whole clamp
    range; then mult = 2^14, shift = 20 makes every acc = 32 (mod 64) an exact
    rounding tie."""
    if bits == 4:
        L = qi.Layer("stress4", 4, 28, 28, 128, 64, 3, 3, 1, 1, w_range=(-7, 7))
    else:
        L = qi.Layer("stress8", 2, 28, 28, 64, 64, 3, 3, 1, 1, 8, True, True, qi.S8, qi.S8,
                     qi.Epilogue(relu=False, lo=-128, hi=127))
    t = qi.layer_tensors(200, bits, L)
    sh = stress_shift(L, L.x_range, L.w_range)
    for relu, lo, hi in ((True, 0, 15), (False, -8, 7)) if bits == 4 else ((False, -128, 127), (True, -128, 127)):
        ref = ref_layer(L, t, requant=True, shift=sh, relu=relu, lo=lo, hi=hi)
        vals = ref["y"]
        assert len(np.unique(vals)) >= (12 if bits == 4 else 100), "stress case does not spread"
        announce(f"stress bits={bits} relu={relu} clamp=({lo},{hi}) shift={sh}")
        got = gpu_layer(L, t, requant=True, shift=sh, relu=relu, lo=lo, hi=hi)
        assert_same(got["y"], ref["y_packed"], "stress requant")
    # exact ties
    t2 = dict(t, mult=np.full(L.k, 1 << 14, dtype=np.int32))
    ref = ref_layer(L, t2, requant=True, shift=20, relu=False, lo=lo, hi=hi)
    ties = int(((ref["acc"].astype(np.int64) % 64) == 32).sum())
    assert ties > 100
    announce(f"ties bits={bits} count={ties}")
    got = gpu_layer(L, t2, requant=True, shift=20, relu=False, lo=lo, hi=hi)
    assert_same(got["y"], ref["y_packed"], "ties")


# ----------------------------------------------------------------- operands at the accumulator bound

# The requantiser's shift for these cases: with multipliers near 2^14.5 an
# output is about acc / 2^9.5, so the two-ends 4-bit outputs spread over the
# clamp range while the constant ones and most 8-bit ones saturate.
SHIFT_EXTREME = 24

EXTREME_CASES = [
    # name, n, h, w, c, k, r, stride, pad, bits, x_signed, (x extremes), (w extremes)
    ("u4_15_by_m8_c256_3x3_ragged", 3, 13, 11, 256, 72, 3, 1, 1, 4, False, (15, 0), (-8, 7)),
    ("s4_m8_by_m8_c512_3x3", 2, 9, 9, 512, 64, 3, 1, 1, 4, True, (-8, 7), (-8, 7)),
    ("s8_m128_by_m128_c512_3x3", 2, 9, 9, 512, 64, 3, 1, 1, 8, True, (-128, 127), (-128, 127)),
    ("s8_m128_by_127_c2048_1x1", 2, 7, 7, 2048, 64, 1, 1, 0, 8, True, (-128, 127), (127, -128)),
    ("s8_127_by_127_c256_5x5_s2", 2, 11, 11, 256, 32, 5, 2, 2, 8, True, (127, -128), (127, -128)),
]


def _valid_tap_counts(h, w, r, s, stride, pad):
    """Per output pixel, the number of filter taps that land inside the image."""
    p = (h + 2 * pad - r) // stride + 1
    q = (w + 2 * pad - s) // stride + 1
    rows = np.array([sum(0 <= i * stride - pad + a < h for a in range(r)) for i in range(p)], dtype=np.int64)
    cols = np.array([sum(0 <= j * stride - pad + b < w for b in range(s)) for j in range(q)], dtype=np.int64)
    return rows[:, None] * cols[None, :]


@pytest.mark.parametrize("case", EXTREME_CASES, ids=[c[0] for c in EXTREME_CASES])
def test_extreme_operands_every_tile(case):
    """Sec. 3.2.1: the int32 accumulator must hold C*R*S products of the
    largest magnitudes.  Constant operands at one extreme give the closed form
    x*w*C*(valid taps) (checked on the oracle first), then operands drawn from
    the two ends of their ranges exercise the signs at the same magnitude; every
    tile that runs the shape (and the wide ones at their largest split) must reproduce
    the oracle, raw and requantised (the requantiser's product acc*mult exceeds
    32 bits here)."""
    torch, q = _torch(), _qconv()
    name, n, h, w, c, k, r, stride, pad, bits, xs, xe, we = case
    xr = (min(xe), max(xe)) if bits == 8 or xs else (0, 15)
    wr = (min(we), max(we))
    L = qi.Layer(name, n, h, w, c, k, r, r, stride, pad, bits, xs, True, xr, wr)
    assert q.layout(L.desc())["max_abs_acc"] >= abs(xe[0] * we[0]) * c * r * r
    g = np.random.default_rng([1234, c, r, bits])
    mult = g.integers(2 ** 14, 2 ** 15, size=k).astype(np.int32)
    lo, hi = (-128, 127) if bits == 8 else (-8, 7)
    const = {"x": np.full((n, c, h, w), xe[0], dtype=np.int8), "w": np.full((k, c, r, r), we[0], dtype=np.int8),
             "mult": mult}
    ends = {"x": np.where(g.random((n, c, h, w)) < 0.5, xe[0], xe[1]).astype(np.int8),
            "w": np.where(g.random((k, c, r, r)) < 0.5, we[0], we[1]).astype(np.int8), "mult": mult}
    taps = _valid_tap_counts(h, w, r, r, stride, pad)
    want = (int(xe[0]) * int(we[0]) * c) * taps
    dev = torch.device("cuda:0")
    for label, t in (("constant", const), ("two ends", ends)):
        ref = ref_layer(L, t, requant=True, shift=SHIFT_EXTREME, relu=False, lo=lo, hi=hi)
        if label == "constant":
            assert np.array_equal(ref["acc"], np.broadcast_to(want[None, :, :, None], ref["acc"].shape))
        xp = q.pack(torch.from_numpy(t["x"]).to(dev), bits, xs)
        wp = q.pack(torch.from_numpy(t["w"]).to(dev), bits, True)
        m_dev = torch.from_numpy(mult).to(dev)
        for tid in _valid_tiles(L):
            announce(f"extreme {name} {label} tile {tid} raw")
            y = q.conv2d(L.desc(), xp, wp, tile=tid)
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["acc"], f"{name} {label} tile {tid} raw")
            announce(f"extreme {name} {label} tile {tid} requant")
            y = q.conv2d(L.desc(), xp, wp, tile=tid, requant=True, mult=m_dev, shift=SHIFT_EXTREME, relu=False,
                         clamp=(lo, hi))
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["y_packed"], f"{name} {label} tile {tid} requant")
            if q.tiles()[tid]["variant"] != 2 or q.max_splits(L.desc(), tid) < 2:
                continue
            splits = q.max_splits(L.desc(), tid)
            wprep = q.prepare_filters(L.desc(), wp, tid)
            ws = q.make_workspace(L.desc(), tid, splits, dev)
            announce(f"extreme {name} {label} tile {tid} splits {splits} raw")
            y = q.conv2d(L.desc(), xp, wprep, tile=tid, prepared=True, splits=splits, workspace=ws)
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["acc"], f"{name} {label} tile {tid} splits {splits} raw")


# ----------------------------------------------------------------- plans of shapes that differ in one axis

def test_shapes_differing_only_in_width_stride_or_padding():
    """Layers equal in every field but the horizontal stride or padding have
    different output widths, so a workgroup's band spans a different number of
    input rows; run one after another in one process (narrow bands first),
    each must get its own plan and equal the oracle on every wide tile."""
    torch, q = _torch(), _qconv()
    n, h, w, c, k = 2, 11, 24, 64, 64
    variants = [(1, 1), (2, 1), (3, 1), (1, 0), (1, 2)]   # (stride_w, pad_w); stride_h = pad_h = 1
    base = dict(n=n, h=h, w=w, c=c, k=k, r=3, s=3, stride_h=1, pad_h=1, bits=4, x_signed=0, w_signed=1)
    tiles = [t["id"] for t in q.tiles() if t["variant"] == 2 and
             all(q.tile_status(dict(base, stride_w=sw, pad_w=pw), t["id"]) == 0 for sw, pw in variants)]
    assert tiles
    g = np.random.default_rng(2024)
    x = g.integers(0, 16, size=(n, c, h, w)).astype(np.int8)
    f = g.integers(-7, 8, size=(k, c, 3, 3)).astype(np.int8)
    dev = torch.device("cuda:0")
    xp = q.pack(torch.from_numpy(x).to(dev), 4, False)
    wp = q.pack(torch.from_numpy(f).to(dev), 4, True)
    for sw, pw in variants:
        d = dict(base, stride_w=sw, pad_w=pw)
        ref = oracle.qconv_layer(x, f, bits=4, x_signed=False, w_signed=True, stride=(1, sw), pad=(1, pw),
                                 threads=oracle_threads())
        for tid in tiles:
            announce(f"stride_w {sw} pad_w {pw} tile {tid}")
            y = q.conv2d(d, xp, wp, tile=tid)
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["acc"], f"stride_w {sw} pad_w {pw} tile {tid}")


# ----------------------------------------------------------------- buffers, determinism, chaining

def test_every_output_written_and_nothing_past_the_end():
    torch, q = _torch(), _qconv()
    L = qi.Layer("canary", 3, 13, 11, 64, 40, 3, 3, 1, 1)
    t = qi.layer_tensors(300, 0, L)
    ref = ref_layer(L, t, requant=False)
    xp = q.pack(torch.from_numpy(t["x"]).cuda(), 4, False)
    wp = q.pack(torch.from_numpy(t["w"]).cuda(), 4, True)
    n_out = ref["acc"].size
    for sentinel in (0x5A5A5A5A, -1):
        buf = torch.full((n_out + 4096,), sentinel, dtype=torch.int32, device="cuda")
        announce(f"sentinel {sentinel:#x}")
        q.conv2d(L.desc(), xp, wp, out=buf[:n_out].view(ref["acc"].shape))
        torch.cuda.synchronize()
        host = buf.cpu().numpy()
        assert_same(host[:n_out].reshape(ref["acc"].shape), ref["acc"], "raw")
        assert (host[n_out:] == sentinel).all(), "write past the end of y"


def test_run_twice_identical():
    L = qi.workload1()[0]
    t = qi.layer_tensors(1, 0, L)
    announce("determinism")
    a = gpu_layer(L, t, requant=True)["y"]
    b = gpu_layer(L, t, requant=True)["y"]
    assert np.array_equal(a, b)


def test_chained_layers_need_no_relayout():
    """Layer 1's packed output is layer 2's input as-is (Sec. 3.3)."""
    L1 = qi.Layer("chain1", 2, 20, 20, 64, 128, 3, 3, 1, 1, w_range=(-7, 7))
    L2 = qi.Layer("chain2", 2, 20, 20, 128, 64, 3, 3, 2, 1, w_range=(-7, 7))
    t1 = qi.layer_tensors(400, 1, L1)
    t2 = qi.layer_tensors(400, 2, L2)
    s1 = stress_shift(L1, L1.x_range, L1.w_range)
    s2 = stress_shift(L2, L2.x_range, L2.w_range)
    r1 = ref_layer(L1, t1, requant=True, shift=s1)
    r2 = ref_layer(L2, t2, requant=True, shift=s2, packed_x=r1["y_packed"])
    announce("chain layer 1")
    g1 = gpu_layer(L1, t1, requant=True, shift=s1)
    assert_same(g1["y"], r1["y_packed"], "layer 1")
    announce("chain layer 2")
    g2 = gpu_layer(L2, t2, requant=True, shift=s2, x_packed_dev=g1["y_dev"])
    assert_same(g2["y"], r2["y_packed"], "layer 2")


def test_graph_replays_match_eager():
    """A captured chain replayed several times, with eager work and
    synchronisation between replays, reproduces the eager outputs every time."""
    torch, q = _torch(), _qconv()
    from paper_2202_06819_amd import nets
    L1 = qi.Layer("g1", 2, 14, 14, 64, 64, 3, 3, 1, 1, w_range=(-7, 7))
    L2 = qi.Layer("g2", 2, 14, 14, 64, 128, 1, 1, 2, 0, w_range=(-7, 7))
    t1, t2 = qi.layer_tensors(600, 1, L1), qi.layer_tensors(600, 2, L2)
    s1, s2 = stress_shift(L1, L1.x_range, L1.w_range), stress_shift(L2, L2.x_range, L2.w_range)
    xp = q.pack(torch.from_numpy(t1["x"]).cuda(), 4, False)
    specs = []
    for L, t, sh, src in ((L1, t1, s1, -1), (L2, t2, s2, 0)):
        wp = q.pack(torch.from_numpy(t["w"]).cuda(), 4, True)
        specs.append(nets.LayerSpec(L.desc(), wp, torch.from_numpy(t["mult"]).cuda(), sh, True, (0, 15), src=src))
    chain = nets.Chain(specs, xp)
    announce("graph: eager pass")
    eager = [o.clone() for o in chain.forward()]
    torch.cuda.synchronize()
    r1 = ref_layer(L1, t1, requant=True, shift=s1)
    assert_same(eager[0].cpu().numpy(), r1["y_packed"], "eager layer 1")
    chain.capture()
    for i in range(4):
        for o in chain.outputs:
            o.zero_()
        announce(f"graph: replay {i}")
        outs = chain.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs, eager):
            assert torch.equal(a, b), f"replay {i} differs from the eager pass"
        chain.forward()   # eager work between replays
        torch.cuda.synchronize()


# ----------------------------------------------------------------- split-K

SPLIT_SHAPES = [
    # name, n, h, c, k, r, stride, pad
    ("s7_512to512", 2, 7, 512, 512, 3, 1, 1),
    ("s14_256to256", 2, 14, 256, 256, 3, 1, 1),
    ("s14_256to512_s2", 2, 14, 256, 512, 3, 2, 1),
    ("s7_1x1_1024to256", 2, 7, 1024, 256, 1, 1, 0),
    ("s9_ragged_192to72", 3, 9, 192, 72, 3, 1, 1),
]


@pytest.mark.parametrize("shape", SPLIT_SHAPES, ids=lambda v: v[0])
def test_split_k_matches_oracle(shape):
    """Every wide tile and split factor; each configuration runs twice on one
    workspace (the arrival counters must return to zero between calls)."""
    torch, q = _torch(), _qconv()
    name, n, h, c, k, r, stride, pad = shape
    L = qi.Layer(name, n, h, h, c, k, r, r, stride, pad, w_range=(-7, 7))
    t = qi.layer_tensors(700, c + k, L)
    sh = stress_shift(L, L.x_range, L.w_range)
    ref = ref_layer(L, t, requant=True, shift=sh)
    ref_raw = ref_layer(L, t, requant=False)
    dev = torch.device("cuda:0")
    xp = q.pack(torch.from_numpy(t["x"]).to(dev), 4, False)
    wp = q.pack(torch.from_numpy(t["w"]).to(dev), 4, True)
    mult = torch.from_numpy(t["mult"]).to(dev)
    wide = [tt["id"] for tt in q.tiles() if tt["variant"] == 2 and q.tile_status(L.desc(), tt["id"]) == 0]
    assert wide
    for tid in wide:
        wprep = q.prepare_filters(L.desc(), wp, tid)
        chunks = q.max_splits(L.desc(), tid)
        for splits in sorted({2, 3, chunks} & set(range(2, chunks + 1))):
            ws = q.make_workspace(L.desc(), tid, splits, dev)
            for rep in range(2):
                announce(f"split-K {name} tile {tid} splits {splits} rep {rep}")
                y = q.conv2d(L.desc(), xp, wprep, tile=tid, prepared=True, splits=splits, workspace=ws,
                             requant=True, mult=mult, shift=sh)
                torch.cuda.synchronize()
                assert_same(y.cpu().numpy(), ref["y_packed"], f"{name} tile {tid} splits {splits} rep {rep}")
            announce(f"split-K {name} tile {tid} splits {splits} raw")
            y = q.conv2d(L.desc(), xp, wprep, tile=tid, prepared=True, splits=splits, workspace=ws)
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref_raw["acc"], f"{name} tile {tid} splits {splits} raw")
            info = q.layout(L.desc())
            tinfo = q.tiles()[tid]
            ntiles = -(-info["m"] // tinfo["tile_p"]) * -(-L.k // tinfo["tile_k"])
            part = -(-(ntiles * (-(-chunks // -(-chunks // splits))) * tinfo["tile_p"] * tinfo["tile_k"] * 4) // 256) * 256
            counters = ws[part:part + 4 * ntiles]
            assert int(counters.count_nonzero()) == 0, "arrival counters not reset"


# ----------------------------------------------------------------- bias and residual epilogue

BIAS_SHAPES = [
    # name, n, h, c, k, r, stride, pad, bits
    ("e_2x14_64to64_3x3", 2, 14, 64, 64, 3, 1, 1, 4),
    ("e_2x28_128to256_1x1_s2", 2, 28, 128, 256, 1, 2, 0, 4),
    ("e_2x7_512to512_3x3", 2, 7, 512, 512, 3, 1, 1, 4),
    ("e8_2x14_64to64_3x3", 2, 14, 64, 64, 3, 1, 1, 8),
]


@pytest.mark.parametrize("shape", BIAS_SHAPES, ids=lambda v: v[0])
def test_bias_and_residual_every_tile(shape):
    """Bias (fast and 64-bit paths), residual (unsigned and signed, in place),
    on every tile from packed and from prepared filters, and with split-K."""
    torch, q = _torch(), _qconv()
    name, n, h, c, k, r, stride, pad, bits = shape
    if bits == 4:
        L = qi.Layer(name, n, h, h, c, k, r, r, stride, pad, w_range=(-7, 7))
    else:
        L = qi.Layer(name, n, h, h, c, k, r, r, stride, pad, bits=8, x_signed=True, w_signed=True,
                     x_range=qi.S8, w_range=qi.S8, epilogue=qi.Epilogue(relu=False, lo=-128, hi=127))
    t = qi.layer_tensors(910, c + k + bits, L)
    g = np.random.default_rng([910, c, k, bits])
    sh = stress_shift(L, L.x_range, L.w_range)
    p = (h + 2 * pad - r) // stride + 1
    dev = torch.device("cuda:0")
    xp = q.pack(torch.from_numpy(t["x"]).to(dev), bits, L.x_signed)
    wp = q.pack(torch.from_numpy(t["w"]).to(dev), bits, L.w_signed)
    acc_mag = int(np.sqrt(c * r * r) * 8 * (8 if bits == 4 else 80))
    small_bias = g.integers(-acc_mag, acc_mag, size=k).astype(np.int32)
    # the largest bias the contract allows for this shape (accumulator + bias in int32)
    acc_shift = 4 * (int(L.x_signed) + int(L.w_signed)) if bits == 4 else 0
    bmax = (2 ** 31 - 1) // 2 ** acc_shift - _qconv().layout(L.desc())["max_abs_acc"]
    big_bias = g.integers(-bmax, bmax + 1, size=k).astype(np.int32)
    if bits == 4:
        ranges = [(True, 0, 15, False), (False, -8, 7, True)]   # relu, lo, hi, signed residual
    else:
        ranges = [(False, -128, 127, True), (True, -128, 127, True)]
    # multipliers too large for the one-instruction requantiser take the 64-bit form
    big_mult = g.integers(2 ** 29, 2 ** 30, size=k).astype(np.int32)
    cases = []
    for relu, lo, hi, rsig in ranges:
        rlo, rhi = (-(2 ** (bits - 1)), 2 ** (bits - 1) - 1) if rsig else (0, 2 ** bits - 1)
        res_vals = g.integers(rlo, rhi + 1, size=(n, p, p, k)).astype(np.int32)
        res_packed = oracle.pack_output(res_vals, bits, rsig)
        for bias, mlt, shift in ((small_bias, t["mult"], sh), (big_bias, t["mult"], sh), (None, t["mult"], sh),
                                 (small_bias, big_mult, sh + 15)):
            for use_res in (True, False):
                if bias is None and not use_res:
                    continue
                ref = oracle.qconv_layer(t["x"], t["w"], bits=bits, x_signed=L.x_signed, w_signed=L.w_signed,
                                         stride=(stride, stride), pad=(pad, pad), mult=mlt, shift=shift, relu=relu,
                                         lo=lo, hi=hi, bias=bias, residual=res_vals if use_res else None,
                                         threads=oracle_threads())
                cases.append((relu, lo, hi, rsig, bias, mlt, shift, res_packed if use_res else None, ref["y_packed"]))
    tiles = _valid_tiles(L)
    for tid in tiles:
        wide = q.tiles()[tid]["variant"] == 2
        wprep = q.prepare_filters(L.desc(), wp, tid) if wide else None
        for ci, (relu, lo, hi, rsig, bias, mlt, shift, res_packed, want) in enumerate(cases):
            b = None if bias is None else torch.from_numpy(bias).to(dev)
            res = None if res_packed is None else torch.from_numpy(np.ascontiguousarray(res_packed)).to(dev)
            kw = dict(requant=True, mult=torch.from_numpy(mlt).to(dev), shift=shift, relu=relu, clamp=(lo, hi),
                      bias=b, residual=res, residual_signed=rsig)
            announce(f"{name} tile {tid} case {ci} packed filters")
            y = q.conv2d(L.desc(), xp, wp, tile=tid, **kw)
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), want, f"{name} tile {tid} case {ci}")
            if wide:
                announce(f"{name} tile {tid} case {ci} prepared")
                y = q.conv2d(L.desc(), xp, wprep, tile=tid, prepared=True, **kw)
                torch.cuda.synchronize()
                assert_same(y.cpu().numpy(), want, f"{name} tile {tid} case {ci} prepared")
                if res is not None:
                    announce(f"{name} tile {tid} case {ci} in place")
                    yy = res.clone()
                    kw_in = dict(kw, residual=yy)
                    q.conv2d(L.desc(), xp, wprep, tile=tid, prepared=True, out=yy, **kw_in)
                    torch.cuda.synchronize()
                    assert_same(yy.cpu().numpy(), want, f"{name} tile {tid} case {ci} in place")
                chunks = q.max_splits(L.desc(), tid)
                if chunks > 1:
                    ws = q.make_workspace(L.desc(), tid, 2, dev)
                    announce(f"{name} tile {tid} case {ci} split 2")
                    y = q.conv2d(L.desc(), xp, wprep, tile=tid, prepared=True, splits=2, workspace=ws, **kw)
                    torch.cuda.synchronize()
                    assert_same(y.cpu().numpy(), want, f"{name} tile {tid} case {ci} split 2")


@pytest.mark.parametrize("branches", [False, True], ids=["one_stream", "two_streams"])
def test_residual_blocks_chain_eager_and_graph(branches):
    """Two basic residual blocks (conv-bias-ReLU, conv-bias-+shortcut-ReLU; the
    second block with a strided 1x1 projection shortcut), chained on the GPU
    with no relayout, eager and as replays of a captured graph, against the
    oracle layer by layer; with `branches` the projection runs on a second
    stream."""
    torch, q = _torch(), _qconv()
    from paper_2202_06819_amd import nets
    dev = torch.device("cuda:0")
    n, h = 2, 16
    # name, c, k, r, stride, pad, src, residual_src
    spec = [("b1c1", 64, 64, 3, 1, 1, -1, None), ("b1c2", 64, 64, 3, 1, 1, 0, -1),
            ("b2c1", 64, 128, 3, 2, 1, 1, None), ("b2ds", 64, 128, 1, 2, 0, 1, None),
            ("b2c2", 128, 128, 3, 1, 1, 2, 3)]
    g = np.random.default_rng(77)
    x = g.integers(0, 16, size=(n, 64, h, h)).astype(np.int8)
    layers, refs, specs = [], [], []
    xp_ref = oracle.relayout_pack(x, 4, False)
    outs_vals = []
    in_vals = oracle.unpack_tensor(xp_ref, 64, 4, False)
    for i, (name, c, k, r, stride, pad, src, rsrc) in enumerate(spec):
        hin = h if src < 0 else refs[src]["y"].shape[1]
        L = qi.Layer(name, n, hin, hin, c, k, r, r, stride, pad, w_range=(-7, 7))
        t = qi.layer_tensors(950, i, L)
        sh = stress_shift(L, L.x_range, L.w_range)
        bias = g.integers(-400, 400, size=k).astype(np.int32)
        packed_in = xp_ref if src < 0 else refs[src]["y_packed"]
        res = None if rsrc is None else (in_vals if rsrc < 0 else refs[rsrc]["y"])
        ref = oracle.qconv_layer(None, t["w"], bits=4, x_signed=False, w_signed=True, stride=(stride, stride),
                                 pad=(pad, pad), mult=t["mult"], shift=sh, relu=True, lo=0, hi=15, bias=bias,
                                 residual=res, packed_x=packed_in, threads=oracle_threads())
        refs.append(ref)
        wp = q.pack(torch.from_numpy(t["w"]).to(dev), 4, True)
        specs.append(nets.LayerSpec(L.desc(), wp, torch.from_numpy(t["mult"]).to(dev), sh, True, (0, 15), src=src,
                                    bias=torch.from_numpy(bias).to(dev), residual_src=rsrc))
    xp = q.pack(torch.from_numpy(x).to(dev), 4, False)
    chain = nets.Chain(specs, xp, branches=branches)
    assert chain.on_side == [False, False, False, branches, False]
    announce(f"residual chain eager, branches={branches}")
    outs = [o.clone() for o in chain.forward()]
    torch.cuda.synchronize()
    for (name, *_), o, ref in zip(spec, outs, refs):
        assert_same(o.cpu().numpy(), ref["y_packed"], f"eager {name}")
    chain.capture()
    for i in range(3):
        for o in chain.outputs:
            o.zero_()
        announce(f"residual chain replay {i}, branches={branches}")
        got = chain.replay()
        torch.cuda.synchronize()
        for (name, *_), o, ref in zip(spec, got, refs):
            assert_same(o.cpu().numpy(), ref["y_packed"], f"replay {i} {name}")
        chain.forward()
        torch.cuda.synchronize()


@pytest.mark.parametrize("shape", [
    ("a_2x56_64to64", 2, 56, 64, 64),
    ("a_2x28_128to128", 2, 28, 128, 128),
    ("a_8x7_512to512", 8, 7, 512, 512),
], ids=lambda v: v[0])
def test_ablation_instances_match_oracle(shape):
    """The kernels with any subset of duplicate-aware loading, register-level
    packing and widening at staging switched off (measurement instances)
    compute the same bytes."""
    torch, q = _torch(), _qconv()
    name, n, h, c, k = shape
    L = qi.Layer(name, n, h, h, c, k, 3, 3, 1, 1, w_range=(-7, 7))
    t = qi.layer_tensors(960, c, L)
    sh = stress_shift(L, L.x_range, L.w_range)
    ref = ref_layer(L, t, requant=True, shift=sh)
    ref_raw = ref_layer(L, t, requant=False)
    dev = torch.device("cuda:0")
    xp = q.pack(torch.from_numpy(t["x"]).to(dev), 4, False)
    wp = q.pack(torch.from_numpy(t["w"]).to(dev), 4, True)
    mult = torch.from_numpy(t["mult"]).to(dev)
    names = {tt["name"]: tt["id"] for tt in q.tiles()}
    ran = 0
    for tname in ("wide_b4_w4x1_f1x4_c64", "wide_b4_w8x1_f1x4_c64", "wide_b4_w4x1_f2x4_c64"):
        tid = names[tname]
        wprep = q.prepare_filters(L.desc(), wp, tid)
        for mask in range(1, 8):
            sch = {"tile_id": tid, "ablation": mask}
            if q.schedule_status(L.desc(), sch) != 0:
                continue
            ran += 1
            announce(f"{name} {tname} ablation {mask}")
            y = q.Conv2dCall(L.desc(), xp, wprep, schedule=sch, requant=True, mult=mult, shift=sh)()
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["y_packed"], f"{name} {tname} ablation {mask}")
            y = q.Conv2dCall(L.desc(), xp, wprep, schedule=sch)()
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref_raw["acc"], f"{name} {tname} ablation {mask} raw")
    assert ran >= 9


@pytest.mark.parametrize("fold", ["rows", "all"])
def test_stem_7x7_by_patch_unrolling(fold):
    """The 3-channel 7x7 stride-2 stem (8-bit): the input and the filters are
    patch-unrolled on the GPU (row pairs and columns into 64 channels, or
    every tap into 192) and the folded convolution runs on every tile that
    takes it; the result equals the oracle's direct 7x7 convolution of the
    original tensors."""
    torch, q = _torch(), _qconv()
    n, h, c, k = 2, 224, 3, 64
    L = qi.Layer("stem", n, h, h, c, k, 7, 7, 2, 3, bits=8, x_signed=True, w_signed=True, x_range=qi.S8,
                 w_range=qi.S8, epilogue=qi.Epilogue(relu=True, lo=-128, hi=127))
    t = qi.layer_tensors(990, 0, L)
    sh = stress_shift(L, L.x_range, L.w_range)
    ref = oracle.qconv_layer(t["x"], t["w"], bits=8, x_signed=True, w_signed=True, stride=(2, 2), pad=(3, 3),
                             mult=t["mult"], shift=sh, relu=True, lo=-128, hi=127, threads=oracle_threads())
    dev = torch.device("cuda:0")
    c_out = 64 if fold == "rows" else 192
    plan = q.few_channel_plan(L.desc(), c_out, fold)
    announce(f"stem unroll, fold {fold}")
    xu = q.unroll(torch.from_numpy(t["x"]).to(dev), c_out, **plan["x"])
    wu = q.unroll(torch.from_numpy(t["w"]).to(dev), c_out, **plan["w"])
    torch.cuda.synchronize()
    # the unrolled layouts against their definition, written out on the host
    assert np.array_equal(xu.cpu().numpy(), unroll_def(t["x"], c_out, **plan["x"]))
    assert np.array_equal(wu.cpu().numpy(), unroll_def(t["w"], c_out, **plan["w"]))
    d = plan["desc"]
    mult = torch.from_numpy(t["mult"]).to(dev)
    ran = 0
    for tt in q.tiles():
        if q.tile_status(d, tt["id"]) != 0:
            continue
        ran += 1
        announce(f"stem folded conv ({fold}) tile {tt['name']}")
        y = q.conv2d(d, xu, wu, tile=tt["id"], requant=True, mult=mult, shift=sh, relu=True, clamp=(-128, 127))
        torch.cuda.synchronize()
        assert_same(y.cpu().numpy(), ref["y_packed"], f"stem {fold} {tt['name']}")
        if tt["variant"] == 2:
            wprep = q.prepare_filters(d, wu, tt["id"])
            y = q.conv2d(d, xu, wprep, tile=tt["id"], prepared=True)
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["acc"], f"stem {fold} {tt['name']} prepared raw")
    assert ran >= 2


# ------------------------------------------------- batch-interleaved layout

def interleave(a: np.ndarray, nb: int) -> np.ndarray:
    """N x H x W x ... -> N/nb x H x W x nb x ... : the batch-interleaved
    layout's definition (image i's pixel (y, x) at [i // nb, y, x, i % nb])."""
    n = a.shape[0]
    b = a.reshape(n // nb, nb, *a.shape[1:])
    return np.ascontiguousarray(b.transpose(0, 2, 3, 1, *range(4, b.ndim)))


INTERLEAVED_CASES = [
    # name, n, h, w, c, k, r, (stride_h, stride_w), pad, bits, nb
    ("i4_3x3_ragged_nb2", 4, 13, 11, 64, 64, 3, (1, 1), 1, 4, 2),
    ("i4_3x3_nb4", 8, 14, 14, 128, 64, 3, (1, 1), 1, 4, 4),
    ("i4_1x1_nb4", 4, 9, 7, 64, 128, 1, (1, 1), 0, 4, 4),
    ("i4_5x5_nb2", 2, 12, 12, 64, 64, 5, (1, 1), 2, 4, 2),
    ("i4_3x3_rows_s2_nb2", 4, 15, 9, 64, 64, 3, (2, 1), 1, 4, 2),
    ("i8_3x3_nb2", 4, 10, 10, 64, 64, 3, (1, 1), 1, 8, 2),
    ("i4_7x7_512_nb16", 16, 7, 7, 256, 256, 3, (1, 1), 1, 4, 16),
]


@pytest.mark.parametrize("case", INTERLEAVED_CASES, ids=[c[0] for c in INTERLEAVED_CASES])
def test_interleaved_layout(case):
    """Pack into the batch-interleaved layout and convolve in it (input,
    output and residual interleaved) on every tile that reads it, from packed
    and prepared filters, raw and requantised, with a bias and a residual, and
    split over channel chunks where there are several; every result equals
    the oracle's plain-layout result put in the interleaved order."""
    ran = _check_interleaved(case)
    assert ran >= 2, f"{case[0]}: only {ran} tiles read the interleaved layout"


def _random_interleaved_case(seed: int):
    g = np.random.default_rng([7171, seed])
    bits = 8 if seed % 3 == 2 else 4
    nb = int(g.choice([2, 4, 8, 16]))
    n = nb * int(g.integers(1, 4))
    r = int(g.choice([1, 3, 3, 5]))
    pad = int(g.integers(0, r // 2 + 2))
    h, w = int(g.integers(max(1, r - 2 * pad), 30)), int(g.integers(max(1, r - 2 * pad), 30))
    strides = (int(g.choice([1, 1, 2])), int(g.choice([1, 1, 2])))
    c, k = (32 if bits == 4 else 16) * int(g.integers(1, 9)), 8 * int(g.integers(1, 33))
    return (f"ir{seed}", n, h, w, c, k, r, strides, pad, bits, nb)


@pytest.mark.parametrize("first", [0, 40])
def test_interleaved_layout_random_shapes(first):
    """The same checks on random shapes (interleave factors 2-16, 1x1 to 5x5,
    strides 1-2 per axis, ragged sizes); shapes no tile reads are skipped."""
    q = _qconv()
    ran = 0
    for seed in range(first, first + 40):
        case = _random_interleaved_case(seed)
        _, n, h, w, c, k, r, (sh_, sw_), pad, bits, nb = case
        d = dict(n=n, h=h, w=w, c=c, k=k, r=r, s=r, stride_h=sh_, stride_w=sw_, pad_h=pad, pad_w=pad, bits=bits,
                 x_signed=int(bits == 8), w_signed=1, nb=nb)
        if any(q.tile_status(d, t["id"]) == 0 for t in q.tiles()):
            ran += _check_interleaved(case)
    assert ran > 0


def _check_interleaved(case) -> int:
    """Run one interleaved-layout case on every tile that reads it; returns
    the number of tiles run."""
    torch, q = _torch(), _qconv()
    name, n, h, w, c, k, r, (sh_, sw_), pad, bits, nb = case
    signed8 = bits == 8
    g = np.random.default_rng([977, n, h, w, c, k, r, sh_, bits, nb])
    xr = qi.S8 if signed8 else (0, 15)
    wr = qi.S8 if signed8 else (-7, 7)
    x = g.integers(xr[0], xr[1] + 1, size=(n, c, h, w)).astype(np.int8)
    f = g.integers(wr[0], wr[1] + 1, size=(k, c, r, r)).astype(np.int8)
    mult = g.integers(2 ** 14, 2 ** 15, size=k).astype(np.int32)
    d = dict(n=n, h=h, w=w, c=c, k=k, r=r, s=r, stride_h=sh_, stride_w=sw_, pad_h=pad, pad_w=pad, bits=bits,
             x_signed=int(signed8), w_signed=1, nb=nb)
    L = qi.Layer(name, n, h, w, c, k, r, r, 1, pad, bits=bits, x_signed=signed8, w_signed=True, x_range=xr,
                 w_range=wr)
    sh = stress_shift(L, xr, wr)
    lo, hi, relu = (-128, 127, False) if signed8 else (0, 15, True)
    p, qq = (h + 2 * pad - r) // sh_ + 1, (w + 2 * pad - r) // sw_ + 1
    bias = g.integers(-4000, 4000, size=k).astype(np.int32)
    rlo, rhi = (-128, 127) if signed8 else (0, 15)
    res_vals = g.integers(rlo, rhi + 1, size=(n, p, qq, k)).astype(np.int32)
    res_packed = oracle.pack_output(res_vals, bits, signed8)
    kw = dict(bits=bits, x_signed=signed8, w_signed=True, stride=(sh_, sw_), pad=(pad, pad), mult=mult, shift=sh,
              relu=relu, lo=lo, hi=hi, threads=oracle_threads())
    ref = oracle.qconv_layer(x, f, **kw)
    ref_ext = oracle.qconv_layer(x, f, bias=bias, residual=res_vals, **kw)
    dev = torch.device("cuda:0")
    announce(f"{name}: interleaved pack")
    xp = q.pack(torch.from_numpy(x).to(dev), bits, signed8, nb=nb)
    torch.cuda.synchronize()
    assert_same(xp.cpu().numpy(), interleave(ref["x_packed"], nb), f"{name} pack")
    wp = q.pack(torch.from_numpy(f).to(dev), bits, True)
    m_dev = torch.from_numpy(mult).to(dev)
    b_dev = torch.from_numpy(bias).to(dev)
    res_dev = torch.from_numpy(interleave(res_packed, nb)).to(dev)
    want_y, want_acc, want_ext = (interleave(ref["y_packed"], nb), interleave(ref["acc"], nb),
                                  interleave(ref_ext["y_packed"], nb))
    rq = dict(requant=True, mult=m_dev, shift=sh, relu=relu, clamp=(lo, hi))
    ran = 0
    for t in q.tiles():
        if q.tile_status(d, t["id"]) != 0:
            continue
        ran += 1
        tid = t["id"]
        announce(f"{name} tile {t['name']} packed filters")
        y = q.conv2d(d, xp, wp, tile=tid, **rq)
        torch.cuda.synchronize()
        assert_same(y.cpu().numpy(), want_y, f"{name} {t['name']}")
        wprep = q.prepare_filters(d, wp, tid)
        announce(f"{name} tile {t['name']} prepared, raw")
        y = q.conv2d(d, xp, wprep, tile=tid, prepared=True)
        torch.cuda.synchronize()
        assert_same(y.cpu().numpy(), want_acc, f"{name} {t['name']} raw")
        announce(f"{name} tile {t['name']} prepared, bias and residual")
        y = q.conv2d(d, xp, wprep, tile=tid, prepared=True, bias=b_dev, residual=res_dev, residual_signed=signed8,
                     **rq)
        torch.cuda.synchronize()
        assert_same(y.cpu().numpy(), want_ext, f"{name} {t['name']} bias+residual")
        if q.max_splits(d, tid) > 1:
            announce(f"{name} tile {t['name']} split 2")
            y = q.conv2d(d, xp, wprep, tile=tid, prepared=True, splits=2,
                         workspace=q.make_workspace(d, tid, 2, dev), **rq)
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), want_y, f"{name} {t['name']} split 2")
    return ran


# ------------------------------------------------ the pack fused into the conv

FUSED_CASES = [
    # name, n, h, w, c, k, stride, bits, value range of x
    ("b4_56x56_64_n8", 8, 56, 56, 64, 64, 1, 4, (0, 15)),
    ("b4_out_of_range", 2, 20, 24, 64, 64, 1, 4, (-128, 127)),   # saturation of every kind
    ("b4_ragged_w14_c128", 4, 14, 14, 128, 64, 1, 4, (0, 15)),   # byte loads, two channel chunks
    ("b4_odd_13x11", 3, 13, 11, 64, 128, 1, 4, (-3, 20)),
    ("b4_stride2", 4, 28, 28, 64, 128, 2, 4, (0, 15)),
    ("b4_persistent_n32", 32, 56, 56, 64, 64, 1, 4, (0, 15)),    # several tiles per workgroup
    ("b8_28x28_64", 4, 28, 28, 64, 64, 1, 8, (-128, 127)),
    ("b8_24x32_64_octets", 3, 24, 32, 64, 64, 1, 8, (-128, 127)),   # 8-pixel loads, 8-bit
    ("b4_octets_c128_16x16", 2, 16, 16, 128, 64, 1, 4, (-20, 30)),   # 8-pixel loads over two chunks, saturation
    ("b8_octets_stride2_32x32", 2, 32, 32, 64, 64, 2, 8, (-128, 127)),   # 8-pixel loads, strided band rows
]


@pytest.mark.parametrize("case", FUSED_CASES, ids=[c[0] for c in FUSED_CASES])
def test_fused_pack_conv(case):
    """qconv2d_packing on every tile that has the fused instance: y (requant
    and raw) equals the oracle's layer on the same int8 NCHW input (which the
    oracle packs with saturation), and the packed copy equals the oracle's
    packed input."""
    torch, q = _torch(), _qconv()
    name, n, h, w, c, k, stride, bits, xr = case
    signed = bits == 8
    g = np.random.default_rng([991, n, h, w, c, k, stride, bits])
    x = g.integers(xr[0], xr[1] + 1, size=(n, c, h, w)).astype(np.int8)
    wr = (-128, 127) if signed else (-7, 7)
    f = g.integers(wr[0], wr[1] + 1, size=(k, c, 3, 3)).astype(np.int8)
    mult = g.integers(2 ** 14, 2 ** 15, size=k).astype(np.int32)
    L = qi.Layer(name, n, h, w, c, k, 3, 3, stride, 1, bits=bits, x_signed=signed, w_signed=True,
                 x_range=(0, 15) if not signed else qi.S8, w_range=wr)
    sh = stress_shift(L, L.x_range, L.w_range)
    lo, hi, relu = (-128, 127, False) if signed else (0, 15, True)
    ref = oracle.qconv_layer(x, f, bits=bits, x_signed=signed, w_signed=True, stride=(stride, stride), pad=(1, 1),
                             mult=mult, shift=sh, relu=relu, lo=lo, hi=hi, threads=oracle_threads())
    d = L.desc()
    dev = torch.device("cuda:0")
    x_dev = torch.from_numpy(x).to(dev)
    wp = q.pack(torch.from_numpy(f).to(dev), bits, True)
    m_dev = torch.from_numpy(mult).to(dev)
    ran = 0
    for t in q.tiles():
        if t["variant"] != 2 or q.tile_status(d, t["id"]) != 0:
            continue
        ran += 1
        tid = t["id"]
        wprep = q.prepare_filters(d, wp, tid)
        announce(f"fused pack {name} tile {t['name']}")
        call = q.PackingConv2dCall(d, x_dev, wprep, tile=tid, mult=m_dev, shift=sh, relu=relu, clamp=(lo, hi),
                                   x_packed=True)
        y = call()
        torch.cuda.synchronize()
        assert_same(y.cpu().numpy(), ref["y_packed"], f"{name} {t['name']} y")
        assert_same(call.x_packed.cpu().numpy(), ref["x_packed"], f"{name} {t['name']} packed copy")
        announce(f"fused pack {name} tile {t['name']} raw, no packed copy")
        y = q.PackingConv2dCall(d, x_dev, wprep, tile=tid, requant=False)()
        torch.cuda.synchronize()
        assert_same(y.cpu().numpy(), ref["acc"], f"{name} {t['name']} raw")
    assert ran >= 4


@pytest.mark.parametrize("shape", [
    # name, n, h, c, k, stride, bits -- strided 3x3 layers whose bands take
    # several staging rounds, and multi-chunk ones with a single band buffer
    ("b8_s2_28to14_128to256", 4, 28, 128, 256, 2, 8),
    ("b8_s2_14to7_256to512", 4, 14, 256, 512, 2, 8),
    ("b8_s2_56to28_64to128", 2, 56, 64, 128, 2, 8),
    ("b4_s2_28to14_128to256", 4, 28, 128, 256, 2, 4),
    ("b8_s3_30to10_64to64", 2, 30, 64, 64, 3, 8),
], ids=lambda v: v[0])
def test_strided_bands_every_wide_tile(shape):
    q = _qconv()
    name, n, h, c, k, stride, bits = shape
    if bits == 8:
        L = qi.Layer(name, n, h, h, c, k, 3, 3, stride, 1, bits=8, x_signed=True, w_signed=True, x_range=qi.S8,
                     w_range=qi.S8, epilogue=qi.Epilogue(relu=False, lo=-128, hi=127))
    else:
        L = qi.Layer(name, n, h, h, c, k, 3, 3, stride, 1, w_range=(-7, 7))
    t = qi.layer_tensors(800, c + k + stride, L)
    sh = stress_shift(L, L.x_range, L.w_range)
    ref = ref_layer(L, t, requant=True, shift=sh)
    ref_raw = ref_layer(L, t, requant=False)
    wide = [tt["id"] for tt in q.tiles() if tt["variant"] == 2 and q.tile_status(L.desc(), tt["id"]) == 0]
    assert len(wide) >= 2
    for tid in wide:
        announce(f"{name} tile {tid} prepared requant shift={sh}")
        assert_same(gpu_layer(L, t, requant=True, tile=tid, shift=sh, prepared=True)["y"], ref["y_packed"],
                    f"{name} tile {tid} prepared")
        announce(f"{name} tile {tid} prepared raw")
        assert_same(gpu_layer(L, t, requant=False, tile=tid, prepared=True)["y"], ref_raw["acc"],
                    f"{name} tile {tid} prepared raw")


# ------------------------------------------------------------ persistent grids

PIPE_CASES = [
    # name, n, h, bits, relu, lo, hi  (n*h*h is not a multiple of any tile's pixels: a ragged last tile)
    ("u4_relu_n33_55", 33, 55, 4, True, 0, 15),
    ("s4_n33_55", 33, 55, 4, False, -8, 7),
    ("s8_n33_55", 33, 55, 8, False, -128, 127),
]


@pytest.mark.parametrize("case", PIPE_CASES, ids=lambda c: c[0])
def test_persistent_3x3_requant_every_tile(case):
    """Persistent grids of single-chunk 3x3 layers with the requantising
    epilogue: sized for one workgroup per CU, every workgroup walks several
    tiles through both band buffers.  Every wide tile's output, and the
    generic instance's, equals the oracle's at every pixel (the ragged tail
    included); unsigned 4-bit, signed 4-bit and signed 8-bit outputs."""
    torch, q = _torch(), _qconv()
    name, n, h, bits, relu, lo, hi = case
    signed = bits == 8
    L = qi.Layer(name, n, h, h, 64, 64, 3, 3, 1, 1, bits=bits, x_signed=signed, w_signed=True,
                 x_range=qi.S8 if signed else qi.U4, w_range=qi.S8 if signed else qi.S4)
    t = qi.layer_tensors(970, bits, L)
    sh = stress_shift(L, L.x_range, L.w_range)
    d = L.desc()
    dev = torch.device("cuda:0")
    xp = q.pack(torch.from_numpy(t["x"]).to(dev), bits, signed)
    wp = q.pack(torch.from_numpy(t["w"]).to(dev), bits, True)
    kw = dict(requant=True, mult=torch.from_numpy(t["mult"]).to(dev), shift=sh, relu=relu, clamp=(lo, hi))
    announce(f"{name}: generic instance")
    ref = q.conv2d(d, xp, wp, **kw)
    torch.cuda.synchronize()
    ref_np = ref.cpu().numpy()
    m = n * h * h
    want = oracle.qconv_layer(t["x"], t["w"], bits=bits, x_signed=signed, w_signed=True, stride=(1, 1), pad=(1, 1),
                              mult=t["mult"], shift=sh, relu=relu, lo=lo, hi=hi, threads=oracle_threads())["y_packed"]
    assert_same(ref_np, want, f"{name}: generic instance vs the oracle")
    ran = 0
    for tt in q.tiles():
        if not tt["name"].startswith("wide") or q.tile_status(d, tt["id"]) != 0 or 64 % tt["tile_k"]:
            continue
        tiles = -(-m // tt["tile_p"]) * (64 // tt["tile_k"])
        assert tiles > 256, "the grid of one workgroup per CU must be persistent"
        wprep = q.prepare_filters(d, wp, tt["id"])
        announce(f"{name}: tile {tt['name']}, one workgroup per CU, {tiles} tiles")
        y = q.Conv2dCall(d, xp, wprep, tile=tt["id"], prepared=True,
                         schedule={"tile_id": tt["id"], "wg_per_cu": 1}, **kw)()
        torch.cuda.synchronize()
        y_np = y.cpu().numpy()
        assert_same(y_np, want, f"{name} tile {tt['name']} vs the oracle")
        ran += 1
    assert ran >= 3


@pytest.mark.parametrize("shape", [
    # name, n, h, c, k, r, splits, wg_per_cu -- deep layers with several channel tiles
    ("x_4x14_256to256_3x3_split2", 4, 14, 256, 256, 3, 2, 0),
    ("x_2x7_512to512_3x3_persistent", 2, 7, 512, 512, 3, 1, 1),
    ("x_3x7_512to384_1x1", 3, 7, 512, 384, 1, 1, 0),
], ids=lambda v: v[0])
def test_xcd_orders_match_oracle(shape):
    """Every workgroup order (hardware, pixel tiles outermost, channel tiles
    outermost, the library's choice) computes the same bytes, with split-K and
    with persistent grids."""
    torch, q = _torch(), _qconv()
    name, n, h, c, k, r, splits, wg = shape
    L = qi.Layer(name, n, h, h, c, k, r, r, 1, r // 2, w_range=(-7, 7))
    t = qi.layer_tensors(980, c + k + r, L)
    sh = stress_shift(L, L.x_range, L.w_range)
    ref = ref_layer(L, t, requant=True, shift=sh)
    dev = torch.device("cuda:0")
    xp = q.pack(torch.from_numpy(t["x"]).to(dev), 4, False)
    wp = q.pack(torch.from_numpy(t["w"]).to(dev), 4, True)
    mult = torch.from_numpy(t["mult"]).to(dev)
    ran = 0
    for tt in q.tiles():
        if tt["variant"] != 2 or q.tile_status(L.desc(), tt["id"]) != 0 or -(-k // tt["tile_k"]) < 2:
            continue
        if splits > q.max_splits(L.desc(), tt["id"]):
            continue
        wprep = q.prepare_filters(L.desc(), wp, tt["id"])
        ws = q.make_workspace(L.desc(), tt["id"], splits, dev)
        for xo in (-1, 0, 1, 2):
            sch = {"tile_id": tt["id"], "splits": splits, "wg_per_cu": wg, "xcd_order": xo}
            announce(f"{name} tile {tt['name']} xcd_order {xo}")
            y = q.Conv2dCall(L.desc(), xp, wprep, schedule=sch, workspace=ws, requant=True, mult=mult, shift=sh)()
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["y_packed"], f"{name} {tt['name']} xcd_order {xo}")
        ran += 1
        if ran == 4:
            break
    assert ran >= 2
