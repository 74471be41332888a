"""GPU parity over many random shapes: every tile that runs a shape, from packed
and from prepared filters, with a random split-K factor on the wide tiles and,
for 3x3 shapes, the pack fused into the convolution.  Shapes mix ragged pixel
counts and channel counts, strides 1-3, paddings beyond the filter's half
width, filters from 1x1 to 7x7 (non-square ones too), signed and unsigned
operands and both output signednesses; half of them are large enough that
workgroups walk several output tiles and bands take several staging rounds.
A second set adds a bias and a residual to the requantiser, also through the
no-alloc entry; a third chains random residual networks; a fourth runs
few-channel layers by patch unrolling; a fifth varies stride and padding per
axis, also for the fused pack.
"""
import numpy as np
import pytest

import oracle
import qconv_inputs as qi
from _util import announce, assert_same, gpu_layer, oracle_threads, random_layer, ref_layer, stress_shift

pytestmark = pytest.mark.gpu

BLOCK = 25
BLOCKS = [(b * BLOCK, False) for b in range(4)] + [(1000 + b * BLOCK, True) for b in range(4)]


def _fused(q, torch, L, t, sh, g, dev):
    """The pack fused in: int8 NCHW input over the whole int8 range (the oracle
    packs it with saturation); the packed copy too where the bands cover every
    input row (the library refuses the copy otherwise)."""
    d, e = L.desc(), L.epilogue
    tiles = [tt for tt in q.tiles() if tt["variant"] == 2 and q.tile_status(d, tt["id"]) == 0]
    if not tiles:
        return
    x8 = g.integers(-128, 128, size=(L.n, L.c, L.h, L.w)).astype(np.int8)
    ref = oracle.qconv_layer(x8, t["w"], bits=L.bits, x_signed=L.x_signed, w_signed=L.w_signed,
                             stride=(L.stride, L.stride), pad=(L.pad, L.pad), mult=t["mult"], shift=sh, relu=e.relu,
                             lo=e.lo, hi=e.hi, threads=oracle_threads())
    x_dev = torch.from_numpy(x8).to(dev)
    wp = q.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
    mult = torch.from_numpy(t["mult"]).to(dev)
    for tt in tiles:
        wprep = q.prepare_filters(d, wp, tt["id"])
        announce(f"{L.name} fused tile {tt['name']}")
        call = q.PackingConv2dCall(d, x_dev, wprep, tile=tt["id"], mult=mult, shift=sh, relu=e.relu,
                                   clamp=(e.lo, e.hi), x_packed=True)
        try:
            y = call()
            copy = True
        except q.QConvError as ex:
            assert "no packed copy" in str(ex), str(ex)
            y = q.PackingConv2dCall(d, x_dev, wprep, tile=tt["id"], mult=mult, shift=sh, relu=e.relu,
                                    clamp=(e.lo, e.hi))()
            copy = False
        torch.cuda.synchronize()
        assert_same(y.cpu().numpy(), ref["y_packed"], f"{L.name} fused {tt['name']}")
        if copy:
            assert_same(call.x_packed.cpu().numpy(), ref["x_packed"], f"{L.name} fused {tt['name']} packed copy")


@pytest.mark.parametrize("block", BLOCKS, ids=lambda b: f"{'large' if b[1] else 'small'}_{b[0]}")
def test_random_shapes_every_tile(block):
    import torch
    from paper_2202_06819_amd import qconv as q

    first, big = block
    dev = torch.device("cuda:0")
    tiles_all = q.tiles()
    ran = 0
    for seed in range(first, first + BLOCK):
        L = random_layer(seed, big)
        if L.h + 2 * L.pad < L.r or L.w + 2 * L.pad < L.s:
            continue
        tiles = [tt["id"] for tt in tiles_all if q.tile_status(L.desc(), tt["id"]) == 0]
        assert tiles, f"no tile runs {L.desc()}"
        t = qi.layer_tensors(4242, seed, L)
        sh = stress_shift(L, L.x_range, L.w_range)
        ref = ref_layer(L, t, requant=True, shift=sh)
        g = np.random.default_rng([77, seed])
        e = L.epilogue
        for tid in tiles:
            announce(f"{L.name} {L.desc()} tile {tid}")
            assert_same(gpu_layer(L, t, requant=False, tile=tid)["y"], ref["acc"], f"{L.name} tile {tid} raw")
            assert_same(gpu_layer(L, t, requant=True, tile=tid, shift=sh)["y"], ref["y_packed"],
                        f"{L.name} tile {tid} requant")
            ran += 1
            if tiles_all[tid]["variant"] != 2:
                continue
            got = gpu_layer(L, t, requant=True, tile=tid, shift=sh, prepared=True)
            assert_same(got["y"], ref["y_packed"], f"{L.name} tile {tid} prepared")
            most = q.max_splits(L.desc(), tid)
            if most < 2:
                continue
            splits = int(g.integers(2, most + 1))
            wp = q.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
            wprep = q.prepare_filters(L.desc(), wp, tid)
            xp = q.pack(torch.from_numpy(t["x"]).to(dev), L.bits, L.x_signed)
            ws = q.make_workspace(L.desc(), tid, splits, dev)
            for rep in range(2):
                announce(f"{L.name} tile {tid} splits {splits} rep {rep}")
                y = q.conv2d(L.desc(), xp, wprep, tile=tid, prepared=True, splits=splits, workspace=ws, requant=True,
                             mult=torch.from_numpy(t["mult"]).to(dev), shift=sh, relu=e.relu, clamp=(e.lo, e.hi))
                torch.cuda.synchronize()
                assert_same(y.cpu().numpy(), ref["y_packed"], f"{L.name} tile {tid} splits {splits} rep {rep}")
        if L.r == 3 and L.s == 3:
            _fused(q, torch, L, t, sh, g, dev)
    assert ran > 0


@pytest.mark.parametrize("block", [(2000, False), (2025, False), (3000, True), (3025, True)],
                         ids=lambda b: f"{'large' if b[1] else 'small'}_{b[0]}")
def test_random_shapes_bias_residual(block):
    """The requantiser with a per-channel bias and a packed residual (of the
    output's signedness) on random shapes: every tile from packed filters; on
    the wide tiles also prepared, in place (y over the residual), with a random
    split through a caller workspace and through the no-alloc entry."""
    import torch
    from paper_2202_06819_amd import qconv as q

    first, big = block
    dev = torch.device("cuda:0")
    tiles_all = q.tiles()
    scratch = q.noalloc_limits()["scratch_bytes"]
    ran = 0
    for seed in range(first, first + BLOCK):
        L = random_layer(seed, big)
        if L.h + 2 * L.pad < L.r or L.w + 2 * L.pad < L.s:
            continue
        d, e = L.desc(), L.epilogue
        t = qi.layer_tensors(6161, seed, L)
        g = np.random.default_rng([6161, seed])
        sh = stress_shift(L, L.x_range, L.w_range)
        acc_mag = int(np.sqrt(L.c * L.r * L.s) * 8 * (8 if L.bits == 4 else 80))
        bias = g.integers(-acc_mag, acc_mag + 1, size=L.k).astype(np.int32)
        rsig = e.lo < 0
        rlo, rhi = (-(2 ** (L.bits - 1)), 2 ** (L.bits - 1) - 1) if rsig else (0, 2 ** L.bits - 1)
        res_vals = g.integers(rlo, rhi + 1, size=(L.n, L.p, L.q, L.k)).astype(np.int32)
        want = oracle.qconv_layer(t["x"], t["w"], bits=L.bits, x_signed=L.x_signed, w_signed=L.w_signed,
                                  stride=(L.stride, L.stride), pad=(L.pad, L.pad), mult=t["mult"], shift=sh,
                                  relu=e.relu, lo=e.lo, hi=e.hi, bias=bias, residual=res_vals,
                                  threads=oracle_threads())["y_packed"]
        xp = q.pack(torch.from_numpy(t["x"]).to(dev), L.bits, L.x_signed)
        wp = q.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
        res = torch.from_numpy(np.ascontiguousarray(oracle.pack_output(res_vals, L.bits, rsig))).to(dev)
        kw = dict(requant=True, mult=torch.from_numpy(t["mult"]).to(dev), shift=sh, relu=e.relu,
                  clamp=(e.lo, e.hi), bias=torch.from_numpy(bias).to(dev), residual=res, residual_signed=rsig)
        for tid in [tt["id"] for tt in tiles_all if q.tile_status(d, tt["id"]) == 0]:
            announce(f"{L.name} {d} tile {tid} bias+residual")
            y = q.conv2d(d, xp, wp, tile=tid, **kw)
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), want, f"{L.name} tile {tid}")
            ran += 1
            if tiles_all[tid]["variant"] != 2:
                continue
            wprep = q.prepare_filters(d, wp, tid)
            y = q.conv2d(d, xp, wprep, tile=tid, prepared=True, **kw)
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), want, f"{L.name} tile {tid} prepared")
            yy = res.clone()
            q.conv2d(d, xp, wprep, tile=tid, prepared=True, out=yy, **dict(kw, residual=yy))
            torch.cuda.synchronize()
            assert_same(yy.cpu().numpy(), want, f"{L.name} tile {tid} in place")
            most = q.max_splits(d, tid)
            if most < 2:
                continue
            splits = int(g.integers(2, most + 1))
            ws = q.make_workspace(d, tid, splits, dev)
            announce(f"{L.name} tile {tid} bias+residual splits {splits}")
            y = q.conv2d(d, xp, wprep, tile=tid, prepared=True, splits=splits, workspace=ws, **kw)
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), want, f"{L.name} tile {tid} splits {splits}")
            if q.workspace_bytes(d, tid, splits) <= scratch:
                announce(f"{L.name} tile {tid} bias+residual splits {splits} no-alloc")
                y = q.conv2d(d, xp, wprep, tile=tid, prepared=True, splits=splits, noalloc=True, **kw)
                torch.cuda.synchronize()
                assert_same(y.cpu().numpy(), want, f"{L.name} tile {tid} splits {splits} no-alloc")
    assert ran > 0


def _residual_net(seed: int):
    """A random residual network: 1-3 blocks of (3x3 with bias, 3x3 with bias
    plus the shortcut), the shortcut a 1x1 projection where the stride or the
    channel count changes; 4-bit or 8-bit, ReLU on or off per layer."""
    g = np.random.default_rng([8181, seed])
    bits = 8 if seed % 3 == 2 else 4
    n, h, c0 = int(g.integers(1, 9)), int(g.integers(6, 40)), 32 * int(g.integers(1, 5))
    spec, cur, ch = [], -1, c0    # (name, c, k, r, stride, pad, src, residual_src)
    for b in range(int(g.integers(1, 4))):
        stride = int(g.choice([1, 2]))
        k = ch * (2 if stride == 2 else 1) if g.random() < 0.7 else 32 * int(g.integers(1, 9))
        base = len(spec)
        spec.append((f"b{b}c1", ch, k, 3, stride, 1, cur, None))
        short = cur
        if stride != 1 or k != ch:
            spec.append((f"b{b}ds", ch, k, 1, stride, 0, cur, None))
            short = base + 1
        spec.append((f"b{b}c2", k, k, 3, 1, 1, base, short))
        cur, ch = len(spec) - 1, k
    return g, bits, n, h, c0, spec


@pytest.mark.parametrize("first", [0, 10])
def test_random_residual_chains(first):
    """Random residual networks chained with no relayout (projections fused
    into their strided 3x3, or on a second stream): eager and three graph
    replays, each against the oracle layer by layer."""
    import torch
    from paper_2202_06819_amd import nets
    from paper_2202_06819_amd import qconv as q

    dev = torch.device("cuda:0")
    for seed in range(first, first + 10):
        g, bits, n, h, c0, spec = _residual_net(seed)
        xs = bits == 8
        lo, hi = (-128, 127) if xs else (0, 15)
        x = g.integers(-128 if xs else 0, 128 if xs else 16, size=(n, c0, h, h)).astype(np.int8)
        xp_ref = oracle.relayout_pack(x, bits, xs)
        in_vals = oracle.unpack_tensor(xp_ref, c0, bits, xs)
        refs, specs = [], []
        for i, (name, c, k, r, stride, pad, src, rsrc) in enumerate(spec):
            hin = h if src < 0 else refs[src]["y"].shape[1]
            L = qi.Layer(name, n, hin, hin, c, k, r, r, stride, pad, bits, xs, True, qi.S8 if xs else qi.U4,
                         qi.S8 if xs else (-7, 7))
            t = qi.layer_tensors(8181, seed * 100 + i, L)
            sh = stress_shift(L, L.x_range, L.w_range)
            bias = g.integers(-400, 400, size=k).astype(np.int32)
            relu = bool(g.random() < 0.7)
            res = None if rsrc is None else (in_vals if rsrc < 0 else refs[rsrc]["y"])
            refs.append(oracle.qconv_layer(None, t["w"], bits=bits, x_signed=xs, w_signed=True,
                                           stride=(stride, stride), pad=(pad, pad), mult=t["mult"], shift=sh,
                                           relu=relu, lo=lo, hi=hi, bias=bias, residual=res,
                                           packed_x=xp_ref if src < 0 else refs[src]["y_packed"],
                                           threads=oracle_threads()))
            specs.append(nets.LayerSpec(L.desc(), q.pack(torch.from_numpy(t["w"]).to(dev), bits, True),
                                        torch.from_numpy(t["mult"]).to(dev), sh, relu, (lo, hi), src=src,
                                        bias=torch.from_numpy(bias).to(dev), residual_src=rsrc, residual_signed=xs))
        xp = q.pack(torch.from_numpy(x).to(dev), bits, xs)
        for branches in (False, True):
            chain = nets.Chain(specs, xp, branches=branches)
            announce(f"net {seed} {[s[0] for s in spec]} n={n} h={h} bits={bits} branches={branches} eager")
            outs = [o.clone() for o in chain.forward()]
            torch.cuda.synchronize()
            for (name, *_), o, ref in zip(spec, outs, refs):
                assert_same(o.cpu().numpy(), ref["y_packed"], f"net {seed} eager {name}")
            chain.capture()
            for rep in range(3):
                for o in chain.outputs:
                    o.zero_()
                announce(f"net {seed} replay {rep} branches={branches}")
                got = chain.replay()
                torch.cuda.synchronize()
                for (name, *_), o, ref in zip(spec, got, refs):
                    assert_same(o.cpu().numpy(), ref["y_packed"], f"net {seed} replay {rep} {name}")
                chain.forward()
                torch.cuda.synchronize()


def test_random_few_channel_layers_by_unrolling():
    """Random 8-bit layers with 1-4 input channels and 3x3 to 7x7 filters
    (square or not, stride 1 or 2): input and filters patch-unrolled on the GPU
    with either fold (checked against the unroll's definition), then the folded
    convolution on every tile that takes it, against the oracle's direct
    convolution of the original tensors."""
    import torch
    from paper_2202_06819_amd import qconv as q
    from _util import unroll_def

    dev = torch.device("cuda:0")
    ran = 0
    for seed in range(30):
        g = np.random.default_rng([3131, seed])
        c, r = int(g.integers(1, 5)), int(g.choice([3, 5, 7]))
        s = int(g.choice([r, r, 3]))
        stride, pad = int(g.choice([1, 2, 2])), int(g.integers(0, r // 2 + 1))
        h, w, n, k = int(g.integers(r, 65)), int(g.integers(s, 65)), int(g.integers(1, 5)), 8 * int(g.integers(1, 13))
        L = qi.Layer(f"u{seed}", n, h, w, c, k, r, s, stride, pad, bits=8, x_signed=True, w_signed=True,
                     x_range=qi.S8, w_range=qi.S8, epilogue=qi.Epilogue(relu=True, lo=-128, hi=127))
        t = qi.layer_tensors(3131, seed, L)
        sh = stress_shift(L, L.x_range, L.w_range)
        ref = oracle.qconv_layer(t["x"], t["w"], bits=8, x_signed=True, w_signed=True, stride=(stride, stride),
                                 pad=(pad, pad), mult=t["mult"], shift=sh, relu=True, lo=-128, hi=127,
                                 threads=oracle_threads())
        mult = torch.from_numpy(t["mult"]).to(dev)
        for fold in ("rows", "all"):
            c_out = -(-((stride if fold == "rows" else r) * s * c) // 64) * 64
            plan = q.few_channel_plan(L.desc(), c_out, fold)
            announce(f"{L.name} {L.desc()} fold {fold} into {c_out} channels")
            xu = q.unroll(torch.from_numpy(t["x"]).to(dev), c_out, **plan["x"])
            wu = q.unroll(torch.from_numpy(t["w"]).to(dev), c_out, **plan["w"])
            torch.cuda.synchronize()
            assert np.array_equal(xu.cpu().numpy(), unroll_def(t["x"], c_out, **plan["x"])), f"{L.name} x"
            assert np.array_equal(wu.cpu().numpy(), unroll_def(t["w"], c_out, **plan["w"])), f"{L.name} w"
            d = plan["desc"]
            for tt in q.tiles():
                if q.tile_status(d, tt["id"]) != 0:
                    continue
                announce(f"{L.name} fold {fold} tile {tt['name']}")
                y = q.conv2d(d, xu, wu, tile=tt["id"], requant=True, mult=mult, shift=sh, relu=True,
                             clamp=(-128, 127))
                torch.cuda.synchronize()
                assert_same(y.cpu().numpy(), ref["y_packed"], f"{L.name} {fold} {tt['name']}")
                ran += 1
    assert ran > 0


def test_random_shapes_per_axis_strides_and_paddings():
    """Independent strides (1-3) and paddings per axis and non-square filters,
    all in one process (so layers that differ in one axis only follow each
    other): every tile raw and requantised, the wide tiles also from prepared
    filters and with a random split."""
    import torch
    from paper_2202_06819_amd import qconv as q

    dev = torch.device("cuda:0")
    tiles_all = q.tiles()
    ran = 0
    for seed in range(100):
        g = np.random.default_rng([6262, seed])
        bits = 8 if seed % 3 == 2 else 4
        r = int(g.choice([1, 3, 3, 5, 2]))
        s = int(g.choice([r, r, 1, 3]))
        sh, sw = int(g.choice([1, 1, 2, 3])), int(g.choice([1, 1, 2, 3]))
        ph, pw = int(g.integers(0, r // 2 + 2)), int(g.integers(0, s // 2 + 2))
        h, w = int(g.integers(max(1, r - 2 * ph), 40)), int(g.integers(max(1, s - 2 * pw), 40))
        n = int(g.integers(1, 9))
        c, k = (8 if bits == 4 else 4) * int(g.integers(1, 40)), 8 * int(g.integers(1, 30))
        xs = bits == 8 or bool(g.random() < 0.2)
        xr = qi.S8 if bits == 8 else (qi.S4 if xs else qi.U4)
        wr = qi.S8 if bits == 8 else qi.S4
        d = dict(n=n, h=h, w=w, c=c, k=k, r=r, s=s, stride_h=sh, stride_w=sw, pad_h=ph, pad_w=pw, bits=bits,
                 x_signed=int(xs), w_signed=1)
        tiles = [t["id"] for t in tiles_all if q.tile_status(d, t["id"]) == 0]
        if not tiles:
            continue
        x = g.integers(xr[0], xr[1] + 1, size=(n, c, h, w)).astype(np.int8)
        f = g.integers(wr[0], wr[1] + 1, size=(k, c, r, s)).astype(np.int8)
        mult = g.integers(2 ** 14, 2 ** 15, size=k).astype(np.int32)
        shift = stress_shift(qi.Layer("a", n, h, w, c, k, r, s, 1, 0, bits, xs, True, xr, wr), xr, wr)
        lo, hi = (-128, 127) if bits == 8 else (0, 15)
        ref = oracle.qconv_layer(x, f, bits=bits, x_signed=xs, w_signed=True, stride=(sh, sw), pad=(ph, pw),
                                 mult=mult, shift=shift, relu=True, lo=lo, hi=hi, threads=oracle_threads())
        xp = q.pack(torch.from_numpy(x).to(dev), bits, xs)
        wp = q.pack(torch.from_numpy(f).to(dev), bits, True)
        m_dev = torch.from_numpy(mult).to(dev)
        for tid in tiles:
            announce(f"per-axis {d} tile {tid}")
            y = q.conv2d(d, xp, wp, tile=tid)
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["acc"], f"{d} tile {tid} raw")
            y = q.conv2d(d, xp, wp, tile=tid, requant=True, mult=m_dev, shift=shift, relu=True, clamp=(lo, hi))
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["y_packed"], f"{d} tile {tid} requant")
            ran += 1
            if tiles_all[tid]["variant"] != 2:
                continue
            wprep = q.prepare_filters(d, wp, tid)
            y = q.conv2d(d, xp, wprep, tile=tid, prepared=True)
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["acc"], f"{d} tile {tid} prepared")
            most = q.max_splits(d, tid)
            if most > 1:
                splits = int(g.integers(2, most + 1))
                y = q.conv2d(d, xp, wprep, tile=tid, prepared=True, splits=splits,
                             workspace=q.make_workspace(d, tid, splits, dev))
                torch.cuda.synchronize()
                assert_same(y.cpu().numpy(), ref["acc"], f"{d} tile {tid} splits {splits}")
    assert ran > 0


def test_random_fused_pack_per_axis_strides():
    """The pack fused into 3x3 convolutions with independent strides per axis,
    widths with and without whole pixel octets and 1-4 channel chunks, from
    int8 input over the whole int8 range: requantised (with the packed copy
    where the bands cover every input row) and raw, on every wide tile."""
    import torch
    from paper_2202_06819_amd import qconv as q

    dev = torch.device("cuda:0")
    ran = 0
    for seed in range(40):
        g = np.random.default_rng([7373, seed])
        bits = 8 if seed % 3 == 2 else 4
        sh, sw = int(g.choice([1, 1, 2])), int(g.choice([1, 1, 2]))
        h = int(g.integers(1, 48))
        w = int(8 * g.integers(1, 7)) if g.random() < 0.5 else int(g.integers(1, 48))
        n = int(g.integers(1, 9))
        c = 64 * int(g.integers(1, 4)) if bits == 4 else 32 * int(g.integers(1, 5))
        k = 8 * int(g.integers(1, 24))
        signed = bits == 8
        d = dict(n=n, h=h, w=w, c=c, k=k, r=3, s=3, stride_h=sh, stride_w=sw, pad_h=1, pad_w=1, bits=bits,
                 x_signed=int(signed), w_signed=1)
        tiles = [t for t in q.tiles() if t["variant"] == 2 and q.tile_status(d, t["id"]) == 0]
        if not tiles:
            continue
        x = g.integers(-128, 128, size=(n, c, h, w)).astype(np.int8)
        wr = qi.S8 if signed else (-7, 7)
        f = g.integers(wr[0], wr[1] + 1, size=(k, c, 3, 3)).astype(np.int8)
        mult = g.integers(2 ** 14, 2 ** 15, size=k).astype(np.int32)
        L = qi.Layer("f", n, h, w, c, k, 3, 3, 1, 1, bits, signed, True, qi.S8 if signed else (0, 15), wr)
        shift = stress_shift(L, L.x_range, wr)
        lo, hi, relu = (-128, 127, False) if signed else (0, 15, True)
        ref = oracle.qconv_layer(x, f, bits=bits, x_signed=signed, w_signed=True, stride=(sh, sw), pad=(1, 1),
                                 mult=mult, shift=shift, relu=relu, lo=lo, hi=hi, threads=oracle_threads())
        x_dev = torch.from_numpy(x).to(dev)
        wp = q.pack(torch.from_numpy(f).to(dev), bits, True)
        m_dev = torch.from_numpy(mult).to(dev)
        for t in tiles:
            wprep = q.prepare_filters(d, wp, t["id"])
            announce(f"fused per-axis {d} tile {t['name']}")
            call = q.PackingConv2dCall(d, x_dev, wprep, tile=t["id"], mult=m_dev, shift=shift, relu=relu,
                                       clamp=(lo, hi), x_packed=True)
            try:
                y = call()
                copy = True
            except q.QConvError as ex:
                assert "no packed copy" in str(ex), str(ex)
                y = q.PackingConv2dCall(d, x_dev, wprep, tile=t["id"], mult=m_dev, shift=shift, relu=relu,
                                        clamp=(lo, hi))()
                copy = False
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["y_packed"], f"{d} {t['name']}")
            if copy:
                assert_same(call.x_packed.cpu().numpy(), ref["x_packed"], f"{d} {t['name']} packed copy")
            y = q.PackingConv2dCall(d, x_dev, wprep, tile=t["id"], requant=False)()
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["acc"], f"{d} {t['name']} raw")
            ran += 1
    assert ran > 0
