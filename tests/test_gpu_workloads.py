"""The benchmark workloads at their full sizes, in the launch configuration
bench.py times (the tuned tile and split-K factor, prepared filters), on the
same seeded inputs, compared element by element with the oracle: every layer
of every workload, and the chained ResNet-18 stacks (plain and as residual
blocks with biases) layer by layer."""
import numpy as np
import pytest

import oracle
import qconv_inputs as qi
from _util import announce, assert_same, oracle_threads, stress_shift

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


def _layers(cfg):
    layers = qi.WORKLOADS[cfg]()
    return list(enumerate(qi.distinct(layers) if cfg in (2, 3) else layers))


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_workload_layers_full_size(cfg):
    torch = _torch()
    from paper_2202_06819_amd import qconv, sweep
    dev = torch.device("cuda:0")
    for lid, L in _layers(cfg):
        t = qi.layer_tensors(cfg, lid, L)
        e = L.epilogue
        d = L.desc()
        xp = qconv.pack(torch.from_numpy(t["x"]).to(dev), L.bits, L.x_signed)
        wp = qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
        tile, splits = sweep.tuned_config(d, e is not None)
        wprep = qconv.prepare_filters(d, wp, tile)
        ws = qconv.make_workspace(d, tile, splits, dev)
        stride, pad = (L.stride, L.stride), (L.pad, L.pad)
        kw = dict(bits=L.bits, x_signed=L.x_signed, w_signed=L.w_signed, stride=stride, pad=pad,
                  threads=oracle_threads())
        if e is None:
            ref = oracle.qconv_layer(t["x"], t["w"], **kw)
            announce(f"workload {cfg} {L.name} raw, tile {tile} splits {splits}")
            y = qconv.Conv2dCall(d, xp, wprep, tile=tile, prepared=True, splits=splits, workspace=ws)()
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["acc"], f"workload {cfg} {L.name} raw")
            continue
        mult = torch.from_numpy(t["mult"]).to(dev)
        # the literal epilogue (what the benchmark times) and one whose outputs
        # spread over the clamp range (the literal one leaves most of them 0)
        for shift in (e.shift, stress_shift(L, L.x_range, L.w_range)):
            ref = oracle.qconv_layer(t["x"], t["w"], mult=t["mult"], shift=shift, relu=e.relu, lo=e.lo, hi=e.hi,
                                     **kw)
            announce(f"workload {cfg} {L.name} shift {shift}, tile {tile} splits {splits}")
            y = qconv.Conv2dCall(d, xp, wprep, requant=True, mult=mult, shift=shift, relu=e.relu,
                                 clamp=(e.lo, e.hi), tile=tile, prepared=True, splits=splits, workspace=ws)()
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["y_packed"], f"workload {cfg} {L.name} shift {shift}")
            if cfg in (2, 3) and shift == e.shift:
                announce(f"workload {cfg} {L.name} raw")
                y = qconv.Conv2dCall(d, xp, wprep, tile=tile, prepared=True, splits=splits, workspace=ws)()
                torch.cuda.synchronize()
                assert_same(y.cpu().numpy(), ref["acc"], f"workload {cfg} {L.name} raw")


@pytest.mark.parametrize("cfg,residual", [(2, False), (2, True), (3, False), (3, True)])
def test_chain_full_size(cfg, residual):
    """The chained stack as bench.py builds it (inputs, biases, shortcut order),
    on one stream and with the projections on a second stream (eager and as a
    graph replay), every layer's output against the oracle fed with the
    oracle's own packed outputs."""
    torch = _torch()
    import bench
    from paper_2202_06819_amd import nets, qconv
    dev = torch.device("cuda:0")
    layers = qi.WORKLOADS[cfg]()
    t0 = qi.layer_tensors(cfg, 0, layers[0])
    xp = qconv.pack(torch.from_numpy(t0["x"]).to(dev), layers[0].bits, layers[0].x_signed)
    plan = bench.residual_order(layers) if residual else [(L, L.src, None, i) for i, L in enumerate(layers)]
    specs, host = [], []
    for L, src, short, lid in plan:
        t = qi.layer_tensors(cfg, lid, L)
        e = L.epilogue
        bias = None
        if residual:
            bias = np.random.default_rng([cfg, lid, 3]).integers(-256, 256, size=L.k).astype(np.int32)
        specs.append(nets.LayerSpec(L.desc(), qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed),
                                    torch.from_numpy(t["mult"]).to(dev), e.shift, e.relu, (e.lo, e.hi), src=src,
                                    bias=None if bias is None else torch.from_numpy(bias).to(dev),
                                    residual_src=short, residual_signed=e.lo < 0))
        host.append((L, src, short, t, bias))
    announce(f"chain workload {cfg} residual={residual}: {len(specs)} layers")
    chain = nets.Chain(specs, xp)
    outs = [o.cpu().numpy() for o in chain.forward()]
    torch.cuda.synchronize()
    announce(f"chain workload {cfg} residual={residual}: projections on a second stream, eager and replayed")
    chain_b = nets.Chain(specs, xp, branches=True)
    assert sum(chain_b.on_side) == 3
    outs_b = [o.cpu().numpy() for o in chain_b.forward()]
    chain_b.capture()
    for o in chain_b.outputs:
        o.zero_()
    chain_b.replay()
    torch.cuda.synchronize()
    outs_g = [o.cpu().numpy() for o in chain_b.outputs]
    x_packed = oracle.relayout_pack(t0["x"], layers[0].bits, layers[0].x_signed)
    ref_out = []
    for i, (L, src, short, t, bias) in enumerate(host):
        e = L.epilogue
        inp = x_packed if src < 0 else ref_out[src]
        res = None
        if short is not None:
            rp = x_packed if short < 0 else ref_out[short]
            res = oracle.unpack_tensor(rp, L.k, L.bits, e.lo < 0)
        ref = oracle.qconv_layer(None, t["w"], bits=L.bits, x_signed=L.x_signed, w_signed=L.w_signed,
                                 stride=(L.stride, L.stride), pad=(L.pad, L.pad), mult=t["mult"], shift=e.shift,
                                 relu=e.relu, lo=e.lo, hi=e.hi, threads=oracle_threads(), packed_x=inp, bias=bias,
                                 residual=res)
        ref_out.append(ref["y_packed"])
        assert_same(outs[i], ref["y_packed"], f"chain {cfg} layer {i} ({L.name})")
        assert_same(outs_b[i], ref["y_packed"], f"chain {cfg} layer {i} ({L.name}), two streams")
        assert_same(outs_g[i], ref["y_packed"], f"chain {cfg} layer {i} ({L.name}), two streams replayed")
