"""Host logic of chained layers: which layers of a network run on a second
stream and which events order them (no GPU needed)."""
from types import SimpleNamespace

import bench
import qconv_inputs as qi
from paper_2202_06819_amd.nets import branch_plan


def _specs(plan):
    return [SimpleNamespace(name=L.name, src=src, residual_src=short) for L, src, short, _ in plan]


def _check_ordered(specs, on_side, waits):
    """Every input of every layer is produced earlier, and either on the same
    stream or behind an event the layer waits for."""
    for i, s in enumerate(specs):
        for d in (s.src, s.residual_src):
            if d is None or d < 0:
                continue
            assert d < i
            assert on_side[d] == on_side[i] or d in waits[i], (s.name, d)
        for d in waits[i]:
            assert on_side[d] != on_side[i]


def test_resnet18_projections_go_to_the_second_stream():
    layers = qi.workload2()
    plain = _specs([(L, L.src, None, i) for i, L in enumerate(layers)])
    resid = _specs(bench.residual_order(layers))
    for specs in (plain, resid):
        on_side, waits = branch_plan(specs)
        assert [s.name for s, f in zip(specs, on_side) if f] == [f"l{k}.0.downsample" for k in (2, 3, 4)]
        _check_ordered(specs, on_side, waits)
        for i, s in enumerate(specs):
            if on_side[i]:
                assert waits[i] == [s.src]          # the block input, made on the first stream
    # in residual order the block's second 3x3 adds the projection: it waits for it
    on_side, waits = branch_plan(resid)
    for i, s in enumerate(resid):
        if s.residual_src is not None and s.residual_src >= 0 and on_side[s.residual_src]:
            assert waits[i] == [s.residual_src]
    assert sum(1 for w, f in zip(waits, on_side) if w and not f) == 3


def test_straight_chain_stays_on_one_stream():
    specs = [SimpleNamespace(src=i - 1, residual_src=None) for i in range(6)]
    on_side, waits = branch_plan(specs)
    assert not any(on_side) and not any(waits)


def test_layer_feeding_the_next_stays_on_the_first_stream():
    # layer 2 reads layer 0 (not its predecessor) but feeds layer 3, so the
    # main line does not step over it: not a branch
    specs = [SimpleNamespace(src=-1, residual_src=None), SimpleNamespace(src=0, residual_src=None),
             SimpleNamespace(src=0, residual_src=None), SimpleNamespace(src=2, residual_src=1)]
    on_side, waits = branch_plan(specs)
    assert on_side == [False, False, False, False]
    # layer 1 reads the input beside layer 0 and is only added later: a branch
    specs = [SimpleNamespace(src=-1, residual_src=None), SimpleNamespace(src=-1, residual_src=None),
             SimpleNamespace(src=0, residual_src=1), SimpleNamespace(src=2, residual_src=None)]
    on_side, waits = branch_plan(specs)
    assert on_side == [False, True, False, False] and waits == [[], [], [1], []]
    _check_ordered(specs, on_side, waits)
    # the last layer is never a branch, whatever it reads
    specs = [SimpleNamespace(src=-1, residual_src=None), SimpleNamespace(src=0, residual_src=None),
             SimpleNamespace(src=0, residual_src=1)]
    assert branch_plan(specs)[0] == [False, False, False]


def _desc_specs(plan):
    return [SimpleNamespace(name=L.name, desc=L.desc(), src=src, residual_src=short) for L, src, short, _ in plan]


def test_resnet18_stage_entries_pair_with_their_projections():
    """Each stage's strided 3x3 and its 1x1 projection read the block input:
    they form the three fused launches, in plain and in residual order."""
    from paper_2202_06819_amd.nets import projection_pairs
    for layers in (qi.workload2(), qi.workload3()):
        for specs in (_desc_specs([(L, L.src, None, i) for i, L in enumerate(layers)]),
                      _desc_specs(bench.residual_order(layers))):
            pairs = projection_pairs(specs)
            assert sorted((specs[i].name, specs[j].name) for i, j in pairs.items()) == \
                [(f"l{k}.0.conv1", f"l{k}.0.downsample") for k in (2, 3, 4)]
            for i, j in pairs.items():
                assert i < j and specs[i].src == specs[j].src
            assert len(specs) - len(pairs) == 16   # launches per forward pass


def test_projection_pairs_need_the_same_input_and_stride():
    from paper_2202_06819_amd.nets import projection_pairs
    d3 = dict(n=2, h=8, w=8, c=64, k=64, r=3, s=3, stride_h=2, stride_w=2, pad_h=1, pad_w=1, bits=4, x_signed=0,
              w_signed=1)
    d1 = dict(d3, r=1, s=1, pad_h=0, pad_w=0)
    mk = lambda d, src, res=None: SimpleNamespace(desc=d, src=src, residual_src=res)
    assert projection_pairs([mk(d3, -1), mk(d1, -1)]) == {0: 1}
    assert projection_pairs([mk(d3, -1), mk(d1, 0)]) == {}                          # other input
    assert projection_pairs([mk(d3, -1), mk(dict(d1, stride_h=1, stride_w=1), -1)]) == {}   # other stride
    assert projection_pairs([mk(d3, -1), mk(dict(d1, k=128), -1)]) == {}            # other channels
    assert projection_pairs([mk(dict(d3, pad_h=0, pad_w=0), -1), mk(d1, -1)]) == {}  # centre tap moves
    assert projection_pairs([mk(d3, -1), mk(d1, -1, res=0)]) == {}                  # projection with a residual
    assert projection_pairs([mk(d1, -1), mk(d3, -1)]) == {}                         # the 1x1 must come later
