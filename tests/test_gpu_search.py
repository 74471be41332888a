"""Schedules on the GPU: every launch knob of qconv2d_scheduled against the
oracle, random schedules on random shapes, and a short live search whose
measured schedules are all checked."""
import random

import pytest

import qconv_inputs as qi
from _util import announce, assert_same, random_layer, ref_layer, stress_shift

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape", [
    ("n32_56_64to64_3x3", 32, 56, 64, 64, 3, 1, 1),      # persistent single-chunk plans
    ("n4_14_256to256_3x3", 4, 14, 256, 256, 3, 1, 1),    # several chunks, split-K
    ("n16_28_128to256_1x1_s2", 16, 28, 128, 256, 1, 2, 0),
], ids=lambda v: v[0])
def test_scheduled_matches_oracle(shape):
    import torch
    from paper_2202_06819_amd import qconv, search
    name, n, h, c, k, r, stride, pad = shape
    L = qi.Layer(name, n, h, h, c, k, r, r, stride, pad, w_range=(-7, 7))
    t = qi.layer_tensors(800, c + k + r, L)
    sh = stress_shift(L, L.x_range, L.w_range)
    ref = ref_layer(L, t, requant=True, shift=sh)
    dev = torch.device("cuda:0")
    xp = qconv.pack(torch.from_numpy(t["x"]).to(dev), 4, False)
    wp = qconv.pack(torch.from_numpy(t["w"]).to(dev), 4, True)
    mult = torch.from_numpy(t["mult"]).to(dev)
    space = search.ScheduleSpace.for_shape(L.desc())
    rng = random.Random(5)
    picks = rng.sample(space.configs, min(40, len(space)))
    # and every launch-knob combination of one wide tile
    wide = [cfg for cfg in space.configs if cfg[0] == 2]
    tk = wide[0][:6]
    picks += [cfg for cfg in space.configs if cfg[:6] == tk]
    prepared = {}
    for cfg in dict.fromkeys(picks):
        sch = space.schedule(cfg)
        tid = sch["tile_id"]
        if tid not in prepared:
            prepared[tid] = qconv.prepare_filters(L.desc(), wp, tid)
        ws = qconv.make_workspace(L.desc(), tid, sch["splits"], dev)
        announce(f"{name} schedule {sch}")
        for rep in range(2 if sch["splits"] > 1 else 1):
            y = qconv.Conv2dCall(L.desc(), xp, prepared[tid], schedule=sch, workspace=ws, requant=True, mult=mult,
                                 shift=sh)()
            torch.cuda.synchronize()
            assert_same(y.cpu().numpy(), ref["y_packed"], f"{name} {sch} rep {rep}")


def test_live_search_checks_every_schedule():
    import torch
    from paper_2202_06819_amd import search
    L = qi.Layer("live_2x28_128to128", 2, 28, 28, 128, 128, 3, 3, 1, 1)
    meas = search.LiveMeasure(L, torch.device("cuda:0"), reps=10, rounds=2)
    meas.space = search.ScheduleSpace.for_shape(L.desc())
    announce(f"live search over {len(meas.space)} schedules")
    res = search.search(meas.space, meas, trials=24, batch=8, diversity=True, seed=0, n_iter=60)
    assert len(res.trials) == 24
    assert all(t.us > 0 for t in res.trials)


@pytest.mark.parametrize("block", [(0, False), (5000, True)], ids=["small", "large"])
def test_random_shapes_random_schedules(block):
    """Random shapes (the generator of the random-shape parity tests), each
    with up to 30 schedules drawn from its whole space: tile, split-K,
    workgroups per CU, band buffers, block order and grid size."""
    import torch
    from paper_2202_06819_amd import qconv, search
    first, big = block
    dev = torch.device("cuda:0")
    ran = 0
    for seed in range(first, first + 25):
        L = random_layer(seed, big)
        if L.h + 2 * L.pad < L.r or L.w + 2 * L.pad < L.s:
            continue
        d, e = L.desc(), L.epilogue
        space = search.ScheduleSpace.for_shape(d)
        assert len(space) > 0, f"empty schedule space for {d}"
        t = qi.layer_tensors(9191, seed, L)
        sh = stress_shift(L, L.x_range, L.w_range)
        ref = ref_layer(L, t, requant=True, shift=sh)
        xp = qconv.pack(torch.from_numpy(t["x"]).to(dev), L.bits, L.x_signed)
        wp = qconv.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
        mult = torch.from_numpy(t["mult"]).to(dev)
        prepared = {}
        for cfg in random.Random(seed).sample(space.configs, min(30, len(space))):
            sch = space.schedule(cfg)
            tid = sch["tile_id"]
            if tid not in prepared:
                prepared[tid] = qconv.prepare_filters(d, wp, tid)
            ws = qconv.make_workspace(d, tid, sch["splits"], dev)
            announce(f"{L.name} {d} schedule {sch}")
            for rep in range(2 if sch["splits"] > 1 else 1):
                y = qconv.Conv2dCall(d, xp, prepared[tid], schedule=sch, workspace=ws, requant=True, mult=mult,
                                     shift=sh, relu=e.relu, clamp=(e.lo, e.hi))()
                torch.cuda.synchronize()
                assert_same(y.cpu().numpy(), ref["y_packed"], f"{L.name} {sch} rep {rep}")
                ran += 1
    assert ran > 0
