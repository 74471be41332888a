"""The schedule search (cost model + annealing + diversity-aware selection) on
the CPU: its building blocks, a synthetic space with a known optimum, and the
real schedule space the library reports for the benchmark layer."""
import itertools
import random

import numpy as np
import pytest

from paper_2202_06819_amd import search as S


def _synthetic_space():
    # ten knobs like the real space; a few combinations are invalid
    doms = [(0, 2), (1, 2, 4, 8), (1, 2, 4), (1, 2, 4), (1, 2, 4), (64, 128), (1, 2, 4), (0, 1, 2), (0, 1, 2), (0, 1)]
    cfgs = []
    for c in itertools.product(*doms):
        if c[0] == 0 and c[6] != 1:          # "staged" tiles have no split
            continue
        if c[1] * c[2] > 8 or c[3] * c[4] > 8:  # too many waves / fragments
            continue
        cfgs.append(c)
    return S.ScheduleSpace(cfgs)


def _objective(c):
    # smooth in the tile knobs, a few knobs that do nothing, one interaction
    v, wp, wk, fp, fk, ck, sp, wg, bb, xo = c
    us = 10.0 + 3.0 * abs(np.log2(wp * fp) - 3) + 2.0 * abs(np.log2(wk * fk) - 2) + (2.0 if v == 0 else 0.0)
    us += 0.8 * abs(np.log2(sp) - 1) + (0.5 if ck == 128 else 0.0) + (0.3 if xo == 0 else 0.0)
    us += 0.0 * wg + 0.0 * bb
    return float(us)


def test_mutation_changes_one_knob_and_stays_valid():
    space = _synthetic_space()
    rng = random.Random(0)
    for c in rng.sample(space.configs, 200):
        m = space.mutate(c, rng)
        assert m in space.valid
        assert S.ScheduleSpace.distance(c, m) in (0, 1)
    assert sum(S.ScheduleSpace.distance(c, space.mutate(c, rng)) == 1 for c in space.configs[:300]) > 250


def test_diverse_half_is_diverse_and_keeps_the_best():
    space = _synthetic_space()
    rng = random.Random(1)
    base = rng.choice(space.configs)
    cands = [space.mutate(base, rng) for _ in range(40)] + rng.sample(space.configs, 40)
    scores = np.array([-_objective(c) for c in cands])
    sel = S.diverse_half(space, cands, scores, 40)
    assert len(sel) == len(set(sel)) == 40
    assert sel[0] == int(np.argmax(scores))

    by_score = list(np.argsort(-scores)[:40])
    distinct_sel = len({cands[i] for i in sel})
    distinct_top = len({cands[i] for i in by_score})
    assert distinct_sel >= distinct_top


def test_cost_model_ranks_held_out_schedules():
    space = _synthetic_space()
    rng = random.Random(2)
    pts = rng.sample(space.configs, 160)
    train, test = pts[:96], pts[96:]
    m = S.CostModel(0)
    m.fit(space.features(train), np.array([_objective(c) for c in train]))
    pred = m.predict(space.features(test))
    truth = -np.array([_objective(c) for c in test])
    rho = np.corrcoef(np.argsort(np.argsort(pred)), np.argsort(np.argsort(truth)))[0, 1]
    assert rho > 0.8, rho


@pytest.mark.parametrize("diversity", [False, True])
def test_search_finds_the_optimum_of_a_known_space(diversity):
    space = _synthetic_space()
    best = min(_objective(c) for c in space.configs)
    hits = 0
    for seed in range(4):
        res = S.search(space, _objective, trials=96, diversity=diversity, seed=seed, n_iter=150)
        assert len(res.trials) == 96
        assert len({t.cfg for t in res.trials}) == 96                  # nothing measured twice
        assert all(t.best_us == min(u.us for u in res.trials[:t.index + 1]) for t in res.trials)
        hits += res.best().us <= best * 1.02
    # random choice of 96 of these schedules reaches the optimum band rarely
    assert hits >= 3


def test_search_stops_at_the_space_size():
    cfgs = [(2, 1, 1, f, 4, 64, 1, w, 0, 1) for f in (1, 2, 4) for w in (0, 1, 2)]
    space = S.ScheduleSpace(cfgs)
    res = S.search(space, _objective, trials=50, seed=0)
    assert len(res.trials) == len(cfgs)


def test_real_space_of_the_benchmark_layer():
    from paper_2202_06819_amd import build, qconv
    import os
    import qconv_inputs as qi
    if not os.path.exists(build.LIB):
        build.build()
    L = qi.workload1()[0]
    space = S.ScheduleSpace.for_shape(L.desc())
    assert len(space) > 100
    rng = random.Random(3)
    for c in rng.sample(space.configs, 40):
        sch = space.schedule(c)
        assert qconv.schedule_status(L.desc(), sch) == 0
        t = qconv.tiles()[sch["tile_id"]]
        assert (t["variant"], t["waves_p"], t["waves_k"], t["frag_p"], t["frag_k"], t["chunk_c"]) == c[:6]
    assert space.features(space.configs[:5]).shape[0] == 5
