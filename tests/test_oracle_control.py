"""Pins of the controller oracle (Alg. 1, §3.3, App. B.1, App. C.7)
against values worked out by hand from the paper's formulas, the closed
form of the reserve recurrence, special cases, and invariants."""

import numpy as np
from hypothesis import given, settings, strategies as st

from oracle import control as oc
from oracle import lowering as olow

PAGE = 16


def _apply(tags, pairs, value):
    for s, j in pairs:
        tags[s, 2 * j] = tags[s, 2 * j + 1] = value


def test_hand_worked_trace():
    """Two sequences of 320 and 192 tokens (10 and 6 full pairs), sink 1 and
    recent 1 pair protected, B_min = 4, lambda = 2.  Every number below was
    worked out by hand from Alg. 1; F_post = F_t + n_d - D_t (the step's
    demand is allocated after the demotion)."""
    cfg = oc.Config(min_batch=4, decay=2, sink_pairs=1, recent_pairs=1)
    ctl = oc.Controller(cfg)
    lens = np.array([320, 192], dtype=np.int32)
    tags = np.zeros((2, 20), dtype=np.uint8)

    # step 1: D=7, F=5 -> Delta=2, n_d=max(2,4)=4, E=2; F_post=2, R=2, P=0
    d = ctl.demotion(7, 5, tags, lens)
    assert d.tolist() == [[0, 1], [1, 1], [0, 2], [1, 2]]
    assert (ctl.shortage, ctl.surplus) == (2, 2)
    _apply(tags, d, 1)
    p = ctl.promotion(2, 8, tags, lens)
    assert (ctl.reserve, ctl.budget, len(p)) == (2, 0, 0)

    # step 2: D=3, F=2 -> Delta=1, n_d=4, E=3; F_post=3, R=max(0,2-2)+3=3, P=0
    d = ctl.demotion(3, 2, tags, lens)
    assert d.tolist() == [[0, 3], [1, 3], [0, 4], [1, 4]]
    assert (ctl.shortage, ctl.surplus) == (1, 3)
    _apply(tags, d, 1)
    p = ctl.promotion(3, 8, tags, lens)
    assert (ctl.reserve, ctl.budget, len(p)) == (3, 0, 0)

    # step 3: no shortage; F_post=3, R=max(0,3-2)=1, P=2 -> the two newest BASE pairs
    d = ctl.demotion(0, 3, tags, lens)
    assert len(d) == 0 and (ctl.shortage, ctl.surplus) == (0, 0)
    p = ctl.promotion(3, 8, tags, lens)
    assert (ctl.reserve, ctl.budget) == (1, 2)
    assert p.tolist() == [[0, 4], [1, 4]]
    _apply(tags, p, 0)

    # step 4: F=1 after those promotions; R=max(0,1-2)=0, P=1
    d = ctl.demotion(0, 1, tags, lens)
    assert len(d) == 0
    p = ctl.promotion(1, 8, tags, lens)
    assert (ctl.reserve, ctl.budget) == (0, 1)
    assert p.tolist() == [[0, 3]]
    _apply(tags, p, 0)

    # step 5: D=6, F=0 -> Delta=6, n_d=6 of the 7 eligible, E=0
    d = ctl.demotion(6, 0, tags, lens)
    assert d.tolist() == [[0, 3], [0, 4], [1, 4], [0, 5], [0, 6], [0, 7]]
    assert (ctl.shortage, ctl.surplus) == (6, 0)
    _apply(tags, d, 1)
    p = ctl.promotion(0, 8, tags, lens)
    assert (ctl.reserve, ctl.budget, len(p)) == (0, 0, 0)


def _many_pairs(nseq=4, pairs=40):
    lens = np.full(nseq, 32 * pairs, dtype=np.int32)
    return lens, np.zeros((nseq, 2 * pairs), dtype=np.uint8)


@given(st.integers(1, 60), st.integers(1, 6), st.integers(0, 40))
@settings(max_examples=60, deadline=None)
def test_reserve_decay_closed_form(surplus, decay, free_post):
    """One demotion with surplus E, then only steps without shortage:
    R_k = max(0, E - lambda k) and P_k = max(0, F_post - R_k)."""
    lens, tags = _many_pairs()
    ctl = oc.Controller(oc.Config(min_batch=surplus + 1, decay=decay, no_promotion=True))
    d = ctl.demotion(1, 0, tags, lens)         # shortage 1, B_min = E + 1 pairs
    assert len(d) == surplus + 1 and ctl.surplus == surplus
    for k in range(12):
        if k:
            assert len(ctl.demotion(0, 100, tags, lens)) == 0
        ctl.promotion(free_post, 100, tags, lens)
        assert ctl.reserve == max(0, surplus - decay * k)
        assert ctl.budget == max(0, free_post - ctl.reserve)


def test_no_shortage_leaves_native_path_alone():
    lens, tags = _many_pairs()
    ctl = oc.Controller(oc.Config())
    assert len(ctl.demotion(5, 5, tags, lens)) == 0
    assert len(ctl.demotion(0, 9, tags, lens)) == 0
    assert ctl.surplus == 0


def test_min_batch_capped_by_eligible_pairs():
    lens = np.array([32 * 5], dtype=np.int32)          # 5 full pairs
    tags = np.zeros((1, 10), dtype=np.uint8)
    ctl = oc.Controller(oc.Config(min_batch=16, sink_pairs=1, recent_pairs=1))
    d = ctl.demotion(2, 0, tags, lens)
    assert d.tolist() == [[0, 1], [0, 2], [0, 3]]      # only j = 1..3 are eligible
    assert ctl.surplus == 1


def test_capacity_guard_skips_probe():
    lens, tags = _many_pairs()
    ctl = oc.Controller(oc.Config(a_max=10))
    assert len(ctl.demotion(50, 11, tags, lens)) == 0   # F > A_max: no probe
    assert len(ctl.demotion(50, 10, tags, lens)) == 40  # F = A_max: probe, Delta = 40


def test_watermark_policy():
    lens, tags = _many_pairs()
    ctl = oc.Controller(oc.Config(policy=oc.WATERMARK, watermark=30, min_batch=4))
    d = ctl.demotion(0, 20, tags, lens)                 # no shortage, below the mark by 10
    assert len(d) == 10 and ctl.shortage == 0 and ctl.surplus == 10
    assert len(ctl.demotion(100, 30, tags, lens)) == 0  # at the mark: nothing, shortage or not


def test_eager_and_no_promotion():
    lens, tags = _many_pairs()
    for eager, expect in ((False, 0), (True, 5)):
        ctl = oc.Controller(oc.Config(min_batch=16, eager=eager))
        d = ctl.demotion(1, 0, tags.copy(), lens)
        t2 = tags.copy()
        _apply(t2, d, 1)
        p = ctl.promotion(5, 100, t2, lens)               # R = 15 >= F_post = 5
        assert len(p) == expect
    ctl = oc.Controller(oc.Config(no_promotion=True))
    t2 = tags.copy()
    _apply(t2, [(0, 3)], 1)
    assert len(ctl.promotion(50, 50, t2, lens)) == 0


def test_slack_limits_promotions():
    lens, tags = _many_pairs()
    _apply(tags, [(s, j) for s in range(4) for j in range(10)], 1)
    ctl = oc.Controller(oc.Config())
    p = ctl.promotion(30, 7, tags, lens)
    assert len(p) == 7
    assert p.tolist() == [[0, 9], [1, 9], [2, 9], [3, 9], [0, 8], [1, 8], [2, 8]]


@given(st.data())
@settings(max_examples=80, deadline=None)
def test_invariants_and_structure(data):
    """Random demand / free sequences: demoted pairs are distinct eligible
    TARGET pairs, n_d follows the formula, promoted pairs are BASE and at
    most min(P_t, slack); and with the rank orders every sequence's BASE
    pairs stay one run right after its sink, so lowering stays structured."""
    nseq = data.draw(st.integers(1, 4))
    lens = np.array(data.draw(st.lists(st.integers(0, 640), min_size=nseq, max_size=nseq)), dtype=np.int32)
    sink = data.draw(st.integers(0, 2))
    recent = data.draw(st.integers(0, 2))
    cfg = oc.Config(min_batch=data.draw(st.integers(1, 8)), decay=data.draw(st.integers(0, 3)),
                    sink_pairs=sink, recent_pairs=recent)
    ctl = oc.Controller(cfg)
    tags = np.zeros((nseq, 42), dtype=np.uint8)
    for _ in range(data.draw(st.integers(1, 8))):
        demand = data.draw(st.integers(0, 12))
        free = data.draw(st.integers(0, 12))
        before = tags.copy()
        cand = oc.eligible_target_pairs(before, lens, cfg)
        d = ctl.demotion(demand, free, tags, lens)
        delta = max(0, demand - free)
        if delta == 0:
            assert len(d) == 0
        else:
            assert len(d) == min(len(cand), max(delta, cfg.min_batch))
            assert ctl.surplus == max(0, len(d) - delta)
        assert len({(int(s), int(j)) for s, j in d}) == len(d)
        for s, j in d:
            assert before[s, 2 * j] == 0 and before[s, 2 * j + 1] == 0
            assert sink <= j < lens[s] // 32 - recent
        _apply(tags, d, 1)
        slack = data.draw(st.integers(0, 6))
        free_post = data.draw(st.integers(0, 12))
        p = ctl.promotion(free_post, slack, tags, lens)
        assert len(p) <= min(ctl.budget, slack)
        for s, j in p:
            assert tags[s, 2 * j] == 1 and tags[s, 2 * j + 1] == 1
        _apply(tags, p, 0)
        mode, bounds = olow.lower(tags, lens, PAGE)
        assert mode in (olow.NATIVE, olow.STRUCTURED)
        for s in range(nseq):
            b0, b1 = bounds[s]
            if b1 > b0:
                assert b0 == sink
