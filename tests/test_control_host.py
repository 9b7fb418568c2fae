"""The library's fidelity controller (ekv_ctrl_demotion / ekv_ctrl_promotion,
host C++) against the controller oracle, step by step: the same pair lists
in the same order and the same shortage, surplus, reserve and budget.
No GPU is needed."""

import ctypes

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import control as oc
from paper_2609_33536_amd import ekv


@pytest.fixture(scope="module", autouse=True)
def _built():
    from __graft_entry__ import _ensure_built
    _ensure_built()


def _apply(tags, pairs, value):
    for s, j in pairs:
        tags[s, 2 * j] = tags[s, 2 * j + 1] = value


@given(st.data())
@settings(max_examples=150, deadline=None)
def test_controller_matches_oracle(data):
    nseq = data.draw(st.integers(1, 6))
    max_blocks = 40
    lens = np.array(data.draw(st.lists(st.integers(0, 16 * max_blocks), min_size=nseq, max_size=nseq)),
                    dtype=np.int32)
    policy = data.draw(st.sampled_from([oc.SHORTAGE, oc.WATERMARK]))
    kw = dict(min_batch=data.draw(st.integers(0, 10)), decay=data.draw(st.integers(0, 4)),
              a_max=data.draw(st.sampled_from([-1, 3, 8])), sink_pairs=data.draw(st.integers(0, 3)),
              recent_pairs=data.draw(st.integers(0, 3)), watermark=data.draw(st.integers(0, 12)),
              eager=data.draw(st.booleans()), no_promotion=data.draw(st.booleans()))
    ocfg = oc.Config(policy=policy, **kw)
    ccfg = ekv.ctrl_config(policy=policy, **kw)
    octl, cst = oc.Controller(ocfg), ekv.CtrlState()
    tags = np.zeros((nseq, max_blocks), dtype=np.uint8)
    # some BASE pairs to start with (pair-consistent, full pairs only)
    for s in range(nseq):
        for j in range(int(lens[s]) // 32):
            if data.draw(st.booleans()):
                _apply(tags, [(s, j)], 1)
    backed = None
    if data.draw(st.booleans()):
        backed = np.array(data.draw(st.lists(st.integers(0, 1), min_size=nseq * max_blocks,
                                             max_size=nseq * max_blocks)), dtype=np.uint8).reshape(nseq, -1)
    for _ in range(data.draw(st.integers(1, 6))):
        demand, free = data.draw(st.integers(0, 20)), data.draw(st.integers(0, 20))
        od = octl.demotion(demand, free, tags, lens, backed)
        cd = ekv.ctrl_demotion(ccfg, cst, demand, free, tags, lens, backed)
        assert cd.tolist() == od.tolist()
        assert (cst.shortage, cst.surplus) == (octl.shortage, octl.surplus)
        _apply(tags, cd, 1)
        free_post, slack = data.draw(st.integers(0, 20)), data.draw(st.integers(0, 8))
        op = octl.promotion(free_post, slack, tags, lens)
        cp = ekv.ctrl_promotion(ccfg, cst, free_post, slack, tags, lens)
        assert cp.tolist() == op.tolist()
        assert (cst.reserve, cst.budget) == (octl.reserve, octl.budget)
        _apply(tags, cp, 0)


def test_controller_rejects_bad_arguments():
    lens = np.array([320], dtype=np.int32)
    tags = np.zeros((1, 20), dtype=np.uint8)
    cfg, stt = ekv.ctrl_config(min_batch=4), ekv.CtrlState()
    with pytest.raises(ekv.EkvError):
        ekv.ctrl_demotion(cfg, stt, -1, 0, tags, lens)
    with pytest.raises(ekv.EkvError):
        ekv.ctrl_demotion(cfg, stt, 5, 0, tags, np.array([1000], dtype=np.int32))   # length > 20 blocks
    with pytest.raises(ekv.EkvError):
        ekv.ctrl_demotion(ekv.ctrl_config(policy=7), stt, 5, 0, tags, lens)
    # an output array too small for the chosen pairs is an error, and leaves the state alone
    out = np.zeros((2, 2), dtype=np.int32)
    n = ctypes.c_int32(0)
    before = (stt.reserve, stt.surplus, stt.shortage)
    status = ekv.lib().ekv_ctrl_demotion(ctypes.byref(cfg), ctypes.byref(stt), 5, 0,
                                         tags.ctypes.data_as(ctypes.c_void_p), lens.ctypes.data_as(ctypes.c_void_p),
                                         None, 1, 20, 16, out.ctypes.data_as(ctypes.c_void_p), 2, ctypes.byref(n))
    assert status == ekv.ERR_INVALID
    assert (stt.reserve, stt.surplus, stt.shortage) == before
