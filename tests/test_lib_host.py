"""Host-side tests of libekv that need no GPU: the library loads and exports
every function include/ekv.h declares; host lowering and transition-list
validation agree with the oracle; argument errors are reported before any
device work; the host block-state mirror keeps the free pool exact."""

import ctypes
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import lowering as olow
from oracle import transitions as otr
from paper_2609_33536_amd import ekv, kvpool, workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "ekv.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ekv_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from __graft_entry__ import _ensure_built
    _ensure_built()
    return ekv.lib()


def test_library_exports_every_declared_function(lib):
    names = _declared_functions()
    assert len(names) >= 11
    for name in names:
        assert isinstance(getattr(lib, name), ctypes._CFuncPtr), name
    assert set(names) == set(ekv.SIGNATURES), "binding and header disagree"


@settings(max_examples=200, deadline=None)
@given(st.lists(st.tuples(st.integers(0, 200), st.lists(st.integers(0, 1), min_size=7, max_size=7)),
                min_size=1, max_size=5))
def test_lower_matches_oracle(rows):
    max_blocks = 14
    tags = np.zeros((len(rows), max_blocks), dtype=np.uint8)
    lens = np.zeros(len(rows), dtype=np.int32)
    for s, (length, modes) in enumerate(rows):
        lens[s] = length
        for j, m in enumerate(modes):
            tags[s, 2 * j] = tags[s, 2 * j + 1] = m
    mode, bounds = ekv.lower(tags, lens)
    omode, obounds = olow.lower(tags, lens, 16)
    assert mode == omode
    assert np.array_equal(bounds, obounds)


@settings(max_examples=300, deadline=None)
@given(st.integers(0, 2**31 - 1), st.integers(1, 6), st.sampled_from([0.0, 0.02, 0.5, 0.98, 1.0]),
       st.integers(0, 3))
def test_lower_long_rows_match_oracle(seed, bsz, p_base, planted):
    """Rows of 96 blocks (the library scans four pairs at a time): random and
    clustered BASE pairs, lengths anywhere in the row, and now and then a
    planted bad tag value or mixed pair, which both sides must reject."""
    rng = np.random.default_rng(seed)
    max_blocks = 96
    lens = rng.integers(0, max_blocks * 16 + 1, size=bsz).astype(np.int32)
    tags = np.zeros((bsz, max_blocks), dtype=np.uint8)
    for s in range(bsz):
        if rng.random() < 0.5:
            pair = (rng.random(max_blocks // 2) < p_base).astype(np.uint8)
        else:
            a, b = sorted(rng.integers(0, max_blocks // 2 + 1, size=2))
            pair = np.zeros(max_blocks // 2, dtype=np.uint8)
            pair[a:b] = 1
        tags[s] = np.repeat(pair, 2)
    for _ in range(planted):
        s, i = int(rng.integers(0, bsz)), int(rng.integers(0, max_blocks))
        tags[s, i] = int(rng.integers(0, 3))
    # the library also refuses a visible tag value above 1 (the oracle reads any nonzero tag as BASE)
    bad_value = any((tags[s, :-(-int(lens[s]) // 16)] > 1).any() for s in range(bsz))
    try:
        omode, obounds = olow.lower(tags, lens, 16)
    except olow.InvalidTags:
        bad_value = True
    if bad_value:
        with pytest.raises(ekv.EkvError):
            ekv.lower(tags, lens)
        return
    mode, bounds = ekv.lower(tags, lens)
    assert mode == omode
    assert np.array_equal(bounds, obounds)


def test_lower_rejects_mixed_pair():
    tags = np.zeros((1, 4), dtype=np.uint8)
    tags[0, 0] = 1
    with pytest.raises(ekv.EkvError):
        ekv.lower(tags, np.array([64]))


def _case(seed):
    return workloads.make_decode_case([64, 96, 33, 128, 0], 4, 2, seed=seed, base_fraction=0.5,
                                      spare_blocks=6)


@pytest.mark.parametrize("seed", range(6))
def test_check_transition_matches_oracle(seed):
    c = _case(seed)
    rng = np.random.default_rng(seed)
    nb = c["pool"].shape[0]
    bt, tags, lens = c["block_table"], c["tags"], c["seq_lens"]
    cands = [c["pairs"],
             np.vstack([c["pairs"], c["pairs"][:1]]),                  # duplicate
             np.array([[2, 1]], np.int32),                             # 33 tokens: pair 1 partial
             np.array([[4, 0]], np.int32),                             # empty sequence
             np.array([[7, 0]], np.int32),                             # sequence out of range
             rng.integers(0, 4, size=(3, 2)).astype(np.int32)]
    for pairs in cands:
        try:
            otr.check_pairs(pairs, bt, tags, lens, 16, 0)
            expect = True
        except otr.InvalidTransition:
            expect = False
        ok, msg = ekv.check_transition(0, pairs, bt, tags, lens, nb)
        assert ok == expect, (pairs, msg)
    # refinement: TARGET pairs are rejected, BASE pairs with free new blocks accepted
    ok, _ = ekv.check_transition(1, c["pairs"], bt, tags, lens, nb, c["free"][:len(c["pairs"])])
    assert not ok
    _, bt2, tg2, freed, _ = otr.demote(c["pool"], bt, tags, c["pairs"], lens)
    ok, msg = ekv.check_transition(1, c["pairs"], bt2, tg2, lens, nb, freed)
    assert ok, msg
    ok, _ = ekv.check_transition(1, c["pairs"], bt2, tg2, lens, nb, bt2[0, :len(c["pairs"])])  # in use
    assert not ok


def test_argument_errors_before_device_work(lib):
    pool = ekv.Pool(None, 10, 2, 16, 128, 0)
    batch = ekv.Batch(1, 8, 4, 0, 0, None, None, None, None)
    st_ = lib.ekv_attn_decode(ctypes.byref(pool), ctypes.byref(batch), None, None, 0, 1.0, None, 0, None)
    assert st_ == ekv.ERR_INVALID and b"NULL" in lib.ekv_last_error()
    pool = ekv.Pool(1, 10, 2, 16, 64, 0)
    assert lib.ekv_attn_decode(ctypes.byref(pool), ctypes.byref(batch), None, None, 0, 1.0, None, 0,
                               None) == ekv.ERR_UNSUPPORTED
    pool = ekv.Pool(1, 10, 2, 16, 128, 0)
    batch = ekv.Batch(1, 6, 4, 0, 0, 1, 1, None, None)     # group 3
    assert lib.ekv_attn_decode(ctypes.byref(pool), ctypes.byref(batch), 1, 1, 0, 1.0, 1, 1 << 30,
                               None) == ekv.ERR_UNSUPPORTED
    batch = ekv.Batch(1, 8, 4, ekv.MODE_GENERAL, 0, 1, 1, None, None)   # general without tags
    assert lib.ekv_attn_decode(ctypes.byref(pool), ctypes.byref(batch), 1, 1, 0, 1.0, 1, 1 << 30,
                               None) == ekv.ERR_INVALID
    batch = ekv.Batch(1, 8, 4, 0, 0, 1, 1, None, None)
    need = lib.ekv_decode_workspace_bytes(ctypes.byref(pool), ctypes.byref(batch))
    assert need > 0
    assert lib.ekv_attn_decode(ctypes.byref(pool), ctypes.byref(batch), 1, 1, 0, 1.0, 1, need - 1,
                               None) == ekv.ERR_INVALID
    # the workspace's partial rows move in 16-byte accesses: a misaligned ws is refused
    st_ = lib.ekv_attn_decode(ctypes.byref(pool), ctypes.byref(batch), 1, 1, 0, 1.0, 0x1008, need, None)
    assert st_ == ekv.ERR_INVALID and b"aligned" in lib.ekv_last_error()
    assert lib.ekv_demote(ctypes.byref(pool), 1, None, None, None, 1, 4, None, None, None) == ekv.ERR_INVALID
    assert lib.ekv_refine(ctypes.byref(pool), 1, 1, None, 1, 1, 1, 4, None, None) == ekv.ERR_INVALID


def test_host_mirror_commit_after_completion_and_fifo():
    c = _case(1)
    nb = c["pool"].shape[0]
    m = kvpool.HostMirror(c["block_table"], c["seq_lens"], nb, c["free"])
    free0 = list(m.free)
    freed = m.plan_demote(c["pairs"])
    # nothing returns to the pool before the caller commits
    assert list(m.free) == free0
    _, obt, otg, ofreed, _ = otr.demote(c["pool"], c["block_table"], c["tags"], c["pairs"], c["seq_lens"])
    assert np.array_equal(freed, ofreed) and np.array_equal(m.bt, obt) and np.array_equal(m.tags, otg)
    m.commit_freed(freed)
    ofifo = otr.FreeFifo(c["free"])
    ofifo.commit_freed(ofreed)
    assert list(m.free) == ofifo.snapshot().tolist()
    sel = c["pairs"][:2]
    new = m.plan_refine(sel)
    assert new.tolist() == ofifo.acquire(2).tolist()
    # a rejected refinement leaves the free pool exactly as it was
    before = list(m.free)
    with pytest.raises(ekv.EkvError):
        m.plan_refine(sel)                       # already TARGET again
    assert list(m.free) == before
