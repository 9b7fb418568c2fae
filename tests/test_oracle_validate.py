"""Pins of the metadata-invariant checks (oracle/validate.py), no GPU.

* a pool built by the oracle's own demotions satisfies every invariant in
  the modes the oracle's lowering assigns;
* hand-built tables, each breaking one rule, give hand-derived counts and
  first indices;
* the checks agree with the library's host-side checks, written separately
  in C++: ekv_lower accepts a tag table exactly when there is no length,
  tag-value or mixed-pair violation, and ekv_check_transition accepts a
  list exactly when the list checks find nothing.
"""

import numpy as np
from hypothesis import given, settings
from hypothesis import strategies as st

from oracle import lowering as olow
from oracle import transitions as otr
from oracle import validate as ov
from paper_2609_33536_amd import ekv, workloads

PAGE = 16


def _found(counts, first):
    return {k: (int(counts[k]), int(first[k])) for k in range(ov.KINDS) if counts[k]}


def _demoted_case(seed=3, fraction=0.5, placement="random"):
    c = workloads.make_decode_case([64, 300, 1024, 77, 512], 8, 2, seed=seed, base_fraction=fraction,
                                   placement=placement, spare_blocks=8)
    pool, bt, tg, _, _ = otr.demote(c["pool"], c["block_table"], c["tags"], c["pairs"], c["seq_lens"])
    return c, pool, bt, tg


def test_valid_pool_has_no_violation_in_any_mode():
    for placement in ("random", "oldest"):
        c, pool, bt, tg = _demoted_case(placement=placement)
        nb = pool.shape[0]
        mode, bounds = olow.lower(tg, c["seq_lens"], PAGE)
        assert _found(*ov.batch_violations(c["seq_lens"], bt, tg, bounds, mode, nb)) == {}
        assert _found(*ov.batch_violations(c["seq_lens"], bt, tg, None, ov.GENERAL, nb)) == {}
    # the untouched TARGET pool in native mode, with and without its tags
    assert _found(*ov.batch_violations(c["seq_lens"], c["block_table"], c["tags"], None, ov.NATIVE, nb)) == {}
    assert _found(*ov.batch_violations(c["seq_lens"], c["block_table"], None, None, ov.NATIVE, nb)) == {}


def _small():
    """2 sequences, 6-block rows, lengths 80 (5 blocks: pairs 0, 1 full, the
    lone block 4) and 40 (3 blocks: pair 0 full, block 2 partial); pair 0 of
    sequence 0 is BASE (packed into block 10)."""
    bt = np.array([[10, 10, 12, 13, 14, 99], [20, 21, 22, 99, 99, 99]], dtype=np.int32)
    tags = np.zeros((2, 6), dtype=np.uint8)
    tags[0, 0:2] = 1
    lens = np.array([80, 40], dtype=np.int32)
    bounds = np.array([[0, 1], [0, 0]], dtype=np.int32)
    return bt, tags, lens, bounds


def test_hand_built_batch_violations():
    nb = 30
    bt, tags, lens, bounds = _small()
    # valid in general and structured mode; only entries past the visible blocks hold 99
    assert _found(*ov.batch_violations(lens, bt, tags, None, ov.GENERAL, nb)) == {}
    assert _found(*ov.batch_violations(lens, bt, tags, bounds, ov.STRUCTURED, nb)) == {}
    # native mode with a BASE pair: one mode violation at pair (0, 0)
    assert _found(*ov.batch_violations(lens, bt, tags, None, ov.NATIVE, nb)) == {ov.MODE: (1, 0)}
    # sequence 1 block 1 maps outside the pool: index 1 * 6 + 1
    b2 = bt.copy()
    b2[1, 1] = nb
    assert _found(*ov.batch_violations(lens, b2, tags, None, ov.GENERAL, nb)) == {ov.BLOCK_RANGE: (1, 7)}
    # mixed pair (0, 1): block 2 BASE, block 3 TARGET; executed as BASE (member 0's
    # tag) it is two full blocks with two table entries
    t2 = tags.copy()
    t2[0, 2] = 1
    assert _found(*ov.batch_violations(lens, bt, t2, None, ov.GENERAL, nb)) == {
        ov.PAIR_MIXED: (1, 2), ov.BASE_ALIAS: (1, 2)}
    # the lone block 4 of sequence 0 tagged BASE: not two full blocks
    t3 = tags.copy()
    t3[0, 4] = 1
    assert _found(*ov.batch_violations(lens, bt, t3, None, ov.GENERAL, nb)) == {ov.BASE_PARTIAL: (1, 4)}
    # a tag value of 2 on sequence 1 block 2 (visible, lone): also executed as BASE
    t4 = tags.copy()
    t4[1, 2] = 2
    assert _found(*ov.batch_violations(lens, bt, t4, None, ov.GENERAL, nb)) == {
        ov.TAG_VALUE: (1, 8), ov.BASE_PARTIAL: (1, 8)}
    # lengths: negative, and beyond the table (clamped to 6 blocks for the rest)
    l2 = np.array([-1, 97], dtype=np.int32)
    assert _found(*ov.batch_violations(l2, bt, tags, None, ov.GENERAL, nb)) == {
        ov.SEQ_LEN: (2, 0), ov.BLOCK_RANGE: (3, 9)}
    # max_seq_len 64 makes length 80 too long, but nothing else changes
    assert _found(*ov.batch_violations(lens, bt, tags, None, ov.GENERAL, nb, max_seq_len=64)) == {
        ov.SEQ_LEN: (1, 0)}
    # boundaries that disagree with the tags: range [1, 2) on sequence 0 marks
    # pair 0 TARGET (BASE tag) and pair 1 BASE (TARGET tag, two entries)
    b3 = bounds.copy()
    b3[0] = (1, 2)
    assert _found(*ov.batch_violations(lens, bt, tags, b3, ov.STRUCTURED, nb)) == {
        ov.MODE: (2, 0), ov.BASE_ALIAS: (1, 2)}
    # an unordered range, and (-1, -1) without tags
    b4 = bounds.copy()
    b4[1] = (1, 0)
    assert _found(*ov.batch_violations(lens, bt, tags, b4, ov.STRUCTURED, nb)) == {ov.MODE: (1, 6)}
    b5 = np.array([[0, 1], [-1, -1]], dtype=np.int32)
    assert _found(*ov.batch_violations(lens, bt, None, b5, ov.STRUCTURED, nb)) == {ov.MODE: (1, 6)}


def test_pairs_ending_at_the_length_are_full():
    """Boundaries of 'two full blocks': a BASE pair ending exactly at the
    sequence length is valid, one token short is not."""
    nb = 30
    bt = np.array([[10, 10, 12, 13]], dtype=np.int32)
    tags = np.array([[1, 1, 0, 0]], dtype=np.uint8)
    assert _found(*ov.batch_violations(np.array([32]), bt, tags, None, ov.GENERAL, nb)) == {}
    assert _found(*ov.batch_violations(np.array([31]), bt, tags, None, ov.GENERAL, nb)) == {ov.BASE_PARTIAL: (1, 0)}
    tg2 = np.zeros_like(tags)
    assert _found(*ov.list_violations(0, [[0, 1]], np.array([[10, 11, 12, 13]]), tg2, nb, np.array([64]))) == {}
    assert _found(*ov.list_violations(0, [[0, 1]], np.array([[10, 11, 12, 13]]), tg2, nb, np.array([63]))) == {
        ov.LIST_PARTIAL: (1, 0)}


def test_hand_built_list_violations():
    nb = 30
    bt, tags, lens, _ = _small()
    # demotion of (0, 1) and (1, 0): valid
    assert _found(*ov.list_violations(0, [[0, 1], [1, 0]], bt, tags, nb, lens)) == {}
    # (0, 0) is already BASE; (1, 0) twice; (2, 0) and (0, 3) out of range
    found = _found(*ov.list_violations(0, [[0, 0], [1, 0], [1, 0], [2, 0], [0, 3]], bt, tags, nb, lens))
    assert found == {ov.LIST_STATE: (1, 0), ov.LIST_DUPLICATE: (1, 2), ov.LIST_RANGE: (2, 3)}
    # (0, 2): blocks 4, 5 of sequence 0, not two full blocks (and block 5 is 99)
    assert _found(*ov.list_violations(0, [[0, 2]], bt, tags, nb, lens)) == {
        ov.LIST_PARTIAL: (1, 0), ov.LIST_RANGE: (1, 0)}
    assert _found(*ov.list_violations(0, [[0, 2]], bt, tags, nb)) == {ov.LIST_RANGE: (1, 0)}
    # refinement of (0, 0) into block 25: valid; into 12 (visible in sequence
    # 0), 30 (outside), or 25 twice
    assert _found(*ov.list_violations(1, [[0, 0]], bt, tags, nb, lens, [25])) == {}
    assert _found(*ov.list_violations(1, [[0, 0]], bt, tags, nb, lens, [12])) == {ov.NEW_BLOCK: (1, 0)}
    assert _found(*ov.list_violations(1, [[0, 0]], bt, tags, nb, None, [12])) == {}
    assert _found(*ov.list_violations(1, [[0, 0]], bt, tags, nb, lens, [30])) == {ov.NEW_BLOCK: (1, 0)}
    t2 = tags.copy()
    t2[1, 0:2] = 1
    b2 = bt.copy()
    b2[1, 1] = 20
    assert _found(*ov.list_violations(1, [[0, 0], [1, 0]], b2, t2, nb, lens, [25, 25])) == {ov.NEW_BLOCK: (1, 1)}
    # a refinement of a TARGET pair; block 10 (the packed pair's, two entries) as new block
    assert _found(*ov.list_violations(1, [[0, 1]], bt, tags, nb, lens, [10])) == {
        ov.LIST_STATE: (1, 0), ov.NEW_BLOCK: (2, 0)}


@settings(max_examples=150, deadline=None)
@given(st.lists(st.tuples(st.integers(-5, 230), st.lists(st.integers(0, 2), min_size=14, max_size=14)),
                min_size=1, max_size=5))
def test_batch_checks_agree_with_host_lowering(rows):
    max_blocks = 14
    tags = np.array([r[1] for r in rows], dtype=np.uint8)
    lens = np.array([r[0] for r in rows], dtype=np.int32)
    bt = np.arange(len(rows) * max_blocks, dtype=np.int32).reshape(len(rows), max_blocks)
    counts, _ = ov.batch_violations(lens, bt, tags, None, ov.GENERAL, 10 ** 6)
    bad = counts[ov.SEQ_LEN] + counts[ov.TAG_VALUE] + counts[ov.PAIR_MIXED] > 0
    try:
        ekv.lower(tags, lens, PAGE)
        accepted = True
    except ekv.EkvError:
        accepted = False
    assert accepted == (not bad)


@settings(max_examples=150, deadline=None)
@given(st.integers(0, 1), st.lists(st.tuples(st.integers(-1, 3), st.integers(-1, 4)), min_size=1, max_size=6),
       st.lists(st.integers(-1, 44), min_size=6, max_size=6), st.integers(0, 2**31 - 1))
def test_list_checks_agree_with_host_transition_check(kind, pairs, new, seed):
    rng = np.random.default_rng(seed)
    bsz, max_blocks, nb = 3, 8, 40
    lens = rng.integers(0, max_blocks * PAGE + 1, size=bsz).astype(np.int32)
    tags = np.repeat(rng.integers(0, 2, size=(bsz, max_blocks // 2)), 2, axis=1).astype(np.uint8)
    bt = rng.integers(-1, nb + 1, size=(bsz, max_blocks)).astype(np.int32)
    pairs = np.array(pairs, dtype=np.int32).reshape(-1, 2)
    new_blocks = np.array(new[:len(pairs)], dtype=np.int32)
    counts, _ = ov.list_violations(kind, pairs, bt, tags, nb, lens, new_blocks if kind else None)
    ok, _ = ekv.check_transition(kind, pairs, bt, tags, lens, nb, new_blocks if kind else None)
    assert ok == (counts.sum() == 0)
