"""Pins for oracle.transitions: invariants the paper states, checked directly.

* refine(demote(x)) restores the whole pool bit for bit (§3; App. B.2);
* demotion frees exactly one block per pair and refinement reacquires one
  (§3.1), with the free pool conserved;
* every packed byte is the high byte of the word it came from, every emitted
  refinement byte its low byte (indices checked by plain loops here);
* the freed block's bytes and every other block are untouched;
* the block table stays a valid mapping: each used block is referenced by
  one TARGET logical block or by both members of one BASE pair;
* invalid lists are rejected.
"""

import numpy as np
import pytest

from oracle import paged, transitions
from paper_2609_33536_amd import workloads


def _case(seed=0, fraction=0.5, lens=(64, 96, 33, 128), hkv=2, spare=6):
    return workloads.make_decode_case(list(lens), 2 * hkv, hkv, seed=seed, base_fraction=fraction,
                                      spare_blocks=spare, head_dim=16, page=4)


def _check_mapping(bt, tags, seq_lens, nb, page, free_ids):
    refs = {}
    for s, length in enumerate(seq_lens):
        nblk = -(-int(length) // page)
        for i in range(nblk):
            refs.setdefault(int(bt[s, i]), []).append((s, i, int(tags[s, i])))
    for blk, users in refs.items():
        if len(users) == 1:
            assert users[0][2] == paged.TARGET
        else:
            assert len(users) == 2
            (s0, i0, t0), (s1, i1, t1) = sorted(users)
            assert s0 == s1 and i0 % 2 == 0 and i1 == i0 + 1 and t0 == t1 == paged.BASE
    used = set(refs)
    assert used.isdisjoint(set(int(b) for b in free_ids))
    assert len(used) + len(free_ids) == nb


def test_round_trip_restores_every_byte():
    c = _case()
    fifo = transitions.FreeFifo(c["free"])
    pool, bt, tg, freed, lo = transitions.demote(c["pool"], c["block_table"], c["tags"], c["pairs"],
                                                 c["seq_lens"])
    fifo.commit_freed(freed)
    new = fifo.acquire(len(c["pairs"]))
    pool2, bt2, tg2 = transitions.refine(pool, bt, tg, c["pairs"], new, lo, c["seq_lens"])
    # member-1 data now lives in the reacquired blocks; compare logically
    for s, length in enumerate(c["seq_lens"]):
        for i in range(-(-int(length) // 4)):
            a = c["pool"][c["block_table"][s, i]]
            b = pool2[bt2[s, i]]
            assert np.array_equal(a, b)
    assert not tg2.any()
    # when each freed block is reacquired by its own pair, the pool is identical
    pool3, bt3, tg3 = transitions.refine(pool, bt, tg, c["pairs"], freed, lo, c["seq_lens"])
    assert np.array_equal(pool3, c["pool"]) and np.array_equal(bt3, c["block_table"])


def test_demote_bytes_and_bookkeeping():
    c = _case(seed=3)
    pool0, bt0 = c["pool"], c["block_table"]
    pool, bt, tg, freed, lo = transitions.demote(pool0, bt0, c["tags"], c["pairs"], c["seq_lens"])
    n = len(c["pairs"])
    assert n > 0 and len(freed) == n == len(set(freed.tolist()))
    nb, planes, hkv, page, d = pool0.shape
    touched = set()
    for i, (s, j) in enumerate(c["pairs"]):
        b0, b1 = int(bt0[s, 2 * j]), int(bt0[s, 2 * j + 1])
        assert freed[i] == b1 and bt[s, 2 * j] == b0 and bt[s, 2 * j + 1] == b0
        assert tg[s, 2 * j] == tg[s, 2 * j + 1] == 1
        raw = pool[b0].tobytes()
        for pl in range(planes):
            for h in range(hkv):
                for m, src in enumerate((b0, b1)):
                    for o in range(page):
                        for c_ in range(d):
                            w = int(pool0[src, pl, h, o, c_])
                            off = (((pl * hkv + h) * 2 + m) * page + o) * d + c_
                            assert raw[off] == w // 256
                            assert lo[i, pl, h, m, o, c_] == w % 256
        touched.add(b0)
    for b in range(nb):
        if b not in touched:
            assert np.array_equal(pool[b], pool0[b])   # includes every freed block
    fifo = transitions.FreeFifo(c["free"])
    fifo.commit_freed(freed)
    _check_mapping(bt, tg, c["seq_lens"], nb, page, fifo.snapshot())
    assert len(fifo) == len(c["free"]) + n


def test_refine_reacquires_one_block_per_pair_fifo_order():
    c = _case(seed=4, fraction=1.0)
    fifo = transitions.FreeFifo(c["free"])
    head = fifo.snapshot()[:3].tolist()
    pool, bt, tg, freed, lo = transitions.demote(c["pool"], c["block_table"], c["tags"], c["pairs"],
                                                 c["seq_lens"])
    fifo.commit_freed(freed)
    sel = c["pairs"][:3]
    new = fifo.acquire(3)
    assert new.tolist() == head                       # oldest free ids first
    pool2, bt2, tg2 = transitions.refine(pool, bt, tg, sel, new, lo[:3], c["seq_lens"])
    nb, _, _, page, _ = pool.shape
    _check_mapping(bt2, tg2, c["seq_lens"], nb, page, fifo.snapshot())
    assert len(fifo) == len(c["free"]) + len(c["pairs"]) - 3


@pytest.mark.parametrize("bad", ["duplicate", "already_base", "partial", "range"])
def test_invalid_demote_lists_rejected(bad):
    c = _case(seed=5)
    pairs = c["pairs"].copy()
    bt, tg = c["block_table"], c["tags"]
    if bad == "duplicate":
        pairs = np.vstack([pairs, pairs[:1]])
    elif bad == "already_base":
        _, bt, tg, _, _ = transitions.demote(c["pool"], bt, tg, pairs[:1], c["seq_lens"])
    elif bad == "partial":
        pairs = np.array([[2, 4]], dtype=np.int32)       # seq 2 has 33 tokens: pair 4 = blocks 8, 9
    elif bad == "range":
        pairs = np.array([[9, 0]], dtype=np.int32)
    with pytest.raises(transitions.InvalidTransition):
        transitions.demote(c["pool"], bt, tg, pairs, c["seq_lens"])


def test_invalid_refine_lists_rejected():
    c = _case(seed=6)
    with pytest.raises(transitions.InvalidTransition):     # TARGET pair in a refine list
        transitions.refine(c["pool"], c["block_table"], c["tags"], c["pairs"][:1],
                           np.array([0]), np.zeros((1, 2, 2, 2, 4, 16), np.uint8), c["seq_lens"])


def test_touched_block_harness_equals_whole_pool_oracle():
    """The GPU tests run the oracle's transitions on only the blocks a list
    touches; that must give exactly what the oracle gives on the whole pool."""
    from tests.gpu_util import oracle_transition_on_touched
    c = workloads.make_decode_case([64, 130, 96, 200], 4, 2, seed=9, spare_blocks=12)
    rng = np.random.default_rng(9)
    lens, bt0 = c["seq_lens"], c["block_table"]
    tg0 = np.zeros(bt0.shape, dtype=np.uint8)
    pairs = np.array([(s, j) for s in range(4) for j in range(int(lens[s]) // 32)], dtype=np.int32)
    dp = pairs[rng.permutation(len(pairs))[:6]]
    whole = transitions.demote(c["pool"], bt0, tg0, dp, lens)
    host = c["pool"].copy()
    bt, tg, freed, lo, touched = oracle_transition_on_touched("demote", host, bt0, tg0, lens, dp)
    assert np.array_equal(host, whole[0]) and np.array_equal(bt, whole[1]) and np.array_equal(tg, whole[2])
    assert np.array_equal(freed, whole[3]) and np.array_equal(lo, whole[4])
    assert len(touched) == 2 * len(dp)
    fifo = transitions.FreeFifo(c["free"])
    fifo.commit_freed(freed)
    rp = dp[[4, 0, 2]]
    new = fifo.acquire(len(rp))
    rlo = lo[[4, 0, 2]]
    whole_r = transitions.refine(whole[0], whole[1], whole[2], rp, new, rlo, lens)
    bt2, tg2, _, _, _ = oracle_transition_on_touched("refine", host, bt, tg, lens, rp, new, rlo)
    assert np.array_equal(host, whole_r[0]) and np.array_equal(bt2, whole_r[1])
    assert np.array_equal(tg2, whole_r[2])
