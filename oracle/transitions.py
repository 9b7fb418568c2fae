"""Fidelity transitions, append and free-block bookkeeping (oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Demotion TARGET -> BASE (§3.1; §3.4 "Transition protocols"; App. B.2): for
each selected pair the high-order bytes of its two TARGET blocks are packed
into one physical block and the other block is returned to the pool, but
only once the GPU work has completed.  Exactly one block is released per
pair.

Refinement BASE -> TARGET (§3.1; §3.3; App. B.2): one block is reacquired,
the pair is restored exactly from the stored high bytes plus the refinement
bytes, and only then is the new mapping published.

Readings where the paper is silent:

* pairs are logical blocks (2j, 2j+1) of one sequence and both must be full
  blocks (new KV is TARGET and sits in the protected recent region, §3.2);
* demotion keeps member 0's block ``bt[s][2j]`` and frees member 1's
  ``bt[s][2j+1]``, whose bytes are left as they were;
* the packed layout is the one documented in :mod:`oracle.paged`;
* the refinement bytes of one pair are exactly one block's worth, laid out
  ``uint8 [2 planes][Hkv][member][page][d]``; demotion can emit them and
  refinement consumes them (the paper keeps them as CPU backing);
* refinement writes member 0 back into the packed block in place and member
  1 into the reacquired block;
* the free pool is a FIFO: unused ids start in ascending order, blocks
  freed by a demotion batch are appended in list order after completion,
  and reacquired blocks are popped from the head in list order.

Lists are processed one pair at a time, in list order.
"""

from collections import deque

import numpy as np

from . import encoding, paged


class InvalidTransition(ValueError):
    """A transition list that violates the pair contract."""


def pair_is_complete(seq_len, j, page):
    """Both blocks of pair j hold ``page`` valid tokens."""
    return j >= 0 and 2 * page * (j + 1) <= int(seq_len)


def check_pairs(pairs, block_table, tags, seq_lens, page, want_tag):
    """Raise InvalidTransition unless every (s, j) names a distinct complete
    pair whose two tags both equal ``want_tag``."""
    seen = set()
    bsz, max_blocks = block_table.shape
    for s, j in np.asarray(pairs, dtype=np.int64).reshape(-1, 2):
        s, j = int(s), int(j)
        if not (0 <= s < bsz) or j < 0 or 2 * j + 1 >= max_blocks:
            raise InvalidTransition(f"pair ({s},{j}) out of range")
        if (s, j) in seen:
            raise InvalidTransition(f"pair ({s},{j}) listed twice")
        seen.add((s, j))
        if not pair_is_complete(seq_lens[s], j, page):
            raise InvalidTransition(f"pair ({s},{j}) is not two full blocks")
        if int(tags[s, 2 * j]) != want_tag or int(tags[s, 2 * j + 1]) != want_tag:
            raise InvalidTransition(f"pair ({s},{j}) is not in the expected state")


def demote(pool, block_table, tags, pairs, seq_lens=None, emit_lo=True):
    """Demote TARGET pairs to packed BASE.

    Returns (pool, block_table, tags, freed, lo) as new arrays:
    freed int32 [n] (member 1's old block, in list order) and lo uint8
    [n][2][Hkv][2][page][d] (refinement bytes) or None.
    """
    pool = np.array(pool, dtype=np.uint16, copy=True)
    bt = np.array(block_table, dtype=np.int32, copy=True)
    tg = np.array(tags, dtype=np.uint8, copy=True)
    nb, planes, hkv, page, d = pool.shape
    pairs = np.asarray(pairs, dtype=np.int64).reshape(-1, 2)
    if seq_lens is not None:
        check_pairs(pairs, bt, tg, seq_lens, page, paged.TARGET)
    n = len(pairs)
    freed = np.zeros(n, dtype=np.int32)
    lo = np.zeros((n, planes, hkv, 2, page, d), dtype=np.uint8) if emit_lo else None
    for i, (s, j) in enumerate(pairs):
        b0, b1 = int(bt[s, 2 * j]), int(bt[s, 2 * j + 1])
        w0, w1 = pool[b0].copy(), pool[b1].copy()           # [2][Hkv][page][d]
        packed = np.empty((planes, hkv, 2, page, d), dtype=np.uint8)
        packed[:, :, 0] = encoding.hi_byte(w0)
        packed[:, :, 1] = encoding.hi_byte(w1)
        paged.packed_bytes(pool, b0)[...] = packed
        if emit_lo:
            lo[i, :, :, 0] = encoding.lo_byte(w0)
            lo[i, :, :, 1] = encoding.lo_byte(w1)
        bt[s, 2 * j + 1] = b0
        tg[s, 2 * j] = tg[s, 2 * j + 1] = paged.BASE
        freed[i] = b1
    return pool, bt, tg, freed, lo


def refine(pool, block_table, tags, pairs, new_blocks, lo, seq_lens=None):
    """Refine BASE pairs back to TARGET exactly.

    ``new_blocks[i]`` is the block reacquired for pair i's member 1 and
    ``lo[i]`` its refinement bytes.  Returns (pool, block_table, tags).
    """
    pool = np.array(pool, dtype=np.uint16, copy=True)
    bt = np.array(block_table, dtype=np.int32, copy=True)
    tg = np.array(tags, dtype=np.uint8, copy=True)
    pairs = np.asarray(pairs, dtype=np.int64).reshape(-1, 2)
    if seq_lens is not None:
        check_pairs(pairs, bt, tg, seq_lens, pool.shape[3], paged.BASE)
    for i, (s, j) in enumerate(pairs):
        p_blk, q_blk = int(bt[s, 2 * j]), int(new_blocks[i])
        packed = paged.packed_bytes(pool, p_blk).copy()      # [2][Hkv][2][page][d]
        w0 = encoding.refine_word(packed[:, :, 0], lo[i][:, :, 0])
        w1 = encoding.refine_word(packed[:, :, 1], lo[i][:, :, 1])
        pool[p_blk] = w0
        pool[q_blk] = w1
        bt[s, 2 * j + 1] = q_blk
        tg[s, 2 * j] = tg[s, 2 * j + 1] = paged.TARGET
    return pool, bt, tg


def append(pool, slots, k_new, v_new):
    """Write new K/V rows as TARGET (§3.2; App. B.3) at slot ``phys*page+off``.

    k_new, v_new: uint16 [n][Hkv][d].  Returns the new pool.
    """
    pool = np.array(pool, dtype=np.uint16, copy=True)
    page = pool.shape[3]
    for i, slot in enumerate(np.asarray(slots, dtype=np.int64)):
        blk, off = int(slot) // page, int(slot) % page
        pool[blk, 0, :, off, :] = k_new[i]
        pool[blk, 1, :, off, :] = v_new[i]
    return pool


class FreeFifo:
    """Free-block pool: ascending initial order, FIFO reuse (reading of §3.1
    and App. B.2; the paper fixes no order)."""

    def __init__(self, free_ids):
        self.q = deque(int(b) for b in sorted(free_ids))

    def commit_freed(self, freed):
        """Return blocks to the pool after the demotion has completed."""
        self.q.extend(int(b) for b in freed)

    def acquire(self, n):
        """Reacquire ``n`` blocks for refinement, oldest first."""
        if n > len(self.q):
            raise InvalidTransition("not enough free blocks")
        return np.array([self.q.popleft() for _ in range(n)], dtype=np.int32)

    def __len__(self):
        return len(self.q)

    def snapshot(self):
        return np.array(self.q, dtype=np.int32)
