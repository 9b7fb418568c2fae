"""Metadata invariants of the mixed-fidelity pool (oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The invariants the attention and transition steps rely on:

* §3.1: the two logical blocks (2j, 2j+1) of a pair share one fidelity; a
  BASE pair is two full blocks packed into ONE physical block, so both table
  entries of a BASE pair name that block;
* §3.2 / App. B.3: the batch mode and the per-sequence boundaries describe
  the tags (NATIVE: no visible BASE block; STRUCTURED: pairs b0 <= j < b1 are
  BASE, or (-1, -1) to read the tags);
* App. B.1: a demotion takes TARGET pairs, a refinement BASE pairs, each
  listed once; a refinement's new blocks are distinct, inside the pool and
  not used by any visible logical block.

Each function returns ``(counts, first)``: for every violation kind the
number of violations and the smallest index at which one occurs
(``NONE`` when there is none).  The kinds and their indices:

* batch checks, index ``s * max_blocks + block`` (checks of a whole
  sequence use block 0): ``SEQ_LEN``, ``BLOCK_RANGE``, ``TAG_VALUE``,
  ``PAIR_MIXED`` (at member 0), ``BASE_PARTIAL`` / ``BASE_ALIAS`` (for a pair
  the mode executes as BASE), ``MODE``;
* list checks, index = list entry: ``LIST_RANGE``, ``LIST_STATE``,
  ``LIST_PARTIAL``, ``LIST_DUPLICATE``, ``NEW_BLOCK`` (a new block out of
  range or repeated counts at its own entry; a visible table entry holding a
  new block counts once per table entry, at the new block's entry).

Which pair a mode executes as BASE (the reading of §3.2 used by the
kernels): NATIVE none; STRUCTURED with b0 >= 0 the range; otherwise the tag
of the pair's member 0.  Plain loops, no vectorisation.
"""

import numpy as np

(SEQ_LEN, BLOCK_RANGE, TAG_VALUE, PAIR_MIXED, BASE_PARTIAL, BASE_ALIAS, MODE,
 LIST_RANGE, LIST_STATE, LIST_PARTIAL, LIST_DUPLICATE, NEW_BLOCK) = range(12)
KINDS = 12
NONE = 0x7FFFFFFF

NATIVE, STRUCTURED, GENERAL = 0, 1, 2


class _Report:
    def __init__(self):
        self.counts = np.zeros(KINDS, dtype=np.int64)
        self.first = np.full(KINDS, NONE, dtype=np.int64)

    def flag(self, kind, index):
        self.counts[kind] += 1
        self.first[kind] = min(self.first[kind], index)


def full_pair(j, length, page):
    """Pair j holds two full blocks of a sequence of this length (§3.1)."""
    return 2 * page * (j + 1) <= length


def executed_as_base(mode, by_range, b0, b1, j, t0, t1):
    """Whether the attention kernels execute pair j as BASE: never in NATIVE
    mode; by the range [b0, b1) in STRUCTURED mode when the sequence has one;
    otherwise by the tag t0 of member 0 (t1 is member 1's)."""
    if mode == NATIVE:
        return False
    if by_range:
        return b0 <= j < b1
    return t0 != 0


def batch_violations(seq_lens, block_table, tags, boundaries, mode, num_blocks, max_seq_len=0, page=16):
    """Checks of a batch as the attention calls execute it.  tags and
    boundaries may be None."""
    bt = np.asarray(block_table)
    bsz, max_blocks = bt.shape
    rep = _Report()
    table_cap = max_blocks * page
    cap = min(table_cap, max_seq_len) if max_seq_len > 0 else table_cap
    for s in range(bsz):
        row0 = s * max_blocks
        raw = int(seq_lens[s])
        structured = mode == STRUCTURED and boundaries is not None
        b0, b1 = (int(boundaries[s][0]), int(boundaries[s][1])) if structured else (-1, -1)
        if raw < 0 or raw > cap:
            rep.flag(SEQ_LEN, row0)
        if structured and b0 >= 0 and b1 < b0:
            rep.flag(MODE, row0)
        if structured and b0 < 0 and tags is None:
            rep.flag(MODE, row0)
        length = max(0, min(raw, table_cap))
        nblk = -(-length // page)
        for i in range(nblk):
            idx = row0 + i
            e = int(bt[s, i])
            if e < 0 or e >= num_blocks:
                rep.flag(BLOCK_RANGE, idx)
            t = int(tags[s, i]) if tags is not None else 0
            if t > 1:
                rep.flag(TAG_VALUE, idx)
            if i % 2:
                continue
            j = i // 2
            has1 = i + 1 < nblk
            e1 = int(bt[s, i + 1]) if has1 else e
            t1 = int(tags[s, i + 1]) if (has1 and tags is not None) else t
            if has1 and t != t1:
                rep.flag(PAIR_MIXED, idx)
            by_range = structured and b0 >= 0
            exec_base = executed_as_base(mode, by_range, b0, b1, j, t, t1)
            if mode == NATIVE and (t != 0 or t1 != 0):
                rep.flag(MODE, idx)
            if mode != NATIVE and by_range and tags is not None and (t != 0) != exec_base:
                rep.flag(MODE, idx)
            if exec_base:
                if not full_pair(j, length, page):
                    rep.flag(BASE_PARTIAL, idx)
                elif e1 != e:
                    rep.flag(BASE_ALIAS, idx)
    return rep.counts, rep.first


def list_violations(kind, pairs, block_table, tags, num_blocks, seq_lens=None, new_blocks=None, page=16):
    """Checks of a demotion (kind 0) or refinement (kind 1) list."""
    bt = np.asarray(block_table)
    bsz, max_blocks = bt.shape
    pairs = np.asarray(pairs).reshape(-1, 2)
    rep = _Report()
    want = 0 if kind == 0 else 1
    use_new = kind == 1 and new_blocks is not None
    for i, (s, j) in enumerate(pairs.tolist()):
        if any(pairs[k, 0] == s and pairs[k, 1] == j for k in range(i)):
            rep.flag(LIST_DUPLICATE, i)
        if use_new:
            b = int(new_blocks[i])
            if b < 0 or b >= num_blocks or any(int(new_blocks[k]) == b for k in range(i)):
                rep.flag(NEW_BLOCK, i)
        if s < 0 or s >= bsz or j < 0 or 2 * j + 1 >= max_blocks:
            rep.flag(LIST_RANGE, i)
            continue
        e0, e1 = int(bt[s, 2 * j]), int(bt[s, 2 * j + 1])
        if not (0 <= e0 < num_blocks and 0 <= e1 < num_blocks):
            rep.flag(LIST_RANGE, i)
        if int(tags[s, 2 * j]) != want or int(tags[s, 2 * j + 1]) != want:
            rep.flag(LIST_STATE, i)
        if seq_lens is not None and not full_pair(j, int(seq_lens[s]), page):
            rep.flag(LIST_PARTIAL, i)
    if use_new and seq_lens is not None:
        for s in range(bsz):
            length = max(0, min(int(seq_lens[s]), max_blocks * page))
            for i in range(-(-length // page)):
                e = int(bt[s, i])
                hits = [k for k in range(len(pairs)) if int(new_blocks[k]) == e]
                if hits:
                    rep.flag(NEW_BLOCK, hits[0])
    return rep.counts, rep.first
