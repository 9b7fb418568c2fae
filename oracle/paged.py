"""Paged KV pool with the pair-structured layout, and the logical gather (oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Pool (§2.1): a set of fixed-size physical blocks; each request maps its
logical blocks, in token order, to physical blocks through a block table.
Here a physical block holds ``page`` tokens of both K (plane 0) and V
(plane 1) for all KV heads:

    pool : uint16 [num_blocks][2][Hkv][page][d]      (raw 16-bit words)

Pairs (§3.1): two logical blocks form the smallest container whose two BASE
halves fit in one target-sized physical block.  Readings taken where the
paper is silent:

* a pair is logical blocks (2j, 2j+1) of one sequence;
* demotion keeps member 0's physical block and returns member 1's;
* inside the kept block, each plane's bytes are laid out as
  ``uint8 [Hkv][member][page][d]``: for every (plane, head) the 4 KiB a
  TARGET block uses for that head holds [BASE bytes of member 0 | BASE
  bytes of member 1];
* both members' block-table entries point at the packed block, and the
  per-block fidelity tag (0 = TARGET, 1 = BASE) is equal across a pair.

TARGET pairs keep the native layout untouched (§3.1, "native path
compatibility").
"""

import numpy as np

from . import encoding

TARGET = 0
BASE = 1


def packed_bytes(pool, block):
    """Byte view ``uint8 [2][Hkv][member][page][d]`` of one physical block
    read as a packed BASE pair (§3.1)."""
    nb, planes, hkv, page, d = pool.shape
    return pool[block].view(np.uint8).reshape(planes, hkv, 2, page, d)


def block_words(pool, bt_row, tag_row, i):
    """Executed 16-bit words ``uint16 [2][Hkv][page][d]`` of logical block ``i``.

    TARGET blocks load their native words; BASE blocks load the stored byte of
    their pair member and zero-fill the low byte (§3.2; App. B.3).
    """
    phys = int(bt_row[i])
    if phys < 0 or phys >= pool.shape[0]:
        raise IndexError(f"block table entry {phys} out of range")
    if int(tag_row[i]) == TARGET:
        return pool[phys].copy()
    member = i % 2
    return encoding.base_word(packed_bytes(pool, phys)[:, :, member])


def gather_sequence(pool, bt_row, tag_row, length, dtype):
    """Dense float64 K and V ``[length][Hkv][d]`` of one sequence, in logical
    token order (§2.1), each block decoded by its mode (§3.2)."""
    nb, planes, hkv, page, d = pool.shape
    nblk = -(-int(length) // page)
    k = np.empty((nblk * page, hkv, d), dtype=np.float64)
    v = np.empty((nblk * page, hkv, d), dtype=np.float64)
    for i in range(nblk):
        w = block_words(pool, bt_row, tag_row, i)                 # [2][Hkv][page][d]
        vals = encoding.words_to_f64(w, dtype)
        k[i * page:(i + 1) * page] = vals[0].transpose(1, 0, 2)
        v[i * page:(i + 1) * page] = vals[1].transpose(1, 0, 2)
    return k[:length], v[:length]
