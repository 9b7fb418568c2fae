"""The 8-bit TARGET / 4-bit BASE instance of the mixed-fidelity contract (oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper states (App. C.5, last paragraph) that the contract does not depend
on TARGET's precision: a runtime whose TARGET is 8 bits wide can add a 4-bit
executable state the same way.  Readings taken here (the paper gives no
details):

* TARGET is an FP8 E5M2 byte: the high byte of an FP16 word, so a TARGET
  byte ``b`` is executed as the FP16 word ``b << 8`` (queries and outputs
  stay FP16, scores and softmax FP32);
* BASE keeps the high-order 4 bits of the byte (sign and the top three
  exponent bits), truncated, and is executed with a zero low nibble, i.e.
  as the FP16 word ``n << 12``; the low nibble is the refinement nibble, and
  ``(n << 4) | lo`` restores TARGET exactly;
* pool: ``uint8 [NB][2][Hkv][page][d]``; pairs, survivor block, tags, block
  table and free order as for 16-bit TARGET;
* packed BASE pair inside member 0's block: for every (plane, head) the
  2 KiB a TARGET block uses for that head hold [nibbles of member 0 | nibbles
  of member 1], each member ``[page][d / 2]`` bytes; element ``e`` of a row
  sits in byte ``e // 2``, in the low nibble when ``e`` is even;
* the refinement nibbles of a pair use the same layout and fill exactly one
  8-bit block: ``uint8 [2][Hkv][member][page][d / 2]``.

Bit operations only; values are read through FP16.
"""

import numpy as np

from . import attention

TARGET = 0
BASE = 1


def hi_nibble(b):
    return (np.asarray(b, dtype=np.uint8) >> np.uint8(4)).astype(np.uint8)


def lo_nibble(b):
    return (np.asarray(b, dtype=np.uint8) & np.uint8(0x0F)).astype(np.uint8)


def base_byte(n):
    """TARGET byte executed for a BASE nibble: nibble high, zero low nibble."""
    return (np.asarray(n, dtype=np.uint8) << np.uint8(4)).astype(np.uint8)


def refine_byte(hi, lo):
    return ((np.asarray(hi, dtype=np.uint8) << np.uint8(4)) | np.asarray(lo, dtype=np.uint8)).astype(np.uint8)


def bytes_to_f64(b):
    """Value of E5M2 bytes: the FP16 word with the byte on top (exact)."""
    w = np.asarray(b, dtype=np.uint8).astype(np.uint16) << np.uint16(8)
    with np.errstate(invalid="ignore"):
        return w.view(np.float16).astype(np.float64)


def pack_nibbles(n):
    """uint8 [..., d] nibbles -> uint8 [..., d / 2]: even elements low."""
    n = np.asarray(n, dtype=np.uint8)
    return (n[..., 0::2] | (n[..., 1::2] << np.uint8(4))).astype(np.uint8)


def unpack_nibbles(p):
    """Inverse of pack_nibbles."""
    p = np.asarray(p, dtype=np.uint8)
    out = np.empty(p.shape[:-1] + (2 * p.shape[-1],), dtype=np.uint8)
    out[..., 0::2] = p & np.uint8(0x0F)
    out[..., 1::2] = p >> np.uint8(4)
    return out


def packed_nibbles(pool, block):
    """uint8 [2][Hkv][member][page][d / 2] view of a block read as a packed BASE pair."""
    nb, planes, hkv, page, d = pool.shape
    return pool[block].reshape(planes, hkv, 2, page, d // 2)


def block_bytes(pool, bt_row, tag_row, i):
    """Executed TARGET bytes uint8 [2][Hkv][page][d] of logical block i."""
    phys = int(bt_row[i])
    if phys < 0 or phys >= pool.shape[0]:
        raise IndexError(f"block table entry {phys} out of range")
    if int(tag_row[i]) == TARGET:
        return pool[phys].copy()
    return base_byte(unpack_nibbles(packed_nibbles(pool, phys)[:, :, i % 2]))


def gather_sequence(pool, bt_row, tag_row, length):
    """Dense float64 K and V [length][Hkv][d] of one sequence."""
    nb, planes, hkv, page, d = pool.shape
    nblk = -(-int(length) // page)
    k = np.empty((nblk * page, hkv, d), dtype=np.float64)
    v = np.empty((nblk * page, hkv, d), dtype=np.float64)
    for i in range(nblk):
        vals = bytes_to_f64(block_bytes(pool, bt_row, tag_row, i))
        k[i * page:(i + 1) * page] = vals[0].transpose(1, 0, 2)
        v[i * page:(i + 1) * page] = vals[1].transpose(1, 0, 2)
    return k[:length], v[:length]


def demote(pool, block_table, tags, pairs, seq_lens=None, emit_lo=True):
    """TARGET pairs -> packed BASE nibbles in member 0's block (list order).
    Returns (pool, block_table, tags, freed, lo) as new arrays."""
    pool = np.array(pool, dtype=np.uint8, copy=True)
    bt = np.array(block_table, dtype=np.int32, copy=True)
    tg = np.array(tags, dtype=np.uint8, copy=True)
    nb, planes, hkv, page, d = pool.shape
    pairs = np.asarray(pairs, dtype=np.int64).reshape(-1, 2)
    freed = np.empty(len(pairs), dtype=np.int32)
    lo = np.empty((len(pairs), planes, hkv, 2, page, d // 2), dtype=np.uint8) if emit_lo else None
    for i, (s, j) in enumerate(pairs):
        if seq_lens is not None and 2 * page * (j + 1) > int(seq_lens[s]):
            raise ValueError(f"pair ({s},{j}) is not two full blocks")
        if tg[s, 2 * j] != TARGET or tg[s, 2 * j + 1] != TARGET:
            raise ValueError(f"pair ({s},{j}) is not TARGET")
        b0, b1 = int(bt[s, 2 * j]), int(bt[s, 2 * j + 1])
        m0, m1 = pool[b0].copy(), pool[b1].copy()
        packed = np.stack([pack_nibbles(hi_nibble(m0)), pack_nibbles(hi_nibble(m1))], axis=2)
        if lo is not None:
            lo[i] = np.stack([pack_nibbles(lo_nibble(m0)), pack_nibbles(lo_nibble(m1))], axis=2)
        pool[b0] = packed.reshape(planes, hkv, page, d)
        freed[i] = b1
        bt[s, 2 * j + 1] = b0
        tg[s, 2 * j] = tg[s, 2 * j + 1] = BASE
    return pool, bt, tg, freed, lo


def refine(pool, block_table, tags, pairs, new_blocks, lo, seq_lens=None):
    """Packed BASE pairs -> TARGET bytes: member 0 in place, member 1 into new_blocks[i]."""
    pool = np.array(pool, dtype=np.uint8, copy=True)
    bt = np.array(block_table, dtype=np.int32, copy=True)
    tg = np.array(tags, dtype=np.uint8, copy=True)
    nb, planes, hkv, page, d = pool.shape
    pairs = np.asarray(pairs, dtype=np.int64).reshape(-1, 2)
    for i, (s, j) in enumerate(pairs):
        if tg[s, 2 * j] != BASE or tg[s, 2 * j + 1] != BASE:
            raise ValueError(f"pair ({s},{j}) is not BASE")
        p = int(bt[s, 2 * j])
        hi = unpack_nibbles(packed_nibbles(pool, p))                       # [2][Hkv][m][page][d]
        lon = unpack_nibbles(np.asarray(lo[i], dtype=np.uint8).reshape(planes, hkv, 2, page, d // 2))
        full = refine_byte(hi, lon)
        pool[p] = full[:, :, 0]
        pool[int(new_blocks[i])] = full[:, :, 1]
        bt[s, 2 * j + 1] = int(new_blocks[i])
        tg[s, 2 * j] = tg[s, 2 * j + 1] = TARGET
    return pool, bt, tg


def append(pool, slots, k_new, v_new):
    """New K/V rows (uint8 [n][Hkv][d]) written as TARGET at slot phys*page+off."""
    pool = np.array(pool, dtype=np.uint8, copy=True)
    page = pool.shape[3]
    for i, slot in enumerate(np.asarray(slots, dtype=np.int64)):
        pool[int(slot) // page, 0, :, int(slot) % page, :] = k_new[i]
        pool[int(slot) // page, 1, :, int(slot) % page, :] = v_new[i]
    return pool


def decode(q_words, pool, block_table, tags, seq_lens, scale=None):
    """Decode attention over an 8-bit pool: q FP16 words uint16 [B][Hq][d];
    each sequence's K/V gathered by mode; float64 result [B][Hq][d]."""
    q = np.asarray(q_words, dtype=np.uint16).view(np.float16).astype(np.float64)
    bsz, hq, d = q.shape
    hkv = pool.shape[2]
    group = hq // hkv
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros((bsz, hq, d), dtype=np.float64)
    for s in range(bsz):
        length = int(seq_lens[s])
        if length == 0:
            continue
        k, v = gather_sequence(pool, block_table[s], tags[s], length)
        for h in range(hq):
            kh = h // group
            out[s, h] = attention._softmax_weighted(scale * (k[:, kh, :] @ q[s, h]), v[:, kh, :])
    return out


def prefill(q_words, cu_q, pool, block_table, tags, seq_lens, scale=None):
    """Chunked-prefill attention over an 8-bit pool (App. A: a chunk attends
    its cached prefix and, causally, itself): q FP16 words uint16
    [total_new][Hq][d], sequence s's rows at cu_q[s]..cu_q[s+1] with their
    K/V already appended; row i of the chunk sees keys 0 .. seq_lens[s] -
    n_s + i.  Float64 result [total_new][Hq][d]."""
    q = np.asarray(q_words, dtype=np.uint16).view(np.float16).astype(np.float64)
    total, hq, d = q.shape
    hkv = pool.shape[2]
    group = hq // hkv
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros((total, hq, d), dtype=np.float64)
    for s in range(len(seq_lens)):
        r0, r1 = int(cu_q[s]), int(cu_q[s + 1])
        n, length = r1 - r0, int(seq_lens[s])
        if n == 0:
            continue
        if n > length:
            raise ValueError("chunk longer than the sequence")
        k, v = gather_sequence(pool, block_table[s], tags[s], length)
        visible = np.arange(length)[None, :] <= (length - n + np.arange(n))[:, None]
        for h in range(hq):
            kh = h // group
            scores = np.where(visible, scale * (q[r0:r1, h] @ k[:, kh, :].T), -np.inf)
            out[r0:r1, h] = attention._softmax_weighted(scores, v[:, kh, :])
    return out
