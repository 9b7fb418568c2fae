"""Pins of the 8-bit TARGET / 4-bit BASE oracle (reading of App. C.5's
generalisation): the E5M2 decoding against torch's float8_e5m2 for all 256
codes, the closed form of the BASE values, exact refinement for every
byte, a hand-packed nibble row, the paged gather against a dense copy, the
transition round trip on a whole pool, attention against SDPA (f = 0)
and against the truncated pool (f = 1), and chunked prefill against causal
SDPA and, with BASE pairs, against the truncated pool."""

import numpy as np
import torch

from oracle import fp8
from paper_2609_33536_amd import workloads

PAGE = 16
ALL = np.arange(256, dtype=np.uint8)


def test_e5m2_decoding_matches_torch_for_every_code():
    ref = torch.from_numpy(ALL.copy()).view(torch.float8_e5m2).to(torch.float64).numpy()
    got = fp8.bytes_to_f64(ALL)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok])


def test_base_values_closed_form_and_exact_refinement():
    x = fp8.bytes_to_f64(ALL)
    base = fp8.bytes_to_f64(fp8.base_byte(fp8.hi_nibble(ALL)))
    # sign and the top three exponent bits: 0 or +-2^(4k - 15), k = 1..7
    mags = {0.0} | {2.0 ** (4 * k - 15) for k in range(1, 8)}
    assert set(np.abs(base).tolist()) == mags
    assert np.array_equal(np.signbit(base), np.signbit(x))
    fin = np.isfinite(x)
    assert (np.abs(base[fin]) <= np.abs(x[fin])).all()
    assert np.array_equal(fp8.refine_byte(fp8.hi_nibble(ALL), fp8.lo_nibble(ALL)), ALL)


def test_nibble_packing_by_hand():
    row = np.array([1, 2, 3, 4, 0xF, 0], dtype=np.uint8)
    assert fp8.pack_nibbles(row).tolist() == [0x21, 0x43, 0x0F]
    assert np.array_equal(fp8.unpack_nibbles(fp8.pack_nibbles(row)), row)


def _pool(nb, hkv, seed):
    rng = np.random.default_rng(seed)
    return rng.integers(0, 256, size=(nb, 2, hkv, PAGE, 128), dtype=np.uint8)


def test_gather_matches_dense_copy_and_base_reads_packed_member():
    pool = _pool(12, 2, 1)
    bt = np.array([[3, 7, 1, 0, 9]], dtype=np.int32)
    tags = np.zeros((1, 5), dtype=np.uint8)
    k, v = fp8.gather_sequence(pool, bt[0], tags[0], 70)
    dense = np.concatenate([pool[b] for b in bt[0]], axis=2)[:, :, :70]      # [2][Hkv][70][d]
    vals = fp8.bytes_to_f64(dense)
    np.testing.assert_array_equal(k, vals[0].transpose(1, 0, 2))
    np.testing.assert_array_equal(v, vals[1].transpose(1, 0, 2))
    # demote pair 0: block 3 holds both members' nibbles, and BASE reads the high nibbles
    p2, bt2, tg2, freed, lo = fp8.demote(pool, bt, tags, [(0, 0)], [70])
    assert freed.tolist() == [7] and bt2[0, :2].tolist() == [3, 3]
    assert np.array_equal(p2[7], pool[7])                    # the freed block is untouched
    k2, _ = fp8.gather_sequence(p2, bt2[0], tg2[0], 70)
    want = fp8.bytes_to_f64(pool[7, 0] & 0xF0).transpose(1, 0, 2)   # member 1 = tokens 16..31
    np.testing.assert_array_equal(k2[16:32], want)


def test_round_trip_restores_every_visible_byte():
    lens = [300, 64, 1000, 33]
    hkv = 2
    nblk = [-(-l // PAGE) for l in lens]
    nb = sum(nblk) + 6
    pool = _pool(nb, hkv, 2)
    perm = np.random.default_rng(3).permutation(nb).astype(np.int32)
    bt = np.zeros((4, 64), dtype=np.int32)
    pos = 0
    for s, n in enumerate(nblk):
        bt[s, :n] = perm[pos:pos + n]
        pos += n
    free = sorted(perm[pos:].tolist())
    tags = np.zeros_like(bt, dtype=np.uint8)
    pairs = workloads.choose_pairs(np.random.default_rng(4), np.array(lens), 0.7, "random")
    p2, bt2, tg2, freed, lo = fp8.demote(pool, bt, tags, pairs, lens)
    assert lo.shape[1:] == (2, hkv, 2, PAGE, 64) and lo[0].size == pool[0].size   # one block per pair
    new = np.array((free + freed.tolist())[:len(pairs)], dtype=np.int32)
    p3, bt3, tg3 = fp8.refine(p2, bt2, tg2, pairs, new, lo, lens)
    assert int(tg3.sum()) == 0
    for s, n in enumerate(nblk):
        for i in range(n):
            assert np.array_equal(p3[bt3[s, i]], pool[bt[s, i]]), (s, i)


def test_attention_f0_matches_sdpa_and_f1_matches_truncated_pool():
    lens = [70, 256, 129]
    hq, hkv = 8, 2
    rng = np.random.default_rng(5)
    pool = fp8.base_byte(rng.integers(0, 16, size=(48, 2, hkv, PAGE, 128), dtype=np.uint8)) | \
        rng.integers(0, 16, size=(48, 2, hkv, PAGE, 128), dtype=np.uint8)
    pool = np.where((pool & 0x7C) == 0x7C, pool & 0xBF, pool).astype(np.uint8)    # no Inf/NaN codes
    bt = np.arange(48, dtype=np.int32).reshape(3, 16)
    tags = np.zeros((3, 16), dtype=np.uint8)
    q = (rng.standard_normal((3, hq, 128)).astype(np.float16)).view(np.uint16)
    out = fp8.decode(q, pool, bt, tags, lens)
    for s, length in enumerate(lens):
        k, v = fp8.gather_sequence(pool, bt[s], tags[s], length)
        qs = torch.from_numpy(q[s].view(np.float16).astype(np.float64))[None, :, None, :]
        kk = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(hq // hkv, 0)[None]
        vv = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(hq // hkv, 0)[None]
        ref = torch.nn.functional.scaled_dot_product_attention(qs, kk, vv)[0, :, 0].numpy()
        np.testing.assert_allclose(out[s], ref, rtol=1e-12, atol=1e-12)
    pairs = np.array([(s, j) for s in range(3) for j in range(lens[s] // 32)], dtype=np.int32)
    p2, bt2, tg2, _, _ = fp8.demote(pool, bt, tags, pairs, lens)
    trunc = pool.copy()
    for s, j in pairs:
        for m in range(2):
            trunc[bt[s, 2 * j + m]] &= 0xF0
    np.testing.assert_allclose(fp8.decode(q, p2, bt2, tg2, lens), fp8.decode(q, trunc, bt, tags, lens),
                               rtol=0, atol=0)


def test_prefill_matches_causal_sdpa_and_base_pairs_match_the_truncated_pool():
    """Chunk row i of a sequence with context L and chunk n sees keys
    0 .. L - n + i: against SDPA with that mask on the dense values, and,
    with BASE pairs, equal to the same prefill over the pool whose BASE
    members hold their truncated bytes."""
    prefix, chunk = [40, 200, 3], [9, 56, 30]
    lens = [p + c for p, c in zip(prefix, chunk)]
    hq, hkv = 8, 2
    rng = np.random.default_rng(6)
    pool = rng.integers(0, 256, size=(48, 2, hkv, PAGE, 128), dtype=np.uint8)
    pool = np.where((pool & 0x7C) == 0x7C, pool & 0xBF, pool).astype(np.uint8)    # no Inf/NaN codes
    bt = np.arange(48, dtype=np.int32).reshape(3, 16)
    tags = np.zeros((3, 16), dtype=np.uint8)
    cu = np.concatenate([[0], np.cumsum(chunk)]).astype(np.int32)
    q = (rng.standard_normal((int(cu[-1]), hq, 128)).astype(np.float16)).view(np.uint16)
    out = fp8.prefill(q, cu, pool, bt, tags, lens)
    for s, (length, n) in enumerate(zip(lens, chunk)):
        k, v = fp8.gather_sequence(pool, bt[s], tags[s], length)
        qs = torch.from_numpy(q[cu[s]:cu[s + 1]].view(np.float16).astype(np.float64)).permute(1, 0, 2)[None]
        kk = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(hq // hkv, 0)[None]
        vv = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(hq // hkv, 0)[None]
        mask = torch.arange(length)[None, :] <= (length - n + torch.arange(n))[:, None]
        ref = torch.nn.functional.scaled_dot_product_attention(qs, kk, vv, attn_mask=mask)[0].permute(1, 0, 2)
        np.testing.assert_allclose(out[cu[s]:cu[s + 1]], ref.numpy(), rtol=1e-12, atol=1e-12)
    pairs = np.array([(s, j) for s in range(3) for j in range(prefix[s] // 32) if j % 2 == 0], dtype=np.int32)
    assert len(pairs) > 0
    p2, bt2, tg2, _, _ = fp8.demote(pool, bt, tags, pairs, lens)
    trunc = pool.copy()
    for s, j in pairs:
        for m in range(2):
            trunc[bt[s, 2 * j + m]] &= 0xF0
    np.testing.assert_allclose(fp8.prefill(q, cu, p2, bt2, tg2, lens), fp8.prefill(q, cu, trunc, bt, tags, lens),
                               rtol=0, atol=0)


def test_append_places_rows_by_flat_index():
    """New TARGET rows land where plain index arithmetic on the flattened pool
    says: byte (((blk * 2 + plane) * Hkv + h) * page + off) * d + c, with
    blk = slot // page and off = slot % page; K goes to plane 0, V to plane 1,
    and every other byte keeps its value (the 8-bit reading of §3.2: new KV
    enters as TARGET)."""
    nb, hkv, d = 6, 3, 128
    rng = np.random.default_rng(11)
    pool = rng.integers(0, 256, size=(nb, 2, hkv, PAGE, d), dtype=np.uint8)
    slots = np.array([0, 17, 95, 40, 41, 63], dtype=np.int32)     # blocks 0, 1, 5, 2, 2, 3
    n = len(slots)
    # K bytes even, V bytes odd, so a swapped plane cannot match by chance
    k_new = (2 * rng.integers(0, 128, size=(n, hkv, d))).astype(np.uint8)
    v_new = (2 * rng.integers(0, 128, size=(n, hkv, d)) + 1).astype(np.uint8)
    got = fp8.append(pool, slots, k_new, v_new).reshape(-1)
    want = pool.reshape(-1).copy()
    for i in range(n):
        blk, off = int(slots[i]) // PAGE, int(slots[i]) % PAGE
        for plane, rows in ((0, k_new), (1, v_new)):
            for h in range(hkv):
                base = (((blk * 2 + plane) * hkv + h) * PAGE + off) * d
                want[base:base + d] = rows[i, h]
    assert np.array_equal(got, want)
    # the input pool is not modified
    assert not np.shares_memory(got, pool)


def test_append_then_gather_reads_the_new_tokens():
    """A sequence whose last tokens were appended reads them back through the
    (separately pinned) paged gather, decoded as E5M2."""
    nb, hkv = 5, 2
    pool = _pool(nb, hkv, 4)
    bt = np.array([[4, 1, 3]], dtype=np.int32)
    length = 40
    tokens = np.arange(30, 40)
    slots = np.array([bt[0, t // PAGE] * PAGE + t % PAGE for t in tokens], dtype=np.int32)
    rng = np.random.default_rng(5)
    k_new = rng.integers(0, 256, size=(len(tokens), hkv, 128), dtype=np.uint8)
    v_new = rng.integers(0, 256, size=(len(tokens), hkv, 128), dtype=np.uint8)
    p2 = fp8.append(pool, slots, k_new, v_new)
    k, v = fp8.gather_sequence(p2, bt[0], np.zeros(3, dtype=np.uint8), length)
    kk, vv = fp8.bytes_to_f64(k_new), fp8.bytes_to_f64(v_new)
    np.testing.assert_array_equal(k[30:40], kk)
    np.testing.assert_array_equal(v[30:40], vv)
    k0, v0 = fp8.gather_sequence(pool, bt[0], np.zeros(3, dtype=np.uint8), 30)
    np.testing.assert_array_equal(k[:30], k0)
    np.testing.assert_array_equal(v[:30], v0)
