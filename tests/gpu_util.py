"""Helpers shared by the GPU parity tests: stage a seeded case on the GPU,
run the library through its C ABI, and run the oracle on the same inputs.
The two sides never exchange intermediate results: each side demotes the
TARGET pool itself, and only the generator's inputs are shared."""

import math

import numpy as np
import pytest

ATOL = 2e-3
RTOL_BF16_OUT = 1e-2


def require_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from __graft_entry__ import _ensure_built
    _ensure_built()
    return torch


def words_to_tensor(words, torch, dtype):
    t = torch.from_numpy(np.ascontiguousarray(words).view(np.int16)).cuda()
    return t.view(torch.bfloat16 if dtype == "bf16" else torch.float16)


def check_attention(got, ref, out_fp32):
    """fp32 output: |g - o| <= 2e-3.  16-bit output: |g - o| <= 2e-3 + 1e-2 |o|
    (the output rounding alone is up to 2^-9 |o|).  Returns (max_abs, max_rel)."""
    got = np.asarray(got, dtype=np.float64)
    err = np.abs(got - ref)
    bound = ATOL if out_fp32 else ATOL + RTOL_BF16_OUT * np.abs(ref)
    bad = err > bound
    assert not bad.any(), (f"{bad.sum()} elements out of tolerance; max abs err {err.max():.3e}; "
                           f"first at {np.argwhere(bad)[0]}")
    big = np.abs(ref) > 1e-3
    rel = float((err[big] / np.abs(ref[big])).max()) if big.any() else 0.0
    return float(err.max()), rel


def host_safety_check(case, kv_pool_words_shape):
    """Every block a kernel will touch lies inside the pool (checked before launch)."""
    nb = kv_pool_words_shape[0]
    bt, lens = case["block_table"], case["seq_lens"]
    page = 16
    assert (np.asarray(lens) <= bt.shape[1] * page).all()
    for s, length in enumerate(lens):
        nblk = -(-int(length) // page)
        assert ((bt[s, :nblk] >= 0) & (bt[s, :nblk] < nb)).all()


def default_scale():
    return 1.0 / math.sqrt(128)


def oracle_transition_on_touched(kind, host_pool, bt, tags, seq_lens, pairs, new_blocks=None, lo=None):
    """Run the oracle's demote/refine on just the blocks the list touches
    (renumbered densely), so that a multi-GB pool is never copied whole.

    Returns (bt, tags, freed, lo, touched blocks) and writes the transformed
    blocks back into ``host_pool`` (the oracle's own copy).  Equivalent to the
    oracle on the whole pool because a transition reads and writes only the
    blocks of its listed pairs (checked on the CPU against the whole-pool
    oracle)."""
    from oracle import transitions as otr
    pairs = np.asarray(pairs, dtype=np.int64).reshape(-1, 2)
    s, j = pairs[:, 0], pairs[:, 1]
    if kind == "demote":
        touched = np.concatenate([bt[s, 2 * j], bt[s, 2 * j + 1]])
    else:
        touched = np.concatenate([bt[s, 2 * j], np.asarray(new_blocks, dtype=np.int64)])
    blocks, inv = np.unique(touched, return_inverse=True)
    local = host_pool[blocks]
    lbt = np.full_like(bt, -1)
    n = len(pairs)
    if kind == "demote":
        lbt[s, 2 * j] = inv[:n]
        lbt[s, 2 * j + 1] = inv[n:]
        lpool, lbt2, tg2, lfreed, lo_out = otr.demote(local, lbt, tags, pairs, seq_lens)
        freed = blocks[lfreed].astype(np.int32)
    else:
        lbt[s, 2 * j] = inv[:n]
        lbt[s, 2 * j + 1] = inv[:n]
        lpool, lbt2, tg2 = otr.refine(local, lbt, tags, pairs, inv[n:], lo, seq_lens)
        freed, lo_out = None, None
    untouched = lbt2 == -1
    assert np.array_equal(untouched, lbt == -1)
    bt2 = bt.copy()
    bt2[~untouched] = blocks[lbt2[~untouched]]
    host_pool[blocks] = lpool
    return bt2, tg2, freed, lo_out, blocks
