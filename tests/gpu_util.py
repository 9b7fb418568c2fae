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
