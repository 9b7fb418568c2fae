"""Pins for oracle.attention / oracle.paged against definitions outside them.

* brute force with pure-Python loops over a dense, un-paged copy of each
  sequence (tiny shapes), with the BASE truncation applied to the dense
  words by integer arithmetic in the test;
* torch's scaled_dot_product_attention on the CPU (a library routine);
* closed forms: a zero query gives the plain mean of V; a sequence whose
  keys are all equal does too;
* invariants: output does not depend on which physical blocks hold the
  sequence; prefill row i equals decode over the first L0+i+1 tokens.
"""

import math

import numpy as np
import pytest
import torch

from oracle import attention, transitions
from paper_2609_33536_amd import workloads


def _vals(words, dtype):
    """Test-side 16-bit -> float conversion through torch (not the oracle's)."""
    t = torch.from_numpy(np.ascontiguousarray(words).view(np.int16))
    t = t.view(torch.bfloat16 if dtype == "bf16" else torch.float16)
    return t.to(torch.float64).numpy()


def _dense_words(pool, bt_row, length, page):
    """[L][2][Hkv][d] words of one sequence, read by plain indexing."""
    out = []
    for t in range(length):
        out.append(pool[bt_row[t // page], :, :, t % page, :])
    return np.stack(out).astype(np.uint16)


def _brute_decode(q_vals, k_vals, v_vals, scale):
    """Pure-Python attention for one head: q [d], k/v [L][d]."""
    scores = [scale * sum(q_vals[c] * k_vals[t][c] for c in range(len(q_vals))) for t in range(len(k_vals))]
    m = max(scores)
    e = [math.exp(s - m) for s in scores]
    z = sum(e)
    return [sum(e[t] * v_vals[t][c] for t in range(len(k_vals))) / z for c in range(len(q_vals))]


def _truncate_pairs(dense, base_pairs_of_seq, page):
    """Zero the low byte of every word of tokens in the listed pairs (test-side)."""
    d = dense.astype(np.int64)
    for j in base_pairs_of_seq:
        lo_t, hi_t = 2 * j * page, 2 * (j + 1) * page
        d[lo_t:hi_t] = (d[lo_t:hi_t] // 256) * 256
    return d.astype(np.uint16)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("fraction", [0.0, 0.5, 1.0])
def test_decode_matches_brute_force(dtype, fraction):
    page, d = 4, 8
    case = workloads.make_decode_case([5, 16, 23, 1], 4, 2, head_dim=d, page=page, dtype=dtype,
                                      seed=11, base_fraction=fraction, spare_blocks=3)
    pool, bt, tags = case["pool"], case["block_table"], case["tags"]
    dense = [_dense_words(pool, bt[s], int(case["seq_lens"][s]), page) for s in range(4)]
    if len(case["pairs"]):
        pool, bt, tags, _, _ = transitions.demote(pool, bt, tags, case["pairs"], case["seq_lens"])
    out = attention.decode(case["q"], pool, bt, tags, case["seq_lens"], dtype)
    scale = 1 / math.sqrt(d)
    for s in range(4):
        js = [int(j) for ss, j in case["pairs"] if ss == s]
        dw = _truncate_pairs(dense[s], js, page)
        kv = _vals(dw, dtype)                         # [L][2][Hkv][d]
        qv = _vals(case["q"][s], dtype)
        for h in range(4):
            ref = _brute_decode(qv[h], kv[:, 0, h // 2], kv[:, 1, h // 2], scale)
            np.testing.assert_allclose(out[s, h], ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("group", [1, 2, 4, 8])
def test_decode_matches_torch_sdpa(group):
    hkv, page, d = 2, 16, 128
    lens = [1, 15, 16, 17, 100, 257]
    case = workloads.make_decode_case(lens, hkv * group, hkv, page=page, seed=group, spare_blocks=5)
    out = attention.decode(case["q"], case["pool"], case["block_table"], case["tags"], case["seq_lens"])
    for s, length in enumerate(lens):
        dw = _dense_words(case["pool"], case["block_table"][s], length, page)
        kv = torch.from_numpy(_vals(dw, "bf16"))          # [L][2][Hkv][d]
        k = kv[:, 0].permute(1, 0, 2).repeat_interleave(group, 0)   # [Hq][L][d]
        v = kv[:, 1].permute(1, 0, 2).repeat_interleave(group, 0)
        q = torch.from_numpy(_vals(case["q"][s], "bf16"))[:, None, :]
        ref = torch.nn.functional.scaled_dot_product_attention(q, k, v)[:, 0]
        np.testing.assert_allclose(out[s], ref.numpy(), rtol=1e-10, atol=1e-12)


def test_zero_query_gives_mean_of_values():
    page, d = 16, 128
    case = workloads.make_decode_case([37, 64], 4, 2, page=page, seed=3, base_fraction=1.0)
    pool, bt, tags, _, _ = transitions.demote(case["pool"], case["block_table"], case["tags"],
                                              case["pairs"], case["seq_lens"])
    q = np.zeros_like(case["q"])
    out = attention.decode(q, pool, bt, tags, case["seq_lens"])
    for s, length in enumerate([37, 64]):
        dw = _dense_words(case["pool"], case["block_table"][s], length, page)
        js = [int(j) for ss, j in case["pairs"] if ss == s]
        v = _vals(_truncate_pairs(dw, js, page), "bf16")[:, 1]      # [L][Hkv][d]
        for h in range(4):
            np.testing.assert_allclose(out[s, h], v[:, h // 2].mean(axis=0), rtol=1e-12, atol=1e-13)


def test_equal_keys_give_mean_of_values():
    page = 16
    case = workloads.make_decode_case([48], 2, 1, page=page, seed=5)
    pool = case["pool"].copy()
    blocks = case["block_table"][0, :3]
    pool[blocks, 0] = pool[blocks[0], 0, :, 0:1, :]       # every key = the first key
    out = attention.decode(case["q"], pool, case["block_table"], case["tags"], case["seq_lens"])
    v = _vals(_dense_words(pool, case["block_table"][0], 48, page), "bf16")[:, 1, 0]
    np.testing.assert_allclose(out[0, 0], v.mean(axis=0), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(out[0, 1], v.mean(axis=0), rtol=1e-12, atol=1e-13)


def test_output_independent_of_physical_placement():
    case = workloads.make_decode_case([100, 64, 33], 8, 2, seed=9, base_fraction=0.5, spare_blocks=4)
    pool, bt, tags, _, _ = transitions.demote(case["pool"], case["block_table"], case["tags"],
                                              case["pairs"], case["seq_lens"])
    out = attention.decode(case["q"], pool, bt, tags, case["seq_lens"])
    rng = np.random.default_rng(1)
    perm = rng.permutation(pool.shape[0])                 # new id of old block b = perm[b]
    pool2 = np.empty_like(pool)
    pool2[perm] = pool
    bt2 = perm[bt].astype(np.int32)
    out2 = attention.decode(case["q"], pool2, bt2, tags, case["seq_lens"])
    assert np.array_equal(out, out2)


@pytest.mark.parametrize("fraction", [0.0, 0.5])
def test_prefill_rows_equal_truncated_decode(fraction):
    case = workloads.make_prefill_case([40, 0, 64], [9, 20, 1], 4, 2, page=16, seed=2,
                                       base_fraction=fraction, spare_blocks=2)
    pool = transitions.append(case["pool"], case["slots"], case["k_new"], case["v_new"])
    bt, tags = case["block_table"], case["tags"]
    if len(case["pairs"]):
        pool, bt, tags, _, _ = transitions.demote(pool, bt, tags, case["pairs"], case["seq_lens"])
    out = attention.prefill(case["q"], case["cu_q"], pool, bt, tags, case["seq_lens"])
    cu = case["cu_q"]
    for s in range(3):
        first = int(case["prefix_lens"][s])
        for i in range(cu[s + 1] - cu[s]):
            row = cu[s] + i
            dec = attention.decode(case["q"][row:row + 1], pool, bt[s:s + 1], tags[s:s + 1],
                                   np.array([first + i + 1]))
            np.testing.assert_allclose(out[row], dec[0], rtol=1e-13, atol=1e-14)


def test_prefill_matches_causal_sdpa():
    group, hkv, page = 4, 2, 16
    case = workloads.make_prefill_case([0, 17], [33, 16], hkv * group, hkv, page=page, seed=4)
    pool = transitions.append(case["pool"], case["slots"], case["k_new"], case["v_new"])
    out = attention.prefill(case["q"], case["cu_q"], pool, case["block_table"], case["tags"],
                            case["seq_lens"])
    cu = case["cu_q"]
    for s in range(2):
        length = int(case["seq_lens"][s])
        n = cu[s + 1] - cu[s]
        kv = torch.from_numpy(_vals(_dense_words(pool, case["block_table"][s], length, page), "bf16"))
        k = kv[:, 0].permute(1, 0, 2).repeat_interleave(group, 0)
        v = kv[:, 1].permute(1, 0, 2).repeat_interleave(group, 0)
        q = torch.from_numpy(_vals(case["q"][cu[s]:cu[s + 1]], "bf16")).permute(1, 0, 2)
        mask = torch.arange(length)[None, :] <= (length - n + torch.arange(n))[:, None]
        ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask)
        np.testing.assert_allclose(out[cu[s]:cu[s + 1]], ref.permute(1, 0, 2).numpy(), rtol=1e-10, atol=1e-12)


def test_prefill_with_base_prefix_matches_causal_sdpa_on_truncated_words():
    """BASE pairs in the prefix with a causal chunk after them."""
    group, hkv, page = 2, 2, 16
    case = workloads.make_prefill_case([96, 64], [20, 7], hkv * group, hkv, page=page, seed=6,
                                       base_fraction=0.5)
    pool = transitions.append(case["pool"], case["slots"], case["k_new"], case["v_new"])
    dense = [_dense_words(pool, case["block_table"][s], int(case["seq_lens"][s]), page) for s in range(2)]
    assert len(case["pairs"]) >= 2
    pool, bt, tags, _, _ = transitions.demote(pool, case["block_table"], case["tags"], case["pairs"],
                                              case["seq_lens"])
    out = attention.prefill(case["q"], case["cu_q"], pool, bt, tags, case["seq_lens"])
    cu = case["cu_q"]
    for s in range(2):
        length = int(case["seq_lens"][s])
        n = cu[s + 1] - cu[s]
        js = [int(j) for ss, j in case["pairs"] if ss == s]
        kv = torch.from_numpy(_vals(_truncate_pairs(dense[s], js, page), "bf16"))
        k = kv[:, 0].permute(1, 0, 2).repeat_interleave(group, 0)
        v = kv[:, 1].permute(1, 0, 2).repeat_interleave(group, 0)
        q = torch.from_numpy(_vals(case["q"][cu[s]:cu[s + 1]], "bf16")).permute(1, 0, 2)
        mask = torch.arange(length)[None, :] <= (length - n + torch.arange(n))[:, None]
        ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask)
        np.testing.assert_allclose(out[cu[s]:cu[s + 1]], ref.permute(1, 0, 2).numpy(), rtol=1e-10, atol=1e-12)


def test_append_writes_target_rows_where_told():
    case = workloads.make_prefill_case([5], [7], 2, 1, page=4, head_dim=8, seed=8)
    pool = transitions.append(case["pool"], case["slots"], case["k_new"], case["v_new"])
    for i in range(7):
        t = 5 + i
        blk = case["block_table"][0, t // 4]
        assert np.array_equal(pool[blk, 0, :, t % 4], case["k_new"][i])
        assert np.array_equal(pool[blk, 1, :, t % 4], case["v_new"][i])
    # nothing else changed
    changed = (pool != case["pool"]).any(axis=(1, 2, 4))   # [NB][page]
    assert changed.sum() <= 7
