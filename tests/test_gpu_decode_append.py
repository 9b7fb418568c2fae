"""The fused append + decode (ekv_attn_decode_append) on the GPU.

Against the two calls it replaces -- ekv_append_kv of every sequence's
newest token, then ekv_attn_decode -- bit for bit (output and the whole
pool), and against the oracle's append followed by its decode (attention
within 2e-3 absolute, fp32 output).  Ragged lengths put the newest token in
every position of a block (first, last, a lone last block, the second member
of a pair), in native, structured and general batches, for 16- and 8-bit
pools and every group size; small work ranges cut the newest token's
(sequence, KV head) into several pieces.
"""

import os

import numpy as np
import pytest

from oracle import attention as oatt
from oracle import fp8 as ofp8
from oracle import transitions as otr
from paper_2609_33536_amd import ekv, kvpool, workloads
from tests.gpu_util import check_attention, default_scale, host_safety_check, require_gpu, words_to_tensor

pytestmark = pytest.mark.gpu

PAGE = 16
LENS = [1, 15, 16, 17, 31, 32, 33, 100, 257, 511, 640, 0, 1000]


def _rows(rng, n, hkv, dtype):
    """New K / V rows [n][Hkv][128]: words of N(0, 1) values, or E5M2 bytes."""
    vals = rng.standard_normal((n, hkv, 128), dtype=np.float32)
    return workloads.to_words(vals, dtype)


def _tensor(a, torch, dtype):
    if dtype == "e5m2":
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).cuda()
    return words_to_tensor(a, torch, dtype)


def _newest_slots(bt, lens):
    return np.array([bt[s, (l - 1) // PAGE] * PAGE + (l - 1) % PAGE for s, l in enumerate(lens) if l > 0],
                    dtype=np.int32)


def _run(lens, group, dtype, fraction, placement="random", min_chunk=None, hkv=2, seed=0, keep_tail_pairs=False):
    torch = require_gpu()
    hq = hkv * group
    c = workloads.make_decode_case(lens, hq, hkv, seed=seed, base_fraction=fraction, placement=placement,
                                   spare_blocks=4, dtype=dtype)
    host_safety_check(c, c["pool"].shape)
    lens_np = np.asarray(lens, dtype=np.int32)
    pairs = c["pairs"]
    if not keep_tail_pairs and len(pairs):   # the newest token's block is TARGET (the caller's invariant)
        newest_pair = (lens_np[pairs[:, 0]] - 1) // PAGE // 2
        pairs = pairs[pairs[:, 1] != newest_pair]
    kv = kvpool.PagedKV(c["pool"], c["block_table"], c["seq_lens"], c["free"], hkv, dtype)
    if len(pairs):
        kv.demote(pairs, emit_lo=False)
        kv.commit()
    mode = kv.relower()
    rng = np.random.default_rng(seed + 7)
    k_new, v_new = _rows(rng, len(lens), hkv, dtype), _rows(rng, len(lens), hkv, dtype)
    kt, vt = _tensor(k_new, torch, dtype), _tensor(v_new, torch, dtype)
    q = words_to_tensor(c["q"], torch, workloads.query_dtype(dtype))
    bt_host = kv.mirror.bt.copy()
    live = [s for s, l in enumerate(lens) if l > 0]
    slots = _newest_slots(bt_host, lens)

    old = os.environ.get("EKV_MIN_CHUNK")
    if min_chunk:
        os.environ["EKV_MIN_CHUNK"] = str(min_chunk)
    try:
        batch = kv.batch(hq)
        ws = ekv.decode_workspace(kv.pool, batch)
        print(f"decode_append: {dtype} G={group} f={fraction} {placement} mode={mode} min_chunk={min_chunk}",
              flush=True)
        # two calls: append the newest rows, then decode
        pool_a = kv.kv.clone()
        out_a = torch.full((len(lens), hq, 128), float("nan"), dtype=torch.float32, device="cuda")
        pa = ekv.make_pool(pool_a, hkv, dtype)
        if len(live):
            idx = torch.tensor(live, dtype=torch.int64, device="cuda")
            ekv.append_kv(pa, torch.from_numpy(slots).cuda(), kt[idx].contiguous(), vt[idx].contiguous())
        ekv.attn_decode(pa, batch, q, out_a, default_scale(), ws)
        # one call
        pool_b = kv.kv.clone()
        out_b = torch.full((len(lens), hq, 128), float("nan"), dtype=torch.float32, device="cuda")
        ekv.attn_decode_append(ekv.make_pool(pool_b, hkv, dtype), batch, q, kt, vt, out_b, default_scale(), ws)
        torch.cuda.synchronize()
    finally:
        if min_chunk:
            if old is None:
                del os.environ["EKV_MIN_CHUNK"]
            else:
                os.environ["EKV_MIN_CHUNK"] = old
    got_a, got_b = out_a.cpu().numpy(), out_b.cpu().numpy()
    assert np.array_equal(got_a.view(np.uint32), got_b.view(np.uint32)), "output differs from append + decode"
    assert torch.equal(pool_a, pool_b), "pool differs from append + decode"

    # the oracle: demote, append the newest rows, decode
    mod = ofp8 if dtype == "e5m2" else otr
    opool, obt, otg = c["pool"], c["block_table"], c["tags"]
    if len(pairs):
        opool, obt, otg, _, _ = mod.demote(opool, obt, otg, pairs, c["seq_lens"])
    if len(live):
        opool = mod.append(opool, slots, k_new[live], v_new[live])
    if dtype == "e5m2":
        ref = ofp8.decode(c["q"], opool, obt, otg, c["seq_lens"], default_scale())
        assert np.array_equal(pool_b.cpu().numpy(), opool)
    else:
        ref = oatt.decode(c["q"], opool, obt, otg, c["seq_lens"], dtype, default_scale())
        assert np.array_equal(pool_b.cpu().numpy().view(np.uint16), opool)
    check_attention(got_b, ref, True)
    return mode


@pytest.mark.parametrize("fraction", [0.0, 0.5, 1.0])
@pytest.mark.parametrize("group", [1, 4, 16])
@pytest.mark.parametrize("dtype", ["bf16", "e5m2"])
def test_decode_append_equals_append_then_decode(dtype, group, fraction):
    mode = _run(LENS, group, dtype, fraction, seed=20 + group)
    assert (mode == ekv.MODE_NATIVE) == (fraction == 0)


@pytest.mark.parametrize("group", [2, 8])
def test_decode_append_fp16_and_structured(group):
    _run(LENS, group, "fp16", 0.5, placement="oldest", seed=40 + group)


@pytest.mark.parametrize("dtype", ["bf16", "e5m2"])
@pytest.mark.parametrize("min_chunk", [1, 3])
def test_decode_append_newest_token_in_a_cut_sequence(dtype, min_chunk):
    """Ranges of 1 or 3 pairs per workgroup: the newest token's (sequence,
    KV head) is one piece of several, merged by another workgroup."""
    _run([300, 1024, 77, 2000, 33], 4, dtype, 0.5, min_chunk=min_chunk, hkv=8, seed=61)


@pytest.mark.parametrize("dtype", ["e5m2", "bf16"])
def test_decode_append_many_one_block_sequences(dtype):
    """96 sequences of 1..16 tokens: every window is one lone block holding
    the newest token, so the issue side runs windows ahead of the consume
    side as far as the ring allows (for the 8-bit ring, into the buffer of
    the window being consumed); the newest token's block must still be
    written where the table says."""
    lens = [1 + (7 * i) % 16 for i in range(96)]
    _run(lens, 4, dtype, 0.0, seed=90)


def test_decode_append_leaves_a_base_tail_block_alone():
    """Lengths that are multiples of 32 with every eligible pair BASE: the
    newest token's block is BASE, so nothing is written and the decode reads
    the pool as it is (the same output as a plain decode)."""
    torch = require_gpu()
    lens, hkv, hq = [64, 96, 128], 2, 8
    c = workloads.make_decode_case(lens, hq, hkv, seed=71, base_fraction=1.0, spare_blocks=4)
    kv = kvpool.PagedKV(c["pool"], c["block_table"], c["seq_lens"], c["free"], hkv)
    kv.demote(c["pairs"], emit_lo=False)
    kv.commit()
    kv.relower()
    tags = kv.mirror.tags
    assert all(tags[s, (l - 1) // PAGE] for s, l in enumerate(lens))
    rng = np.random.default_rng(72)
    kt = words_to_tensor(_rows(rng, 3, hkv, "bf16"), torch, "bf16")
    vt = words_to_tensor(_rows(rng, 3, hkv, "bf16"), torch, "bf16")
    q = words_to_tensor(c["q"], torch, "bf16")
    batch = kv.batch(hq)
    ws = ekv.decode_workspace(kv.pool, batch)
    before = kv.kv.clone()
    out_plain = torch.empty((3, hq, 128), dtype=torch.float32, device="cuda")
    ekv.attn_decode(kv.pool, batch, q, out_plain, default_scale(), ws)
    out = torch.empty((3, hq, 128), dtype=torch.float32, device="cuda")
    ekv.attn_decode_append(kv.pool, batch, q, kt, vt, out, default_scale(), ws)
    torch.cuda.synchronize()
    assert torch.equal(kv.kv, before)
    assert torch.equal(out, out_plain)


def test_decode_append_rejects_missing_rows():
    torch = require_gpu()
    c = workloads.make_decode_case([40], 4, 2, seed=80)
    kv = kvpool.PagedKV(c["pool"], c["block_table"], c["seq_lens"], c["free"], 2)
    kv.relower()
    batch = kv.batch(4)
    ws = ekv.decode_workspace(kv.pool, batch)
    q = words_to_tensor(c["q"], torch, "bf16")
    out = torch.empty((1, 4, 128), dtype=torch.float32, device="cuda")
    before = kv.kv.clone()
    with pytest.raises(ekv.EkvError) as e:
        lib = ekv.lib()
        ekv._check(lib.ekv_attn_decode_append(ekv.ctypes.byref(kv.pool), ekv.ctypes.byref(batch), ekv._ptr(q), None,
                                              None, ekv._ptr(out), ekv.dtype_code(out.dtype), default_scale(),
                                              ekv._ptr(ws), ws.numel(), None))
    assert e.value.status == ekv.ERR_INVALID
    torch.cuda.synchronize()
    assert torch.equal(kv.kv, before)
