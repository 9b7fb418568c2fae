"""Device-side values that point outside the arrays a call was given are
clamped or skipped, never followed: append slots past the pool, demotion
and refinement entries whose sequence is past the table or whose blocks are
past the pool, prefill query offsets past total_q.  Every out-of-range
value here points just past the end, into canary memory allocated behind
the arrays the call sees, so the canaries show any access that was not
skipped; the valid entries of the same calls are checked against the
oracle, bit for bit (attention within the usual tolerance)."""

import numpy as np
import pytest

from oracle import attention as oatt
from oracle import transitions as otr
from paper_2609_33536_amd import ekv, kvpool, workloads
from tests.gpu_util import check_attention, default_scale, host_safety_check, require_gpu, words_to_tensor

pytestmark = pytest.mark.gpu
PAGE = 16


def test_append_skips_slots_past_the_pool():
    torch = require_gpu()
    hkv, nb = 2, 6
    rng = np.random.default_rng(80)
    words = rng.integers(0, 2**16, size=(nb + 1, 2, hkv, PAGE, 128), dtype=np.uint16)   # block nb: canary
    dev = torch.from_numpy(words.view(np.int16).copy()).cuda()
    pool = ekv.make_pool(dev[:nb], hkv, "bf16")
    slots = np.array([2 * PAGE + 5, nb * PAGE + 3], dtype=np.int32)                   # the second is past the pool
    k = rng.integers(0, 2**16, size=(2, hkv, 128), dtype=np.uint16)
    v = rng.integers(0, 2**16, size=(2, hkv, 128), dtype=np.uint16)
    print("append with a slot past the pool", flush=True)
    ekv.append_kv(pool, torch.from_numpy(slots).cuda(), words_to_tensor(k, torch, "bf16"),
                  words_to_tensor(v, torch, "bf16"))
    torch.cuda.synchronize()
    got = dev.cpu().numpy().view(np.uint16)
    want = otr.append(words[:nb], slots[:1], k[:1], v[:1])
    assert np.array_equal(got[:nb], want)
    assert np.array_equal(got[nb], words[nb])                                          # canary untouched


def test_transitions_skip_entries_past_the_table_or_pool():
    torch = require_gpu()
    hkv = 2
    c = workloads.make_decode_case([128, 96], 4 * hkv, hkv, seed=81, spare_blocks=4)
    host_safety_check(c, c["pool"].shape)
    nb = c["pool"].shape[0]
    bsz, mb = c["block_table"].shape
    rng = np.random.default_rng(81)
    canary_block = rng.integers(0, 2**16, size=(1,) + c["pool"].shape[1:], dtype=np.uint16)
    pool_h = np.concatenate([c["pool"], canary_block])                                  # block nb: canary
    bt_h = np.vstack([c["block_table"], np.full((1, mb), nb, dtype=np.int32)])         # row bsz: canary
    tags_h = np.vstack([c["tags"], np.zeros((1, mb), dtype=np.uint8)])
    bt_h[1, 2] = nb                                                                     # pair (1, 1) reaches past the pool
    dev = torch.from_numpy(pool_h.view(np.int16).copy()).cuda()
    pool = ekv.make_pool(dev[:nb], hkv, "bf16")
    bt = torch.from_numpy(bt_h.copy()).cuda()
    tags = torch.from_numpy(tags_h.copy()).cuda()
    pairs = np.array([[0, 1], [bsz, 0], [1, 1], [0, 2]], dtype=np.int32)
    valid = pairs[[0, 3]]
    block_bytes = 2 * hkv * PAGE * 128 * 2
    freed = torch.empty(len(pairs), dtype=torch.int32, device="cuda")
    lo = torch.zeros((len(pairs), block_bytes), dtype=torch.uint8, device="cuda")
    print("demote with entries past the table and the pool", flush=True)
    ekv.demote(pool, torch.from_numpy(pairs).cuda(), bt[:bsz], tags[:bsz], freed, lo)
    torch.cuda.synchronize()
    opool, obt, otg, ofreed, olo = otr.demote(pool_h[:nb], bt_h[:bsz], tags_h[:bsz], valid)
    assert freed.cpu().numpy().tolist() == [int(ofreed[0]), -1, -1, int(ofreed[1])]
    got = dev.cpu().numpy().view(np.uint16)
    assert np.array_equal(got[:nb], opool) and np.array_equal(got[nb], canary_block[0])
    assert np.array_equal(bt.cpu().numpy()[:bsz], obt) and np.array_equal(bt.cpu().numpy()[bsz], bt_h[bsz])
    assert np.array_equal(tags.cpu().numpy()[:bsz], otg) and np.array_equal(tags.cpu().numpy()[bsz], tags_h[bsz])
    lo_h = lo.cpu().numpy()
    assert np.array_equal(lo_h[0].reshape(olo[0].shape), olo[0])
    assert np.array_equal(lo_h[3].reshape(olo[1].shape), olo[1])

    # refine (0, 1) into a free block; (0, 2) names a block past the pool and stays BASE
    new = np.array([int(c["free"][0]), nb], dtype=np.int32)
    lo_in = torch.stack([lo[0], lo[3]])
    print("refine with a new block past the pool", flush=True)
    ekv.refine(pool, torch.from_numpy(valid).cuda(), torch.from_numpy(new).cuda(), bt[:bsz], tags[:bsz], lo_in)
    torch.cuda.synchronize()
    rpool, rbt, rtg = otr.refine(opool, obt, otg, valid[:1], new[:1], olo[:1])
    got = dev.cpu().numpy().view(np.uint16)
    assert np.array_equal(got[:nb], rpool) and np.array_equal(got[nb], canary_block[0])
    assert np.array_equal(bt.cpu().numpy()[:bsz], rbt) and np.array_equal(tags.cpu().numpy()[:bsz], rtg)
    assert rtg[0, 4] == 1 and rtg[0, 5] == 1                                          # (0, 2) still BASE


def test_prefill_clamps_query_offsets_to_total_q():
    torch = require_gpu()
    hq, hkv = 8, 2
    c = workloads.make_prefill_case([64, 32], [20, 10], hq, hkv, seed=82, spare_blocks=2)
    host_safety_check(c, c["pool"].shape)
    kv = kvpool.PagedKV(c["pool"], c["block_table"], c["seq_lens"], c["free"], hkv)
    kv.append(torch.from_numpy(c["slots"]).cuda(), words_to_tensor(c["k_new"], torch, "bf16"),
              words_to_tensor(c["v_new"], torch, "bf16"))
    kv.relower()
    total, canary = 30, 8
    q_all = torch.zeros((total + canary, hq, 128), dtype=torch.bfloat16, device="cuda")
    q_all[:total] = words_to_tensor(c["q"], torch, "bf16")
    out_all = torch.full((total + canary, hq, 128), float("nan"), dtype=torch.float32, device="cuda")
    cu = torch.tensor([0, 20, total + 4], dtype=torch.int32, device="cuda")            # the last offset is past total_q
    print("prefill with a query offset past total_q", flush=True)
    ekv.attn_prefill(kv.pool, kv.batch(hq), q_all[:total], cu, 20, out_all[:total], default_scale())
    torch.cuda.synchronize()
    got = out_all.cpu().numpy()
    assert np.isnan(got[total:]).all()                                                  # canary rows untouched
    ref = oatt.prefill(c["q"], c["cu_q"], otr.append(c["pool"], c["slots"], c["k_new"], c["v_new"]),
                       c["block_table"], c["tags"], c["seq_lens"])
    check_attention(got[:total], ref, True)
