"""GPU parity at the full sizes of the decode workloads, in the launch
configuration the benchmark uses.

* Llama-3-8B-shaped decode layer: 64 sequences, 32/8 heads, context uniform
  in [2048, 8192] (seed 1), 1 % outlier channels, BASE fraction in
  {0, 0.25, 0.5, 1} with random pairs.
* Llama-3-70B-shaped decode layer: 256 sequences of 4096 tokens, 64/8 heads,
  the oldest half of every sequence's pairs BASE (structured), and the same
  batch forced down the general path; every sequence checked.
* Pressure-transition mix: a 200,000-block pool (13.1 GB), 128 sequences with
  context uniform in [1024, 16384]; every step demotes a random 10 % of the
  TARGET pairs, refines a random 5 % of the BASE pairs back, and decodes.

Attention is checked on every sequence of the 8B and 70B layers (bf16 and
fp32 output) and on 8 sampled sequences per step of the pressure mix, which the float64
oracle computes one by one from its own copy of the inputs (it never sees GPU results); the
transitions and all bookkeeping are checked bit for bit.  To keep the oracle
affordable on a multi-GB pool the harness hands it only the blocks a
transition list touches (renumbered), then writes its results back into the
oracle's own host copy of the pool.
"""

import time

import numpy as np
import pytest

from oracle import attention as oatt
from oracle import lowering as olow
from oracle import transitions as otr
from paper_2609_33536_amd import ekv, kvpool, workloads
from tests.gpu_util import check_attention, default_scale, oracle_transition_on_touched, require_gpu

pytestmark = pytest.mark.gpu

PAGE = 16


def _oracle_on_sample(input_pool, bt, seq_lens, pairs, sample, q_host):
    """Oracle decode of the sampled sequences: extract them from the input
    pool, demote their pairs with the oracle, attend."""
    host, sbt, slens = workloads.extract_sequences(input_pool, bt, seq_lens, sample)
    rows = {int(s): r for r, s in enumerate(sample)}
    sp = np.array([(rows[int(s)], int(j)) for s, j in pairs if int(s) in rows], dtype=np.int32).reshape(-1, 2)
    tg = np.zeros(sbt.shape, dtype=np.uint8)
    if len(sp):
        host, sbt, tg, _, _ = otr.demote(host, sbt, tg, sp, slens)
    return oatt.decode(q_host[list(sample)], host, sbt, tg, slens)


def _decode(kv, q, hq, mode=None, use_boundaries=True, out_fp32=False):
    torch = require_gpu()
    batch = kv.batch(hq, mode=mode, use_boundaries=use_boundaries)
    ws = ekv.decode_workspace(kv.pool, batch)
    out = torch.full((q.shape[0], hq, 128), float("nan"), dtype=torch.float32 if out_fp32 else torch.bfloat16,
                     device="cuda")
    ekv.attn_decode(kv.pool, batch, q, out, default_scale(), ws)
    torch.cuda.synchronize()
    return out


def _host_q(q):
    import torch
    return q.view(torch.int16).cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("fraction", [0.0, 0.25, 0.5, 1.0])
def test_decode_llama3_8b_full_size_every_sequence(fraction):
    torch = require_gpu()
    seq_lens = workloads.seq_lens_uniform(np.random.default_rng(1), 64, 2048, 8192)
    case = workloads.make_decode_case_torch(seq_lens, 32, 8, seed=1, outlier_channels=10, spare_blocks=64)
    k = [0.0, 0.25, 0.5, 1.0].index(fraction)
    pairs = workloads.choose_pairs(np.random.default_rng(1000 + k), seq_lens, fraction, "random")
    kv = kvpool.PagedKV(case["pool"].clone(), case["block_table"], seq_lens, case["free"], 8)
    if len(pairs):
        kv.demote(pairs, emit_lo=False)
        kv.commit()
    mode = kv.relower()
    assert mode == (ekv.MODE_NATIVE if fraction == 0 else
                    ekv.MODE_STRUCTURED if fraction == 1.0 else ekv.MODE_GENERAL)
    print(f"8b decode f={fraction}: pairs={len(pairs)} mode={mode}", flush=True)
    out = _decode(kv, case["q"], 32)
    sample = list(range(64))
    ref = _oracle_on_sample(case["pool"], case["block_table"], seq_lens, pairs, sample, _host_q(case["q"]))
    err, _ = check_attention(out[sample].float().cpu().numpy(), ref, out_fp32=False)
    assert np.isfinite(out.float().cpu().numpy()).all()
    # fp32 output: the strict 2e-3 absolute bound (outlier channels make |o| large)
    out32 = _decode(kv, case["q"], 32, out_fp32=True)
    err32, _ = check_attention(out32[sample].cpu().numpy(), ref, out_fp32=True)
    print(f"  max abs err on {len(sample)} sequences: bf16 out {err:.3e}, fp32 out {err32:.3e}", flush=True)


def test_decode_llama3_70b_full_size_structured_and_general():
    torch = require_gpu()
    seq_lens = np.full(256, 4096, dtype=np.int32)
    case = workloads.make_decode_case_torch(seq_lens, 64, 8, seed=2, spare_blocks=64)
    pairs = workloads.choose_pairs(np.random.default_rng(2), seq_lens, 0.5, "oldest")
    assert len(pairs) == 256 * 64
    kv = kvpool.PagedKV(case["pool"].clone(), case["block_table"], seq_lens, case["free"], 8)
    kv.demote(pairs, emit_lo=False)
    kv.commit()
    mode = kv.relower()
    assert mode == ekv.MODE_STRUCTURED
    assert np.array_equal(kv.bounds.cpu().numpy(), np.tile(np.array([0, 64], dtype=np.int32), (256, 1)))
    print("70b decode: structured", flush=True)
    out_s = _decode(kv, case["q"], 64)
    print("70b decode: forced general", flush=True)
    out_g = _decode(kv, case["q"], 64, mode=ekv.MODE_GENERAL, use_boundaries=False)
    # same pairs, same work partition: the two paths differ only in how a
    # pair's mode is looked up, so the outputs agree bit for bit
    assert torch.equal(out_s, out_g)
    # attention of every sequence against the oracle, bf16 and fp32 output
    every = list(range(256))
    ref = _oracle_on_sample(case["pool"], case["block_table"], seq_lens, pairs, every, _host_q(case["q"]))
    err, _ = check_attention(out_s.float().cpu().numpy(), ref, out_fp32=False)
    out32 = _decode(kv, case["q"], 64, out_fp32=True)
    err32, _ = check_attention(out32.cpu().numpy(), ref, out_fp32=True)
    print(f"  max abs err on all 256 sequences: bf16 out {err:.3e}, fp32 out {err32:.3e}", flush=True)
    sample = [0, 1, 100, 201, 255]
    # the demoted pool, block table and tags of the sampled sequences
    host_in, sbt, slens = workloads.extract_sequences(case["pool"], case["block_table"], seq_lens, sample)
    rows = {s: r for r, s in enumerate(sample)}
    sp = np.array([(rows[int(s)], int(j)) for s, j in pairs if int(s) in rows], dtype=np.int32)
    opool, obt, otg, _, _ = otr.demote(host_in, sbt, np.zeros(sbt.shape, np.uint8), sp, slens)
    gbt, gtg = kv.bt.cpu().numpy(), kv.tags.cpu().numpy()
    pool_dev = kv.kv.view(-1, 2, 8, PAGE, 128)
    for r, s in enumerate(sample):
        assert np.array_equal(gtg[s], otg[r])
        # member 1 of every BASE pair points at member 0's block on both sides
        assert np.array_equal(gbt[s] == np.roll(gbt[s], 1), obt[r] == np.roll(obt[r], 1))
        got = pool_dev.index_select(0, torch.from_numpy(gbt[s][::2].astype(np.int64)).cuda()).cpu().numpy()
        assert np.array_equal(got.view(np.uint16), opool[obt[r][::2]])


def test_pressure_transition_mix_200k_blocks():
    torch = require_gpu()
    nb, bsz, hq, hkv, steps = 200_000, 128, 32, 8, 20
    rng = np.random.default_rng(4)
    seq_lens = workloads.seq_lens_uniform(rng, bsz, 1024, 16384)
    used = sum(-(-int(l) // PAGE) for l in seq_lens)
    t0 = time.time()
    case = workloads.make_decode_case_torch(seq_lens, hq, hkv, seed=4, spare_blocks=nb - used)
    assert case["pool"].shape[0] == nb
    host_pool = case["pool"].cpu().numpy().view(np.uint16)          # the oracle's own copy
    kv = kvpool.PagedKV(case["pool"], case["block_table"], seq_lens, case["free"], hkv)
    q_host = _host_q(case["q"])
    obt, otg = case["block_table"].copy(), np.zeros(case["block_table"].shape, dtype=np.uint8)
    ofifo = otr.FreeFifo(case["free"])
    lo_dev, lo_host = {}, {}
    print(f"pressure mix: pool {nb} blocks, {used} in use, set-up {time.time() - t0:.1f}s", flush=True)
    srng = np.random.default_rng(44)
    for step in range(steps):
        t0 = time.time()
        # (1) demote a random 10 % of the TARGET pairs
        tp = np.array([(s, j) for s in range(bsz) for j in range(int(seq_lens[s]) // (2 * PAGE))
                       if otg[s, 2 * j] == 0], dtype=np.int32)
        nd = int(0.1 * len(tp))
        dp = tp[srng.choice(len(tp), nd, replace=False)] if nd else tp[:0]
        if nd:
            freed, lo, host_freed = kv.demote(dp)
            obt, otg, ofreed, olo, touched = oracle_transition_on_touched("demote", host_pool, obt, otg, seq_lens, dp)
            torch.cuda.synchronize()
            assert np.array_equal(freed.cpu().numpy(), ofreed)
            assert np.array_equal(host_freed, ofreed)
            assert np.array_equal(lo.cpu().numpy().reshape(olo.shape), olo)
            for i, (s, j) in enumerate(dp):
                lo_dev[(int(s), int(j))] = lo[i]
                lo_host[(int(s), int(j))] = olo[i]
            kv.commit()
            ofifo.commit_freed(ofreed)
            got = kv.kv.view(-1, 2, hkv, PAGE, 128).index_select(
                0, torch.from_numpy(touched.astype(np.int64)).cuda()).cpu().numpy().view(np.uint16)
            assert np.array_equal(got, host_pool[touched])
        # (2) refine a random 5 % of the BASE pairs (sampled after this step's demotion)
        bp = np.array([(s, j) for s in range(bsz) for j in range(int(seq_lens[s]) // (2 * PAGE))
                       if otg[s, 2 * j] == 1], dtype=np.int32)
        nr = int(0.05 * len(bp))
        rp = bp[srng.choice(len(bp), nr, replace=False)] if nr else bp[:0]
        if nr:
            lo_in = torch.stack([lo_dev[(int(s), int(j))] for s, j in rp])
            new = kv.refine(rp, lo_in)
            onew = ofifo.acquire(nr)
            assert np.array_equal(new, onew)
            olo_in = np.stack([lo_host[(int(s), int(j))] for s, j in rp])
            obt, otg, _, _, touched = oracle_transition_on_touched("refine", host_pool, obt, otg, seq_lens, rp, onew,
                                                         olo_in)
            torch.cuda.synchronize()
            got = kv.kv.view(-1, 2, hkv, PAGE, 128).index_select(
                0, torch.from_numpy(touched.astype(np.int64)).cuda()).cpu().numpy().view(np.uint16)
            assert np.array_equal(got, host_pool[touched])
        # bookkeeping, bit for bit: device tables, host mirror, free FIFO
        assert np.array_equal(kv.bt.cpu().numpy(), obt)
        assert np.array_equal(kv.tags.cpu().numpy(), otg)
        assert np.array_equal(kv.mirror.bt, obt) and np.array_equal(kv.mirror.tags, otg)
        assert np.array_equal(np.array(kv.mirror.free, dtype=np.int32), ofifo.snapshot())
        # (3) decode the whole batch; check sampled sequences against the oracle
        mode = kv.relower()
        omode, obounds = olow.lower(otg, seq_lens, PAGE)
        assert mode == omode and np.array_equal(kv.bounds.cpu().numpy(), obounds)
        out = _decode(kv, case["q"], hq)
        sample = sorted(srng.choice(bsz, 8, replace=False).tolist())
        ref = oatt.decode(q_host[sample], host_pool, obt[sample], otg[sample], seq_lens[sample])
        err, _ = check_attention(out[sample].float().cpu().numpy(), ref, out_fp32=False)
        assert np.isfinite(out.float().cpu().numpy()).all()
        nbase = int(otg.sum())
        print(f"  step {step}: demoted {nd}, refined {nr}, BASE blocks {nbase}, free {len(ofifo)}, "
              f"mode {mode}, max abs err {err:.3e} ({time.time() - t0:.1f}s)", flush=True)
    # the whole pool, bit for bit
    view = kv.kv.view(-1, 2, hkv, PAGE, 128)
    for b0 in range(0, nb, 16384):
        b1 = min(nb, b0 + 16384)
        assert np.array_equal(view[b0:b1].cpu().numpy().view(np.uint16), host_pool[b0:b1]), (b0, b1)
