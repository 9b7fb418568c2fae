"""GPU parity of the 8-bit TARGET (FP8 E5M2) / 4-bit BASE pools against the
oracle: append, demote (with its refinement nibbles), refine (also staged
and over several layers) bit for bit; decode of mixed pools (native,
structured and general paths, every group size, ragged lengths with a lone
last block) and chunked prefill over such pools (every BASE fraction, ragged
chunks, structured and general, FP16 and FP32 output) within the attention
tolerance."""

import numpy as np
import pytest

from oracle import fp8 as ofp8
from oracle import lowering as olow
from paper_2609_33536_amd import ekv, kvpool, workloads
from tests import softmax_rises
from tests.gpu_util import check_attention, default_scale, host_safety_check, require_gpu, words_to_tensor

pytestmark = pytest.mark.gpu
PAGE = 16


def _bytes_tensor(a, torch):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).cuda()


def _run_decode(case, hq, hkv, *, out_fp32=True, use_boundaries=True, force_mode=None, scale=None):
    torch = require_gpu()
    scale = default_scale() if scale is None else scale
    host_safety_check(case, case["pool"].shape)
    kv = kvpool.PagedKV(case["pool"], case["block_table"], case["seq_lens"], case["free"], hkv, "e5m2")
    opool, obt, otg = case["pool"], case["block_table"], case["tags"]
    if len(case["pairs"]):
        freed, lo, _ = kv.demote(case["pairs"])
        opool, obt, otg, ofreed, olo = ofp8.demote(opool, obt, otg, case["pairs"], case["seq_lens"])
        torch.cuda.synchronize()
        assert np.array_equal(freed.cpu().numpy(), ofreed)
        assert np.array_equal(lo.cpu().numpy().reshape(olo.shape), olo)
        assert np.array_equal(kv.bt.cpu().numpy(), obt) and np.array_equal(kv.tags.cpu().numpy(), otg)
        assert np.array_equal(kv.kv.cpu().numpy().reshape(opool.shape), opool)
    mode = kv.relower()
    omode, obounds = olow.lower(otg, case["seq_lens"], PAGE)
    assert mode == omode
    if force_mode is not None:
        mode = force_mode
    q = words_to_tensor(case["q"], torch, "fp16")
    bsz = len(case["seq_lens"])
    out = torch.full((bsz, hq, 128), float("nan"), dtype=torch.float32 if out_fp32 else torch.float16,
                     device="cuda")
    batch = kv.batch(hq, mode=mode, use_boundaries=use_boundaries)
    ws = ekv.decode_workspace(kv.pool, batch)
    print(f"decode e5m2: B={bsz} Hq={hq} Hkv={hkv} mode={mode} fp32={out_fp32}", flush=True)
    ekv.attn_decode(kv.pool, batch, q, out, scale, ws)
    torch.cuda.synchronize()
    ref = ofp8.decode(case["q"], opool, obt, otg, case["seq_lens"], scale)
    return check_attention(out.float().cpu().numpy(), ref, out_fp32)


@pytest.mark.parametrize("scale", [0.03, -0.1, 0.0, -0.0])
def test_decode_e5m2_softmax_scales(scale):
    """Other softmax scales on the 8-bit pool: negative (applied as the
    query's sign) and zero of either sign; structured and general paths."""
    c = workloads.make_decode_case([33, 700, 64, 1500], 16, 4, dtype="e5m2", seed=45, base_fraction=0.5,
                                   spare_blocks=4)
    _run_decode(c, 16, 4, scale=scale)
    _run_decode(c, 16, 4, scale=scale, use_boundaries=False)


@pytest.mark.parametrize("fraction", [0.0, 0.5, 1.0])
@pytest.mark.parametrize("group", [1, 4, 8, 16])
def test_decode_e5m2_groups_fractions_ragged(group, fraction):
    hkv = 2
    lens = [1, 15, 16, 17, 33, 100, 257, 511, 640, 1000, 0, 48]
    c = workloads.make_decode_case(lens, hkv * group, hkv, dtype="e5m2", seed=80 + group, base_fraction=fraction,
                                   spare_blocks=4)
    _run_decode(c, hkv * group, hkv)


def test_decode_e5m2_structured_general_native_and_fp16_output():
    c = workloads.make_decode_case([512, 1024, 768, 96, 333], 32, 8, dtype="e5m2", seed=90, base_fraction=0.5,
                                   placement="oldest", spare_blocks=2)
    _run_decode(c, 32, 8)
    _run_decode(c, 32, 8, use_boundaries=False, force_mode=ekv.MODE_GENERAL)
    _run_decode(c, 32, 8, out_fp32=False)
    c0 = workloads.make_decode_case([700, 64, 1500], 32, 8, dtype="e5m2", seed=91, base_fraction=0.0,
                                    spare_blocks=2)
    _run_decode(c0, 32, 8)                                         # native: no tags read
    _run_decode(c0, 32, 8, force_mode=ekv.MODE_GENERAL, use_boundaries=False)


def test_transitions_e5m2_bit_exact():
    torch = require_gpu()
    hkv = 4
    c = workloads.make_decode_case([300, 1024, 77, 2000], 16, hkv, dtype="e5m2", seed=92, base_fraction=0.6,
                                   spare_blocks=40)
    host_safety_check(c, c["pool"].shape)
    rng = np.random.default_rng(93)
    pool = rng.integers(0, 256, size=c["pool"].shape, dtype=np.uint8)       # every byte pattern
    layers = [pool, rng.integers(0, 256, size=c["pool"].shape, dtype=np.uint8)]
    dev = [_bytes_tensor(p, torch) for p in layers]
    layer_kv = torch.tensor([t.data_ptr() for t in dev], dtype=torch.int64, device="cuda")
    ep = ekv.make_pool(dev[0], hkv, "e5m2")
    pairs = c["pairs"]
    n = len(pairs)
    block_bytes = 2 * hkv * PAGE * 128
    bt = torch.from_numpy(c["block_table"].copy()).cuda()
    tags = torch.from_numpy(c["tags"].copy()).cuda()
    pairs_d = torch.from_numpy(pairs.copy()).cuda()
    freed = torch.empty(n, dtype=torch.int32, device="cuda")
    lo = torch.empty((n, 2, block_bytes), dtype=torch.uint8, device="cuda")
    print(f"demote e5m2 layers: pairs={n}", flush=True)
    ekv.demote_layers(ep, layer_kv, pairs_d, bt, tags, freed, lo)
    torch.cuda.synchronize()
    outs = [ofp8.demote(p, c["block_table"], c["tags"], pairs, c["seq_lens"]) for p in layers]
    _, obt, otg, ofreed, _ = outs[0]
    assert np.array_equal(bt.cpu().numpy(), obt) and np.array_equal(tags.cpu().numpy(), otg)
    assert np.array_equal(freed.cpu().numpy(), ofreed)
    lo_h = lo.cpu().numpy()
    for layer, (op, _, _, _, olo) in enumerate(outs):
        assert np.array_equal(dev[layer].cpu().numpy(), op), layer
        assert np.array_equal(lo_h[:, layer].reshape(olo.shape), olo), layer
    # refine: layer 0 from its lo (single-layer call), layer 1 staged in the new blocks
    new = np.array((sorted(c["free"].tolist()) + ofreed.tolist())[:n], dtype=np.int32)
    new_d = torch.from_numpy(new).cuda()
    lo0 = lo[:, 0].contiguous()
    bt1, tags1 = bt.clone(), tags.clone()
    print("refine e5m2", flush=True)
    ekv.refine(ep, pairs_d, new_d, bt, tags, lo0)
    flat1 = dev[1].view(-1)
    for i, q in enumerate(new):
        flat1[int(q) * block_bytes:(int(q) + 1) * block_bytes].copy_(lo[i, 1])
    ep1 = ekv.make_pool(dev[1], hkv, "e5m2")
    ekv.refine_staged(ep1, pairs_d, new_d, bt1, tags1)
    torch.cuda.synchronize()
    for layer, (op, obt_, otg_, _, olo) in enumerate(outs):
        rp, rbt, rtg = ofp8.refine(op, obt_, otg_, pairs, new, olo, c["seq_lens"])
        assert np.array_equal(dev[layer].cpu().numpy(), rp), layer
    assert np.array_equal(bt.cpu().numpy(), rbt) and np.array_equal(bt1.cpu().numpy(), rbt)
    assert np.array_equal(tags.cpu().numpy(), rtg) and np.array_equal(tags1.cpu().numpy(), rtg)
    # the round trip restores every byte of the visible blocks
    got = dev[0].cpu().numpy()
    for s, length in enumerate(c["seq_lens"]):
        for i in range(-(-int(length) // PAGE)):
            assert np.array_equal(got[rbt[s, i]], pool[c["block_table"][s, i]]), (s, i)


def test_append_e5m2_bit_exact():
    torch = require_gpu()
    hkv = 8
    rng = np.random.default_rng(94)
    pool = rng.integers(0, 256, size=(20, 2, hkv, PAGE, 128), dtype=np.uint8)
    slots = np.array([3 * PAGE + 5, 7 * PAGE, 19 * PAGE + 15, 0], dtype=np.int32)
    k = rng.integers(0, 256, size=(4, hkv, 128), dtype=np.uint8)
    v = rng.integers(0, 256, size=(4, hkv, 128), dtype=np.uint8)
    dev = _bytes_tensor(pool, torch)
    ekv.append_kv(ekv.make_pool(dev, hkv, "e5m2"), torch.from_numpy(slots).cuda(), _bytes_tensor(k, torch),
                  _bytes_tensor(v, torch))
    torch.cuda.synchronize()
    assert np.array_equal(dev.cpu().numpy(), ofp8.append(pool, slots, k, v))


def _run_prefill(case, hq, hkv, *, use_boundaries=True, out_fp32=True, scale=None):
    torch = require_gpu()
    scale = default_scale() if scale is None else scale
    host_safety_check(case, case["pool"].shape)
    assert (case["slots"] >= 0).all() and (case["slots"] < case["pool"].shape[0] * PAGE).all()
    kv = kvpool.PagedKV(case["pool"], case["block_table"], case["seq_lens"], case["free"], hkv, "e5m2")
    kv.append(torch.from_numpy(case["slots"]).cuda(), _bytes_tensor(case["k_new"], torch),
              _bytes_tensor(case["v_new"], torch))
    opool = ofp8.append(case["pool"], case["slots"], case["k_new"], case["v_new"])
    obt, otg = case["block_table"], case["tags"]
    if len(case["pairs"]):
        kv.demote(case["pairs"])
        opool, obt, otg, _, _ = ofp8.demote(opool, obt, otg, case["pairs"], case["seq_lens"])
    kv.relower()
    q = words_to_tensor(case["q"], torch, "fp16")
    flags = tuple(out_fp32) if isinstance(out_fp32, (tuple, list)) else (out_fp32,)
    max_q = int(np.diff(case["cu_q"]).max())
    print(f"prefill e5m2: B={len(case['seq_lens'])} Hq={hq} Hkv={hkv} rows={q.shape[0]} pairs={len(case['pairs'])} "
          f"boundaries={use_boundaries} fp32={flags}", flush=True)
    outs = []
    for fp32 in flags:
        out = torch.full((q.shape[0], hq, 128), float("nan"), dtype=torch.float32 if fp32 else torch.float16,
                         device="cuda")
        ekv.attn_prefill(kv.pool, kv.batch(hq, use_boundaries=use_boundaries), q,
                         torch.from_numpy(case["cu_q"]).cuda(), max_q, out, scale)
        outs.append(out)
    torch.cuda.synchronize()
    ref = ofp8.prefill(case["q"], case["cu_q"], opool, obt, otg, case["seq_lens"], scale)
    for fp32, out in zip(flags, outs):
        res = check_attention(out.float().cpu().numpy(), ref, fp32)
        print(f"  fp32={fp32}: max abs err {res[0]:.3e}", flush=True)
    return res


@pytest.mark.parametrize("fraction", [0.0, 0.5, 1.0])
@pytest.mark.parametrize("group", [1, 4, 16])
def test_prefill_e5m2_groups_fractions_ragged(group, fraction):
    hkv = 2
    c = workloads.make_prefill_case([0, 17, 64, 100, 250, 33], [1, 40, 31, 7, 64, 90], hkv * group, hkv,
                                    dtype="e5m2", seed=96 + group, base_fraction=fraction, spare_blocks=4)
    _run_prefill(c, hkv * group, hkv)


def test_prefill_e5m2_structured_general_and_fp16_output():
    """The BASE run crosses the kernel's 64-block metadata windows."""
    c = workloads.make_prefill_case([2000, 640, 70], [90, 37, 5], 32, 8, dtype="e5m2", seed=97,
                                    base_fraction=0.8, placement="oldest", spare_blocks=2)
    _run_prefill(c, 32, 8)
    _run_prefill(c, 32, 8, use_boundaries=False)
    _run_prefill(c, 32, 8, out_fp32=False)


@pytest.mark.parametrize("scale", [0.03, -0.1, 0.0, -0.0])
def test_prefill_e5m2_empty_chunks_and_scales(scale):
    """Empty chunks, an empty sequence and single-token chunks in one batch,
    at other softmax scales (a negative one included)."""
    c = workloads.make_prefill_case([100, 0, 300, 0, 64, 1], [20, 0, 0, 5, 33, 1], 8, 2, dtype="e5m2", seed=42,
                                    base_fraction=0.5, spare_blocks=4)
    _run_prefill(c, 8, 2, scale=scale)
    _run_prefill(c, 8, 2, scale=scale, use_boundaries=False)


def test_prefill_e5m2_chunks_at_8b_shape():
    """4 x (1024-token prefix, half of its pairs BASE, + 256-token chunk),
    32 query / 8 KV heads: every output checked."""
    c = workloads.make_prefill_case([1024] * 4, [256] * 4, 32, 8, dtype="e5m2", seed=98, base_fraction=0.5,
                                    spare_blocks=2)
    _run_prefill(c, 32, 8, out_fp32=False)


@pytest.mark.parametrize("fraction", [0.0, 0.5, 1.0])
def test_decode_e5m2_8b_full_size_every_sequence(fraction):
    """The 8B decode layer over an 8-bit pool as the benchmark runs it (64
    sequences, context uniform in [2048, 8192], 1 % outlier channels, random
    BASE pairs): every sequence against the oracle, FP16 and FP32 output."""
    torch = require_gpu()
    seq_lens = workloads.seq_lens_uniform(np.random.default_rng(1), 64, 2048, 8192)
    case = workloads.make_decode_case_torch(seq_lens, 32, 8, seed=6, outlier_channels=10, spare_blocks=64,
                                            dtype="e5m2")
    k = [0.0, 0.5, 1.0].index(fraction)
    pairs = workloads.choose_pairs(np.random.default_rng(2000 + k), seq_lens, fraction, "random")
    kv = kvpool.PagedKV(case["pool"].clone(), case["block_table"], seq_lens, case["free"], 8, "e5m2")
    if len(pairs):
        kv.demote(pairs, emit_lo=False)
        kv.commit()
    mode = kv.relower()
    print(f"8-bit 8b decode f={fraction}: pairs={len(pairs)} mode={mode}", flush=True)
    batch = kv.batch(32)
    ws = ekv.decode_workspace(kv.pool, batch)
    sample = list(range(64))
    host, sbt, slens = workloads.extract_sequences(case["pool"], case["block_table"], seq_lens, sample)
    rows = {s: r for r, s in enumerate(sample)}
    sp = np.array([(rows[int(s)], int(j)) for s, j in pairs if int(s) in rows], dtype=np.int32).reshape(-1, 2)
    tg = np.zeros(sbt.shape, dtype=np.uint8)
    if len(sp):
        host, sbt, tg, _, _ = ofp8.demote(host, sbt, tg, sp, slens)
    q_words = case["q"].view(torch.int16).cpu().numpy().view(np.uint16)
    ref = ofp8.decode(q_words[sample], host, sbt, tg, slens)
    for out_dtype in (torch.float16, torch.float32):
        out = torch.full((64, 32, 128), float("nan"), dtype=out_dtype, device="cuda")
        ekv.attn_decode(kv.pool, batch, case["q"], out, default_scale(), ws)
        torch.cuda.synchronize()
        got = out.float().cpu().numpy()
        assert np.isfinite(got).all()
        err, _ = check_attention(got[sample], ref, out_dtype == torch.float32)
        print(f"  {out_dtype}: max abs err {err:.3e} on {len(sample)} sequences", flush=True)


@pytest.mark.parametrize("permille", [1000, 1900])
@pytest.mark.parametrize("fraction", [0.5, 1.0])
def test_decode_e5m2_8b_weighted_ranges(fraction, permille, monkeypatch):
    """The full-size 8-bit layer fills the grid (two waves per SIMD), so the
    launcher gives the first-slot workgroups longer ranges.  At equal ranges
    (1000) and at the largest weight (1900: the other ranges shrink to a few
    pairs, so (sequence, KV head)s are cut into more pieces) every sequence
    still matches the oracle (FP32 output)."""
    torch = require_gpu()
    seq_lens = workloads.seq_lens_uniform(np.random.default_rng(1), 64, 2048, 8192)
    case = workloads.make_decode_case_torch(seq_lens, 32, 8, seed=6, outlier_channels=10, spare_blocks=64,
                                            dtype="e5m2")
    pairs = workloads.choose_pairs(np.random.default_rng(2100 + int(2 * fraction)), seq_lens, fraction, "random")
    kv = kvpool.PagedKV(case["pool"].clone(), case["block_table"], seq_lens, case["free"], 8, "e5m2")
    kv.demote(pairs, emit_lo=False)
    kv.commit()
    kv.relower()
    batch = kv.batch(32)
    ws = ekv.decode_workspace(kv.pool, batch)
    monkeypatch.setenv("EKV_HEAVY_PERMILLE", str(permille))
    print(f"8-bit weighted ranges: f={fraction} permille={permille} pairs={len(pairs)}", flush=True)
    out = torch.full((64, 32, 128), float("nan"), dtype=torch.float32, device="cuda")
    ekv.attn_decode(kv.pool, batch, case["q"], out, default_scale(), ws)
    torch.cuda.synchronize()
    sample = list(range(64))
    host, sbt, slens = workloads.extract_sequences(case["pool"], case["block_table"], seq_lens, sample)
    tg = np.zeros(sbt.shape, dtype=np.uint8)
    host, sbt, tg, _, _ = ofp8.demote(host, sbt, tg, pairs, slens)
    q_words = case["q"].view(torch.int16).cpu().numpy().view(np.uint16)
    ref = ofp8.decode(q_words, host, sbt, tg, slens)
    err, _ = check_attention(out.cpu().numpy(), ref, True)
    print(f"  max abs err {err:.3e} on 64 sequences", flush=True)


@pytest.mark.parametrize("fraction", [0.5, 1.0])
def test_decode_e5m2_weighted_ranges_near_the_minimum_range(fraction):
    """16 sequences of 4608 tokens, 32/8 heads: 18,432 pairs fill the grid
    of 2048 workgroups with 9 pairs each on average, just above the minimum
    range of 8, so the weighted ranges apply at their smallest (11 pairs for
    the first-slot workgroups, 7 for the others) and most (sequence, KV
    head)s are cut into many pieces.  Every sequence against the oracle."""
    torch = require_gpu()
    seq_lens = np.full(16, 4608, dtype=np.int32)
    case = workloads.make_decode_case_torch(seq_lens, 32, 8, seed=8, outlier_channels=10, spare_blocks=16,
                                            dtype="e5m2")
    pairs = workloads.choose_pairs(np.random.default_rng(2200 + int(2 * fraction)), seq_lens, fraction, "random")
    kv = kvpool.PagedKV(case["pool"].clone(), case["block_table"], seq_lens, case["free"], 8, "e5m2")
    kv.demote(pairs, emit_lo=False)
    kv.commit()
    kv.relower()
    batch = kv.batch(32)
    ws = ekv.decode_workspace(kv.pool, batch)
    print(f"8-bit weighted ranges near the minimum: f={fraction} pairs={len(pairs)}", flush=True)
    out = torch.full((16, 32, 128), float("nan"), dtype=torch.float32, device="cuda")
    ekv.attn_decode(kv.pool, batch, case["q"], out, default_scale(), ws)
    torch.cuda.synchronize()
    sample = list(range(16))
    host, sbt, slens = workloads.extract_sequences(case["pool"], case["block_table"], seq_lens, sample)
    tg = np.zeros(sbt.shape, dtype=np.uint8)
    host, sbt, tg, _, _ = ofp8.demote(host, sbt, tg, pairs, slens)
    q_words = case["q"].view(torch.int16).cpu().numpy().view(np.uint16)
    ref = ofp8.decode(q_words, host, sbt, tg, slens)
    err, _ = check_attention(out.cpu().numpy(), ref, True)
    print(f"  max abs err {err:.3e} on 16 sequences", flush=True)


def test_prefill_e5m2_8b_full_size():
    """The chunked-prefill workload over an 8-bit pool as the benchmark runs
    it: 16 x (2048-token prefix, half its pairs BASE, + 512-token chunk), 32
    query / 8 KV heads; every output checked."""
    c = workloads.make_prefill_case([2048] * 16, [512] * 16, 32, 8, dtype="e5m2", seed=3, base_fraction=0.5,
                                    spare_blocks=2)
    _run_prefill(c, 32, 8, out_fp32=(False, True))


@pytest.mark.parametrize("name", ["aligned-e5m2", "scale1-e5m2-g1"])
def test_prefill_e5m2_rescale_of_live_output(name):
    """8-bit pools on inputs that make the kernel rescale accumulators that
    already hold output (shown on the CPU by test_rescale_inputs.py)."""
    case, hq, hkv, scale, dtype = softmax_rises.make(name)
    assert dtype == "e5m2"
    _run_prefill(case, hq, hkv, out_fp32=(True, False), scale=scale)
    _run_prefill(case, hq, hkv, out_fp32=True, scale=scale, use_boundaries=False)


def test_prefill_e5m2_repeatable():
    """The 8-bit chunked prefill at the benchmark's size gives the same bits
    on every launch.  BASE units widen their nibbles into LDS with vector
    writes that other waves read after a barrier; without the wait for
    those writes before the barrier, some launches read stale tile bytes in
    one wave (seen as ~3e3 outputs differing, errors up to 2.7e-3)."""
    torch = require_gpu()
    c = workloads.make_prefill_case([2048] * 16, [512] * 16, 32, 8, dtype="e5m2", seed=3, base_fraction=0.5,
                                    spare_blocks=2)
    kv = kvpool.PagedKV(c["pool"], c["block_table"], c["seq_lens"], c["free"], 8, "e5m2")
    kv.append(torch.from_numpy(c["slots"]).cuda(), _bytes_tensor(c["k_new"], torch), _bytes_tensor(c["v_new"], torch))
    kv.demote(c["pairs"])
    kv.relower()
    q = words_to_tensor(c["q"], torch, "fp16")
    cu = torch.from_numpy(c["cu_q"]).cuda()
    first = None
    for rep in range(12):
        out = torch.full((q.shape[0], 32, 128), float("nan"), dtype=torch.float16, device="cuda")
        ekv.attn_prefill(kv.pool, kv.batch(32), q, cu, 512, out, default_scale())
        torch.cuda.synchronize()
        if first is None:
            first = out
        else:
            differ = int((out != first).sum())
            print(f"repeat {rep}: {differ} outputs differ from the first launch", flush=True)
            assert differ == 0, rep
