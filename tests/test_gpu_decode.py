"""GPU parity of the dual-mode decode path and the transitions against the
float64 oracle, on seeded inputs that span several tiles and ragged tails.

Attention: within 2e-3 absolute (fp32 output) or 2e-3 + 1e-2|o| (16-bit
output).  Demotion, refinement, block tables, tags, freed ids and the
refinement bytes: bit-exact.
"""

import os

import numpy as np
import pytest

from oracle import attention as oatt
from oracle import lowering as olow
from oracle import transitions as otr
from paper_2609_33536_amd import ekv, kvpool, workloads
from tests.gpu_util import check_attention, default_scale, host_safety_check, require_gpu, words_to_tensor

pytestmark = pytest.mark.gpu


def _run(case, hq, hkv, *, out_fp32=True, use_boundaries=True, force_mode=None, min_chunk=None, scale=None):
    """Demote on both sides, decode on the GPU, compare everything."""
    scale = default_scale() if scale is None else scale
    torch = require_gpu()
    dtype = case["dtype"]
    host_safety_check(case, case["pool"].shape)
    kv = kvpool.PagedKV(case["pool"], case["block_table"], case["seq_lens"], case["free"], hkv, dtype)
    opool, obt, otg = case["pool"], case["block_table"], case["tags"]
    if len(case["pairs"]):
        freed, lo, _ = kv.demote(case["pairs"])
        opool, obt, otg, ofreed, olo = otr.demote(opool, obt, otg, case["pairs"], case["seq_lens"])
        torch.cuda.synchronize()
        assert np.array_equal(freed.cpu().numpy(), ofreed)
        assert np.array_equal(lo.cpu().numpy().reshape(olo.shape), olo)
        assert np.array_equal(kv.bt.cpu().numpy(), obt)
        assert np.array_equal(kv.tags.cpu().numpy(), otg)
        assert np.array_equal(kv.kv.cpu().numpy().view(np.uint16), opool)
    mode = kv.relower()
    omode, obounds = olow.lower(otg, case["seq_lens"], 16)
    assert mode == omode and np.array_equal(kv.bounds.cpu().numpy(), obounds)
    if force_mode is not None:
        mode = force_mode
    q = words_to_tensor(case["q"], torch, dtype)
    bsz = len(case["seq_lens"])
    out_dtype = torch.float32 if out_fp32 else q.dtype
    out = torch.full((bsz, hq, 128), float("nan"), dtype=out_dtype, device="cuda")
    old = os.environ.get("EKV_MIN_CHUNK")
    if min_chunk:
        os.environ["EKV_MIN_CHUNK"] = str(min_chunk)
    try:
        batch = kv.batch(hq, mode=mode, use_boundaries=use_boundaries)
        ws = ekv.decode_workspace(kv.pool, batch)
        print(f"decode: B={bsz} Hq={hq} Hkv={hkv} mode={mode} bounds={use_boundaries} "
              f"min_chunk={min_chunk} fp32={out_fp32} {dtype} scale={scale:.4f}", flush=True)
        ekv.attn_decode(kv.pool, batch, q, out, scale, ws)
        torch.cuda.synchronize()
    finally:
        if min_chunk:
            if old is None:
                del os.environ["EKV_MIN_CHUNK"]
            else:
                os.environ["EKV_MIN_CHUNK"] = old
    ref = oatt.decode(case["q"], opool, obt, otg, case["seq_lens"], dtype, scale)
    got = out.float().cpu().numpy()
    return check_attention(got, ref, out_fp32), kv, opool, obt, otg


def test_tiny_decode_mixed_and_round_trip():
    """4 sequences of 64..256 tokens, GQA 4, half the pairs BASE (seed 0);
    then every BASE pair refined back and the pool compared bit for bit."""
    c = workloads.make_decode_case([64, 128, 192, 256], 8, 2, seed=0, base_fraction=0.5, spare_blocks=8)
    (err, rel), kv, opool, obt, otg = _run(c, 8, 2)
    torch = require_gpu()
    kv.commit()
    lo = None
    # refinement needs the bytes demotion emitted; demote again on a fresh pool to get them
    kv2 = kvpool.PagedKV(c["pool"], c["block_table"], c["seq_lens"], c["free"], 2)
    _, lo, host_freed = kv2.demote(c["pairs"])
    kv2.commit()
    new = kv2.refine(c["pairs"], lo)
    torch.cuda.synchronize()
    _, _, _, ofreed, olo = otr.demote(c["pool"], c["block_table"], c["tags"], c["pairs"], c["seq_lens"])
    ofifo = otr.FreeFifo(c["free"])
    ofifo.commit_freed(ofreed)
    onew = ofifo.acquire(len(c["pairs"]))
    assert np.array_equal(new, onew)
    rpool, rbt, rtg = otr.refine(opool, obt, otg, c["pairs"], onew, olo, c["seq_lens"])
    assert np.array_equal(kv2.kv.cpu().numpy().view(np.uint16), rpool)
    assert np.array_equal(kv2.bt.cpu().numpy(), rbt)
    assert not kv2.tags.cpu().numpy().any()
    for s in range(4):
        for i in range(-(-int(c["seq_lens"][s]) // 16)):
            assert np.array_equal(rpool[rbt[s, i]], c["pool"][c["block_table"][s, i]])


@pytest.mark.parametrize("fraction", [0.0, 0.25, 0.5, 1.0])
@pytest.mark.parametrize("group", [1, 2, 4, 8, 16])
def test_decode_groups_fractions_ragged(group, fraction):
    lens = [1, 15, 16, 17, 33, 100, 257, 511, 640, 1000]
    hkv = 2
    c = workloads.make_decode_case(lens, hkv * group, hkv, seed=10 + group, base_fraction=fraction,
                                   spare_blocks=4)
    _run(c, hkv * group, hkv)


@pytest.mark.parametrize("min_chunk", [1, 2, 3, 8, 64])
def test_decode_work_partition(min_chunk):
    """Ranges of 1..64 pairs per workgroup: sequences cut into many pieces
    (both merge paths: <= 64 pieces and more), pieces spanning sequences."""
    c = workloads.make_decode_case([300, 1024, 77, 2000, 0, 4500], 32, 8, seed=3, base_fraction=0.5,
                                   spare_blocks=2)
    _run(c, 32, 8, min_chunk=min_chunk)


@pytest.mark.parametrize("group", [1, 2, 8, 16])
def test_decode_merges_every_group(group):
    """One-pair ranges: the 141-pair (sequence, KV head)s of the 4500-token
    sequence merge 141 pieces each (the serial path), the 63-pair ones 63
    (the batched path), the 10-pair ones 10; the slot layout of the partial
    rows depends on the group size."""
    hkv = 2
    c = workloads.make_decode_case([4500, 300, 2000], hkv * group, hkv, seed=120 + group, base_fraction=0.5,
                                   spare_blocks=2)
    _run(c, hkv * group, hkv, min_chunk=1)


def test_structured_and_general_paths_agree():
    """Oldest pairs BASE (structured); same inputs forced through the tag table."""
    c = workloads.make_decode_case([512, 1024, 768, 96], 16, 2, seed=4, base_fraction=0.5,
                                   placement="oldest", spare_blocks=2)
    (e1, _), kv1, *_ = _run(c, 16, 2)
    assert kv1.mode == ekv.MODE_STRUCTURED
    _run(c, 16, 2, use_boundaries=False, force_mode=ekv.MODE_GENERAL)


def test_native_and_elastic_agree_at_zero_base_fraction():
    c = workloads.make_decode_case([700, 64, 1500], 32, 8, seed=5, base_fraction=0.0, spare_blocks=2)
    _run(c, 32, 8)                                             # native (no tags read)
    _run(c, 32, 8, force_mode=ekv.MODE_GENERAL, use_boundaries=False)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("out_fp32", [True, False])
def test_dtypes_and_outputs(dtype, out_fp32):
    c = workloads.make_decode_case([200, 333, 32, 1024], 16, 4, dtype=dtype, seed=6, base_fraction=0.5,
                                   spare_blocks=2, outlier_channels=5)
    _run(c, 16, 4, out_fp32=out_fp32)


@pytest.mark.parametrize("scale", [0.02, 0.3, -0.088, 0.0, -0.0])
def test_decode_softmax_scales(scale):
    """Other softmax scales, a negative one included (the kernels apply its
    sign to Q), and zero of either sign (uniform attention: a zero scale
    must never multiply a masked score's infinity): structured and general
    paths."""
    c = workloads.make_decode_case([33, 700, 64, 1500], 16, 4, seed=44, base_fraction=0.5, spare_blocks=4)
    _run(c, 16, 4, scale=scale)
    _run(c, 16, 4, scale=scale, use_boundaries=False)


def test_zero_length_and_single_token_sequences():
    c = workloads.make_decode_case([0, 1, 0, 48], 8, 2, seed=7, base_fraction=1.0, spare_blocks=2)
    _run(c, 8, 2)


def test_host_rejects_bad_transitions_before_launch():
    require_gpu()
    c = workloads.make_decode_case([64, 64], 8, 2, seed=8, base_fraction=1.0, spare_blocks=2)
    kv = kvpool.PagedKV(c["pool"], c["block_table"], c["seq_lens"], c["free"], 2)
    kv.demote(c["pairs"])
    with pytest.raises(ekv.EkvError):
        kv.demote(c["pairs"])              # already BASE


def test_workspace_reused_across_calls_and_init():
    """The split-merge counters reset themselves: three calls on one
    workspace (the first after ekv_decode_workspace_init on a dirty buffer)
    all match the oracle."""
    torch = require_gpu()
    c = workloads.make_decode_case([3000, 100, 2048, 5000], 32, 8, seed=9, base_fraction=0.5,
                                   spare_blocks=2)
    kv = kvpool.PagedKV(c["pool"], c["block_table"], c["seq_lens"], c["free"], 8)
    kv.demote(c["pairs"])
    kv.relower()
    opool, obt, otg, _, _ = otr.demote(c["pool"], c["block_table"], c["tags"], c["pairs"], c["seq_lens"])
    ref = oatt.decode(c["q"], opool, obt, otg, c["seq_lens"])
    q = words_to_tensor(c["q"], torch, "bf16")
    batch = kv.batch(32)
    ws = torch.full((ekv.decode_workspace_bytes(kv.pool, batch),), 0xAB, dtype=torch.uint8, device="cuda")
    ekv.decode_workspace_init(ws)
    for call in range(3):
        out = torch.full((4, 32, 128), float("nan"), dtype=torch.float32, device="cuda")
        ekv.attn_decode(kv.pool, batch, q, out, default_scale(), ws)
        torch.cuda.synchronize()
        check_attention(out.cpu().numpy(), ref, True)


def test_one_workspace_for_batches_of_different_grids():
    """A workspace sized for the largest batch serves smaller ones whose
    launches use fewer workgroups (other slot layouts), and the large one
    again after them: every call matches the oracle (the merge counters
    keep one place whatever the grid)."""
    torch = require_gpu()
    cases = [workloads.make_decode_case(lens, 32, 8, seed=90 + k, base_fraction=0.5, spare_blocks=2)
             for k, lens in enumerate(([3000, 100, 2048, 5000, 4000, 700], [40, 900], [3000, 100, 2048, 5000, 4000, 700]))]
    runs = []
    for c in cases:
        kv = kvpool.PagedKV(c["pool"], c["block_table"], c["seq_lens"], c["free"], 8)
        kv.demote(c["pairs"])
        kv.relower()
        opool, obt, otg, _, _ = otr.demote(c["pool"], c["block_table"], c["tags"], c["pairs"], c["seq_lens"])
        runs.append((kv, oatt.decode(c["q"], opool, obt, otg, c["seq_lens"]), words_to_tensor(c["q"], torch, "bf16")))
    need = [ekv.decode_workspace_bytes(kv.pool, kv.batch(32)) for kv, _, _ in runs]
    assert need[1] < need[0]
    ws = torch.full((max(need),), 0xAB, dtype=torch.uint8, device="cuda")
    ekv.decode_workspace_init(ws)
    for k, (kv, ref, q) in enumerate(runs + runs[1:2]):
        out = torch.full((len(kv.mirror.seq_lens), 32, 128), float("nan"), dtype=torch.float32, device="cuda")
        print(f"shared workspace: call {k} B={len(kv.mirror.seq_lens)}", flush=True)
        ekv.attn_decode(kv.pool, kv.batch(32), q, out, default_scale(), ws)
        torch.cuda.synchronize()
        check_attention(out.cpu().numpy(), ref, True)


@pytest.mark.parametrize("dtype", ["bf16", "e5m2"])
def test_decode_batch_of_700_short_sequences(dtype):
    """More sequences than one wave's lanes and than one pass of the range
    scan (700 > 512): lengths 0..96, half the eligible pairs BASE, so the
    work walker reloads its window of lengths every 64 sequences and skips
    empty ones, and most (sequence, KV head)s are cut between workgroups."""
    rng = np.random.default_rng(77)
    lens = rng.integers(0, 97, size=700).tolist()
    c = workloads.make_decode_case(lens, 8, 2, seed=78, base_fraction=0.5, spare_blocks=4, dtype=dtype)
    if dtype == "e5m2":
        from tests import test_gpu_fp8
        test_gpu_fp8._run_decode(c, 8, 2)
    else:
        _run(c, 8, 2)
