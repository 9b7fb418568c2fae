"""The no-allocation decode (ekv_attn_decode_noalloc) against ekv_attn_decode.

Two calls in a row on the library's static scratch, the second with a
smaller batch (fewer workgroups, other slots of the scratch), each compared
with the workspace entry point on the same inputs (bit for bit: the same
kernel and grid) and with the float64 oracle (attention tolerance)."""

import numpy as np
import pytest

from oracle import attention as oatt
from oracle import transitions as otr
from paper_2609_33536_amd import ekv, kvpool, workloads
from tests.gpu_util import check_attention, default_scale, host_safety_check, require_gpu, words_to_tensor

pytestmark = pytest.mark.gpu


def _prepared(lens, hq, hkv, seed, fraction, placement):
    torch = require_gpu()
    c = workloads.make_decode_case(lens, hq, hkv, seed=seed, base_fraction=fraction, placement=placement,
                                   spare_blocks=4)
    host_safety_check(c, c["pool"].shape)
    kv = kvpool.PagedKV(c["pool"], c["block_table"], c["seq_lens"], c["free"], hkv)
    if len(c["pairs"]):
        kv.demote(c["pairs"])
        kv.commit()
    kv.relower()
    opool, obt, otg, _, _ = otr.demote(c["pool"], c["block_table"], c["tags"], c["pairs"], c["seq_lens"])
    ref = oatt.decode(c["q"], opool, obt, otg, c["seq_lens"])
    return kv, words_to_tensor(c["q"], torch, "bf16"), ref


def test_noalloc_decode_matches_workspace_decode_on_two_calls():
    torch = require_gpu()
    rng = np.random.default_rng(71)
    big = _prepared(rng.integers(1, 6000, size=24).tolist(), 32, 8, 72, 0.5, "random")      # general
    small = _prepared([700, 33, 2050, 96], 16, 4, 73, 0.5, "oldest")                           # structured
    scale = default_scale()
    for name, (kv, q, ref) in (("large", big), ("small", small)):
        hq = q.shape[1]
        batch = kv.batch(hq)
        ws = ekv.decode_workspace(kv.pool, batch)
        want = torch.full((q.shape[0], hq, 128), float("nan"), dtype=torch.float32, device="cuda")
        ekv.attn_decode(kv.pool, batch, q, want, scale, ws)
        for out_dtype in (torch.float32, torch.bfloat16):
            got = torch.full((q.shape[0], hq, 128), float("nan"), dtype=out_dtype, device="cuda")
            print(f"noalloc decode: {name} B={q.shape[0]} Hq={hq} mode={kv.mode} out={out_dtype}", flush=True)
            ekv.attn_decode_noalloc(kv.pool, batch, q, got, scale)
            torch.cuda.synchronize()
            if out_dtype == torch.float32:
                assert torch.equal(got, want), name
            check_attention(got.float().cpu().numpy(), ref, out_dtype == torch.float32)
