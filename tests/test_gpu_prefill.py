"""GPU parity of append + chunked prefill against the float64 oracle.

Each case appends the chunk's K/V as TARGET (bit-exact against the
oracle's append), demotes BASE pairs inside the prefix (both sides, each on
its own), and runs causal prefill attention over the mixed prefix and the
chunk.  Tolerance as for decode.
"""

import numpy as np
import pytest

from oracle import attention as oatt
from oracle import transitions as otr
from paper_2609_33536_amd import ekv, kvpool, workloads
from tests import softmax_rises
from tests.gpu_util import check_attention, default_scale, host_safety_check, require_gpu, words_to_tensor

pytestmark = pytest.mark.gpu


def _run_prefill(case, hq, hkv, *, out_fp32=True, use_boundaries=True, scale=None):
    """Runs the case on the GPU and checks it against the oracle.  out_fp32
    may be a tuple of flags: the kernel then runs once per output type
    against one oracle result.  Returns (max abs err, max rel err) of the
    last run."""
    torch = require_gpu()
    flags = tuple(out_fp32) if isinstance(out_fp32, (tuple, list)) else (out_fp32,)
    scale = default_scale() if scale is None else scale
    dtype = case["dtype"]
    host_safety_check(case, case["pool"].shape)
    nb = case["pool"].shape[0]
    assert (case["slots"] >= 0).all() and (case["slots"] < nb * 16).all()
    kv = kvpool.PagedKV(case["pool"], case["block_table"], case["seq_lens"], case["free"], hkv, dtype)
    slots = torch.from_numpy(case["slots"]).cuda()
    k_new = words_to_tensor(case["k_new"], torch, dtype)
    v_new = words_to_tensor(case["v_new"], torch, dtype)
    print(f"prefill: B={len(case['seq_lens'])} Hq={hq} Hkv={hkv} rows={len(case['slots'])} "
          f"pairs={len(case['pairs'])} {dtype} fp32={out_fp32}", flush=True)
    kv.append(slots, k_new, v_new)
    opool = otr.append(case["pool"], case["slots"], case["k_new"], case["v_new"])
    torch.cuda.synchronize()
    assert np.array_equal(kv.kv.cpu().numpy().view(np.uint16), opool)
    obt, otg = case["block_table"], case["tags"]
    if len(case["pairs"]):
        kv.demote(case["pairs"])
        opool, obt, otg, _, _ = otr.demote(opool, obt, otg, case["pairs"], case["seq_lens"])
    kv.relower()
    q = words_to_tensor(case["q"], torch, dtype)
    cu = torch.from_numpy(case["cu_q"]).cuda()
    batch = kv.batch(hq, use_boundaries=use_boundaries)
    max_q = int(np.diff(case["cu_q"]).max())
    outs = []
    for fp32 in flags:
        out = torch.full((q.shape[0], hq, 128), float("nan"), dtype=torch.float32 if fp32 else q.dtype,
                         device="cuda")
        ekv.attn_prefill(kv.pool, batch, q, cu, max_q, out, scale)
        outs.append(out)
    torch.cuda.synchronize()
    ref = oatt.prefill(case["q"], case["cu_q"], opool, obt, otg, case["seq_lens"], dtype, scale)
    for fp32, out in zip(flags, outs):
        res = check_attention(out.float().cpu().numpy(), ref, fp32)
        print(f"  fp32={fp32}: max abs err {res[0]:.3e}", flush=True)
    return res


@pytest.mark.parametrize("fraction", [0.0, 0.5, 1.0])
@pytest.mark.parametrize("group", [1, 2, 4, 8, 16])
def test_prefill_groups_fractions_ragged(group, fraction):
    hkv = 2
    c = workloads.make_prefill_case([0, 17, 64, 100, 250, 33], [1, 40, 31, 7, 64, 90], hkv * group, hkv,
                                    seed=20 + group, base_fraction=fraction, spare_blocks=2)
    _run_prefill(c, hkv * group, hkv)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("out_fp32", [True, False])
def test_prefill_dtypes(dtype, out_fp32):
    c = workloads.make_prefill_case([96, 512, 1], [130, 15, 77], 16, 4, dtype=dtype, seed=31,
                                    base_fraction=0.5, spare_blocks=2)
    _run_prefill(c, 16, 4, out_fp32=out_fp32)


@pytest.mark.parametrize("prefix,chunk,fraction", [([1024, 640], [100, 37], 0.5),
                                                   ([2000, 1500, 70], [90, 300, 5], 0.8)])
def test_prefill_structured_and_general_agree(prefix, chunk, fraction):
    """The BASE run of the second case crosses the kernel's 64-block
    metadata windows (blocks 64 and 128) in both modes."""
    c = workloads.make_prefill_case(prefix, chunk, 32, 8, seed=32, base_fraction=fraction,
                                    placement="oldest", spare_blocks=2)
    _run_prefill(c, 32, 8)
    _run_prefill(c, 32, 8, use_boundaries=False)


@pytest.mark.parametrize("scale", [0.03, -0.1, 0.0, -0.0])
def test_prefill_empty_chunks_and_scales(scale):
    """A batch mixing empty chunks (a 300-token prefix with no new token), an
    empty sequence, single-token chunks and a first chunk with no prefix, at
    other softmax scales, a negative one included."""
    c = workloads.make_prefill_case([100, 0, 300, 0, 64, 1], [20, 0, 0, 5, 33, 1], 8, 2, seed=41,
                                    base_fraction=0.5, spare_blocks=4)
    _run_prefill(c, 8, 2, scale=scale)
    _run_prefill(c, 8, 2, scale=scale, use_boundaries=False)


def test_prefill_llama3_8b_chunk_full_size():
    """16 sequences x (2048-token prefix, half of its pairs BASE, + a
    512-token causal chunk), 32 query / 8 KV heads: every output checked."""
    c = workloads.make_prefill_case([2048] * 16, [512] * 16, 32, 8, seed=3, base_fraction=0.5,
                                    spare_blocks=2)
    err, rel = _run_prefill(c, 32, 8, out_fp32=(False, True))
    print(f"prefill full size: max abs err {err:.3e} (fp32 output, strict 2e-3)", flush=True)


@pytest.mark.parametrize("name", ["aligned-bf16", "aligned-fp16", "scale1-bf16-g16"])
def test_prefill_rescale_of_live_output(name):
    """Inputs whose later 32-key units rise far above the first unit's
    scores (test_rescale_inputs.py shows it from the oracle's keys), so the
    kernel rescales accumulators that already hold output; structured
    (boundaries) and general (tags) lowering, fp32 output at the strict bound
    and 16-bit output."""
    case, hq, hkv, scale, dtype = softmax_rises.make(name)
    assert dtype in ("bf16", "fp16")
    _run_prefill(case, hq, hkv, out_fp32=(True, False), scale=scale)
    _run_prefill(case, hq, hkv, out_fp32=True, scale=scale, use_boundaries=False)
