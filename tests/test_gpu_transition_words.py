"""16-bit demote and refine over every word pattern, bit for bit.

At 8 KV heads one pair's two blocks hold exactly 2^16 words, so a pair
whose blocks hold a permutation of 0 .. 65535 runs every word -- NaN
payloads, infinities, subnormals, both zeros -- through the high/low byte
split (§3 opening, App. B.2: BASE is the high byte, the low byte refines it
exactly).  Each pair gets its own permutation; the pool, low bytes, freed
blocks, table and tags must equal the oracle's, and refinement must
restore every original word."""

import numpy as np
import pytest

from oracle import transitions as otr
from paper_2609_33536_amd import ekv, kvpool, workloads
from tests.gpu_util import host_safety_check, require_gpu

pytestmark = pytest.mark.gpu
PAGE = 16


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_demote_refine_every_word(dtype):
    torch = require_gpu()
    hkv = 8
    c = workloads.make_decode_case([64, 96, 64], 32, hkv, dtype=dtype, seed=61, spare_blocks=6)
    host_safety_check(c, c["pool"].shape)
    pairs = np.array([(0, 0), (0, 1), (1, 0), (1, 1), (2, 0), (2, 1)], dtype=np.int32)
    rng = np.random.default_rng(62)
    pool = c["pool"].copy()
    words_per_pair = 2 * pool[0].size
    assert words_per_pair == 1 << 16
    for s, j in pairs:
        perm = rng.permutation(1 << 16).astype(np.uint16).reshape(2, *pool.shape[1:])
        pool[c["block_table"][s, 2 * j]] = perm[0]
        pool[c["block_table"][s, 2 * j + 1]] = perm[1]
    kv = kvpool.PagedKV(pool, c["block_table"], c["seq_lens"], c["free"], hkv, dtype)
    print(f"every-word demote {dtype}: pairs={len(pairs)}", flush=True)
    freed, lo, _ = kv.demote(pairs)
    torch.cuda.synchronize()
    opool, obt, otg, ofreed, olo = otr.demote(pool, c["block_table"], c["tags"], pairs, c["seq_lens"])
    assert np.array_equal(kv.kv.cpu().numpy().view(np.uint16), opool)
    assert np.array_equal(lo.cpu().numpy().reshape(olo.shape), olo)
    assert np.array_equal(freed.cpu().numpy(), ofreed)
    assert np.array_equal(kv.bt.cpu().numpy(), obt) and np.array_equal(kv.tags.cpu().numpy(), otg)
    kv.commit()
    print(f"every-word refine {dtype}", flush=True)
    new = kv.refine(pairs, lo)
    torch.cuda.synchronize()
    rpool, rbt, rtg = otr.refine(opool, obt, otg, pairs, new, olo, c["seq_lens"])
    got = kv.kv.cpu().numpy().view(np.uint16)
    assert np.array_equal(got, rpool)
    assert np.array_equal(kv.bt.cpu().numpy(), rbt) and np.array_equal(kv.tags.cpu().numpy(), rtg)
    for s, j in pairs:
        for m in range(2):
            assert np.array_equal(got[rbt[s, 2 * j + m]], pool[c["block_table"][s, 2 * j + m]]), (s, j, m)
