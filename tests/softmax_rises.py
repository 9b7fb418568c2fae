"""Prefill inputs on which a streaming softmax must rescale live output.

A kernel that streams keys in 32-key units keeps a running maximum of the
scores (in log2 units, s * scale * log2 e) and rescales its accumulated
output only when a unit's maximum exceeds that reference by more than a
threshold (8 log2 units in libekv's prefill).  Ordinary N(0, 1) inputs at
the default scale never get there after the first unit, so the rescale of
accumulators that already hold output is never exercised.  The cases below
are built so that it is, and :func:`score_rises` shows it on the CPU from
the oracle's own dense keys: for every query column it returns the largest
rise of a later unit's maximum over the running maximum of the units
before it (unit 0 always contributes, so the accumulator is nonzero by
then).
"""

import math

import numpy as np

from oracle import encoding, paged
from oracle import fp8 as ofp8
from oracle import transitions as otr
from paper_2609_33536_amd import workloads

UNIT = 32
LOG2E = 1.0 / math.log(2.0)

# name -> (make_prefill_case arguments, softmax scale, pool dtype)
CASES = {
    # planted keys aligned with one query (x4): that query's score jumps by tens of log2 units
    "aligned-bf16": (dict(prefix_lens=[300, 700, 1000], chunk_lens=[40, 64, 9], num_q_heads=16, num_kv_heads=4,
                          seed=51, base_fraction=0.5, aligned_keys=3, spare_blocks=4), None, "bf16"),
    "aligned-fp16": (dict(prefix_lens=[300, 700, 1000], chunk_lens=[40, 64, 9], num_q_heads=16, num_kv_heads=4,
                          dtype="fp16", seed=52, base_fraction=0.5, aligned_keys=3, spare_blocks=4), None, "fp16"),
    "aligned-e5m2": (dict(prefix_lens=[300, 700, 1000], chunk_lens=[40, 64, 9], num_q_heads=16, num_kv_heads=4,
                          dtype="e5m2", seed=53, base_fraction=0.5, aligned_keys=3, spare_blocks=4), None, "e5m2"),
    # scale 1: scores ~ N(0, 128), so later units often exceed the reference by far
    "scale1-bf16-g16": (dict(prefix_lens=[500, 130, 64], chunk_lens=[33, 70, 16], num_q_heads=32, num_kv_heads=2,
                             seed=54, base_fraction=0.5, spare_blocks=4), 1.0, "bf16"),
    "scale1-e5m2-g1": (dict(prefix_lens=[500, 130, 64], chunk_lens=[33, 70, 16], num_q_heads=4, num_kv_heads=4,
                            dtype="e5m2", seed=55, base_fraction=0.5, spare_blocks=4), 1.0, "e5m2"),
}


def make(name):
    kwargs, scale, dtype = CASES[name]
    kwargs = dict(kwargs)
    prefix, chunk = kwargs.pop("prefix_lens"), kwargs.pop("chunk_lens")
    hq, hkv = kwargs.pop("num_q_heads"), kwargs.pop("num_kv_heads")
    case = workloads.make_prefill_case(prefix, chunk, hq, hkv, **kwargs)
    return case, hq, hkv, (1.0 / math.sqrt(128) if scale is None else scale), dtype


def oracle_state(case, dtype):
    """The oracle's pool, table and tags after appending the chunk and
    demoting the case's pairs (the state the prefill runs on)."""
    mod = ofp8 if dtype == "e5m2" else otr
    pool = mod.append(case["pool"], case["slots"], case["k_new"], case["v_new"])
    bt, tags = case["block_table"], case["tags"]
    if len(case["pairs"]):
        pool, bt, tags, _, _ = mod.demote(pool, bt, tags, case["pairs"], case["seq_lens"])
    return pool, bt, tags


def score_rises(case, pool, bt, tags, scale, dtype):
    """Largest rise (log2 units) of a 32-key unit's score maximum over the
    running maximum of the earlier units, per query column: float64
    [total rows][Hq]; -inf where a column sees a single unit."""
    q = np.asarray(case["q"], dtype=np.uint16)
    qf = q.view(np.float16).astype(np.float64) if dtype == "e5m2" else encoding.words_to_f64(q, dtype)
    total, hq, _ = qf.shape
    hkv = pool.shape[2]
    group = hq // hkv
    cu, lens = case["cu_q"], case["seq_lens"]
    rises = np.full((total, hq), -np.inf)
    for s in range(len(lens)):
        r0, r1, length = int(cu[s]), int(cu[s + 1]), int(lens[s])
        n = r1 - r0
        if n == 0:
            continue
        if dtype == "e5m2":
            k, _ = ofp8.gather_sequence(pool, bt[s], tags[s], length)
        else:
            k, _ = paged.gather_sequence(pool, bt[s], tags[s], length, dtype)
        for h in range(hq):
            scores = abs(scale) * LOG2E * (qf[r0:r1, h] @ k[:, h // group, :].T)   # [n][length]
            if scale < 0:
                scores = -scores
            for i in range(n):
                lim = length - n + i + 1
                units = [scores[i, u:min(u + UNIT, lim)].max() for u in range(0, lim, UNIT)]
                run = units[0]
                best = -np.inf
                for m in units[1:]:
                    best = max(best, m - run)
                    run = max(run, m)
                rises[r0 + i, h] = best
    return rises
