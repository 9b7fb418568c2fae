"""The benchmark's algorithmic byte and flop counts (what its GB/s and
TFLOP/s divide by) against a brute-force count token by token, and its
refusal of more than one GPU.  No GPU needed."""

import subprocess
import sys
from pathlib import Path

import numpy as np

import bench

ROOT = Path(__file__).resolve().parents[1]
PAGE, D = 16, 128


def _brute_kv_bytes(seq_lens, tags, hkv):
    total = 0
    for s, length in enumerate(seq_lens):
        for t in range(int(length)):                    # every visible token once
            width = 1 if tags[s, t // PAGE] == 1 else 2  # BASE: the high byte only
            total += 2 * hkv * D * width                 # K and V of every KV head
    return total


def test_kv_and_decode_bytes_match_a_token_by_token_count():
    rng = np.random.default_rng(0)
    seq_lens = np.array([0, 1, 15, 16, 17, 32, 33, 100, 511, 1000], dtype=np.int32)
    max_blocks = 64
    tags = np.zeros((len(seq_lens), max_blocks), dtype=np.uint8)
    for s, length in enumerate(seq_lens):
        for j in range(int(length) // (2 * PAGE)):     # only pairs of two full blocks can be BASE
            if rng.random() < 0.5:
                tags[s, 2 * j] = tags[s, 2 * j + 1] = 1
    hq, hkv = 32, 8
    kv = _brute_kv_bytes(seq_lens, tags, hkv)
    assert bench.kv_bytes(seq_lens, tags, hkv) == kv
    blocks = sum(-(-int(l) // PAGE) for l in seq_lens)
    q_and_out = 2 * len(seq_lens) * hq * D * 2           # bf16 query in, bf16 output out
    lens = 4 * len(seq_lens)
    for mode, tag_bytes in ((0, 0), (1, 0), (2, blocks)):  # only the general path reads a tag per block
        want = kv + q_and_out + 4 * blocks + tag_bytes + lens
        assert bench.decode_bytes(seq_lens, tags, hq, hkv, mode) == want


def test_prefill_flops_match_a_row_by_row_count():
    prefix, chunk, nseq, hq = 40, 7, 3, 8
    flops = 0
    for _ in range(nseq):
        for i in range(chunk):
            keys = prefix + i + 1                         # causal, the diagonal included
            flops += hq * (2 * keys * D + 2 * keys * D)   # Q.K^T and P.V, a multiply and an add each
    assert bench.prefill_flops(prefix, chunk, nseq, hq) == flops


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, str(ROOT / "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""
