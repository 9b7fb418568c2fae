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


def test_pmc_reduction_scales_by_the_copy_and_follows_launch_order(tmp_path, monkeypatch):
    """Counter files written by hand: a 1 GiB copy reads FETCH_SIZE = half its
    bytes and WRITE_SIZE = its bytes; decode launches rotate over four
    fractions (the native kernel first) in dispatch order, interleaved with
    other kernels.  The reduction must scale each counter by the copy, skip
    the first round, keep the fractions apart by launch order, and average
    the roofline's traffic over the elastic launches only."""
    import csv
    import json

    kib = 1024.0
    nf, rounds = 4, 3
    fetch = [[100.0, 200.0, 300.0, 400.0][i % nf] * (1 + 0.5 * (i < nf)) for i in range(nf * rounds)]  # KiB
    write = [10.0] * (nf * rounds)
    names = ["void ekv::decode_kernel<ekv::Bf16, 4, false, 4, false, false>(ekv::DecodeArgs)"] + \
            ["void ekv::decode_kernel<ekv::Bf16, 4, true, 4, false, false>(ekv::DecodeArgs)"] * 3

    def write_run(run, counter, rows):
        d = tmp_path / f"{run}_{counter}"
        d.mkdir()
        with open(d / "run_counter_collection.csv", "w", newline="") as f:
            w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
            w.writeheader()
            for did, name, v in rows:
                w.writerow({"Dispatch_Id": did, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": v})

    for counter, vals, copy_kib in (("FETCH_SIZE", fetch, 524288.0), ("WRITE_SIZE", write, 1048576.0)):
        write_run("pmc_copy", counter, [(1, "__amd_rocclr_copyBuffer", copy_kib)])
        rows, did = [], 1
        for i, v in enumerate(vals):
            rows.append((did, "at::native::fill_kernel", 7.0))   # other kernels in between
            rows.append((did + 1, names[i % nf], v))
            did += 2
        rows.reverse()                                          # file order need not be launch order
        write_run("pmc_dec", counter, rows)
    (tmp_path / "pmc_copy_FETCH_SIZE.log").write_text(json.dumps({"copy_calibration_bytes": 1 << 30}) + "\n")
    algo = [1000.0, 2000.0, 3000.0, 4000.0]
    (tmp_path / "pmc_dec_FETCH_SIZE.log").write_text(json.dumps(
        {"decode_only_rounds": rounds, "base_fractions": [0.0, 0.25, 0.5, 1.0],
         "kernels": ["native", "elastic", "elastic", "elastic"], "bytes_per_launch": algo}) + "\n")
    out_file = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(out_file))
    bench.reduce_pmc(str(tmp_path))
    t = json.loads(out_file.read_text())
    assert abs(t["fetch_scale"] - 2.0) < 1e-9 and abs(t["write_scale"] - 1.0) < 1e-9
    want_fetch = [2 * v * kib for v in (100.0, 200.0, 300.0, 400.0)]     # first round (x1.5) skipped
    assert t["fetch_bytes"] == [round(v) for v in want_fetch]
    assert t["write_bytes"] == [round(10.0 * kib)] * 4
    hbm = [f + 10.0 * kib for f in want_fetch]
    assert t["hbm_bytes_per_launch"] == round(np.mean(hbm[1:]))
    assert t["algorithmic_bytes_per_launch"] == round(np.mean(algo[1:]))
    assert t["native"]["hbm_bytes_per_launch"] == round(hbm[0])
