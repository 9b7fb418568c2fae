#!/usr/bin/env python3
"""Benchmark of the mixed-fidelity paged-attention hot path on one MI355X.

Decode workload (Llama-3-8B-shaped layer): 64 sequences, 32 query / 8 KV
heads, head dim 128, 16-token pages, context lengths uniform in
[2048, 8192] (seed 1), bf16 K/V ~ N(0,1) with 10 outlier (head, channel)
positions per plane scaled x10.  BASE fraction swept over {0, 0.25, 0.5,
1}: BASE pairs chosen at random (f = 0 -> native path; 0.25, 0.5 ->
general elastic path; 1 -> every complete pair BASE, structured path).  One
pool per BASE fraction, each made by demoting the chosen pairs with the
library itself.

Prefill workload (same layer shape): 16 sequences, each a 2048-token
prefix with half of its pairs BASE plus a 512-token causal chunk.

One step = one pass over every hot-path operation:
  for each decode BASE fraction: append the newest token of every sequence
  as TARGET (rewriting the same values), lower the tags on the host, run
  decode attention;  append the prefill chunk's K/V and run prefill;  one
  transition round on the f=0.5 decode pool: demote 16 TARGET pairs (the
  paper's minimum demotion batch) and refine them back.

Output: one JSON line.  ``value`` = algorithmic HBM bytes of the step's
decode-attention launches / their time (GB/s, HIP events on the launch
stream); ``ms_per_step`` is the wall time of the whole step and
``step_GB_per_s`` its algorithmic bytes over that time;
``tokens_per_s_per_layer`` = decoded query tokens / decode-attention time.
``roofline`` prices the elastic decode kernel (the launches at BASE
fraction 0.25, 0.5 and 1); ``prefill`` reports its own TFLOP/s against the
dense bf16 matrix peak.  ``cpu_baseline`` times the float64 CPU oracle on a
bounded sample (every decode sequence at every BASE fraction, plus 2
prefill sequences), whose outputs also serve as a parity check of the GPU outputs of the same step.
"""

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
WORKLOAD = "llama3-8b-decode"
B, HQ, HKV, D, PAGE = 64, 32, 8, 128, 16
FRACTIONS = (0.0, 0.25, 0.5, 1.0)
ELASTIC = (1, 2, 3)          # indices of the fractions decoded by the elastic kernel
SEED = 1
TRANSITION_PAIRS = 16
PF_SEQS, PF_PREFIX, PF_CHUNK, PF_SEED = 16, 2048, 512, 3
PF_SAMPLE = 16
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_traffic.json")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy (for scaling PMC byte counters)")
    ap.add_argument("--reduce-pmc", metavar="DIR",
                    help="fold the rocprofv3 counter CSVs under DIR (pmc_dec_*, pmc_copy_* runs) "
                         "into the decode traffic summary; no GPU use")
    ap.add_argument("--decode-only", action="store_true",
                    help="only the elastic decode launches (for PMC byte counters of that kernel)")
    ap.add_argument("--prefill-only", action="store_true",
                    help="only the chunked-prefill launches (for PMC counters of that kernel)")
    ap.add_argument("--pressure-only", action="store_true",
                    help="only the pressure-transition mix (for PMC counters of demote / refine)")
    ap.add_argument("--decode-8bit-only", action="store_true",
                    help="only the 8-bit TARGET / 4-bit BASE decode leg (for counter runs)")
    ap.add_argument("--decode-70b-only", action="store_true",
                    help="only the 70B-shaped decode layer (for PMC counters of that launch)")
    ap.add_argument("--timeline", action="store_true",
                    help="per-launch time budget of the 8B decode layer from the instrumented library "
                         "(built by python -m paper_2609_33536_amd.build --timeline)")
    return ap.parse_args()


def kv_bytes(seq_lens, tags_rows, hkv):
    """Algorithmic K/V bytes: every visible element once, 2 B TARGET / 1 B BASE."""
    total = 0
    for s, length in enumerate(seq_lens):
        length = int(length)
        nblk = -(-length // PAGE)
        full = length // PAGE
        per_tok = np.where(tags_rows[s, :nblk] == 1, 1, 2).astype(np.int64) * (2 * hkv * D)
        total += int((per_tok[:full] * PAGE).sum())
        if nblk > full:
            total += int(per_tok[full]) * (length - full * PAGE)
    return total


def decode_bytes(seq_lens, tags_rows, hq, hkv, mode):
    """One decode call: K/V + Q + bf16 output + 4 B of block table per block
    (+ 1 B of tag per block on the general path)."""
    blocks = sum(-(-int(l) // PAGE) for l in seq_lens)
    qo = 2 * len(seq_lens) * hq * D * 2
    meta = blocks * 4 + (blocks if mode == 2 else 0) + len(seq_lens) * 4
    return kv_bytes(seq_lens, tags_rows, hkv) + qo + meta


def prefill_flops(prefix, chunk, nseq, hq):
    return 4 * hq * D * nseq * sum(prefix + i + 1 for i in range(chunk))


def source_digest():
    h = hashlib.sha256()
    for name in ("attn_device.h", "common.h", "decode.hip"):
        with open(os.path.join(ROOT, "paper_2609_33536_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def busy_queue(torch, stream, cycles=1 << 18):
    """Keep the GPU busy (a spin of ~0.1 ms) while the host enqueues the
    launches that follow: a leg that synchronises after every launch would
    otherwise record its start event into an idle queue, and the event time
    would include the host's call overhead as well as the GPU's work."""
    with torch.cuda.stream(stream):
        torch.cuda._sleep(cycles)


def measured_traffic():
    """HBM bytes per f=0.5 decode launch from the committed PMC summary, if it
    was taken from the current decode source."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    return t if t.get("source_digest") == source_digest() else None


def reduce_pmc(directory):
    """Scale the decode launches' FETCH_SIZE / WRITE_SIZE (KiB per dispatch)
    by what the same counters read for a 1 GiB device copy, and write the
    per-launch HBM bytes next to the algorithmic bytes of the same launches."""
    import csv

    def per_kernel(run, counter):
        path = os.path.join(directory, f"{run}_{counter}", "run_counter_collection.csv")
        vals = {}
        with open(path) as f:
            for r in csv.DictReader(f):
                vals.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]) * 1024.0)
        return vals

    def in_dispatch_order(run, counter, key):
        """Bytes of the dispatches whose kernel name contains key, in launch order."""
        path = os.path.join(directory, f"{run}_{counter}", "run_counter_collection.csv")
        rows = []
        with open(path) as f:
            for r in csv.DictReader(f):
                if key in r["Kernel_Name"]:
                    rows.append((int(r["Dispatch_Id"]), float(r["Counter_Value"]) * 1024.0))
        return [v for _, v in sorted(rows)]

    def log_json(run, key):
        with open(os.path.join(directory, f"{run}.log")) as f:
            for line in f:
                if line.startswith("{") and key in line:
                    return json.loads(line)
        raise ValueError(f"no {key} line in {run}.log")

    copy = log_json("pmc_copy_FETCH_SIZE", "copy_calibration_bytes")
    dec = log_json("pmc_dec_FETCH_SIZE", "decode_only_rounds")
    scale, per_launch = {}, {}
    for counter in ("FETCH_SIZE", "WRITE_SIZE"):
        c = [v for k, vs in per_kernel("pmc_copy", counter).items() if "copyBuffer" in k for v in vs]
        scale[counter] = copy["copy_calibration_bytes"] / (sum(c) / len(c))
        d = in_dispatch_order("pmc_dec", counter, "decode_kernel")
        nf = len(dec["base_fractions"])
        rounds = len(d) // nf
        assert rounds * nf == len(d), (counter, len(d), nf)
        # launches rotate over the fractions; skip the first round (cold)
        per_launch[counter] = [float(np.mean(d[nf + i::nf])) * scale[counter] for i in range(nf)]
    hbm = [f + w for f, w in zip(per_launch["FETCH_SIZE"], per_launch["WRITE_SIZE"])]
    # the roofline's kernel is the elastic one; the native launch (fraction 0) is listed beside it
    el = [i for i, k in enumerate(dec["kernels"]) if k == "elastic"]
    out = {"source_digest": source_digest(),
           "kernel": "decode_kernel<Bf16, 4, true, 4, false, false>",
           "base_fractions": dec["base_fractions"], "kernels": dec["kernels"],
           "fetch_scale": round(scale["FETCH_SIZE"], 5), "write_scale": round(scale["WRITE_SIZE"], 5),
           "fetch_bytes": [round(v) for v in per_launch["FETCH_SIZE"]],
           "write_bytes": [round(v) for v in per_launch["WRITE_SIZE"]],
           "algorithmic_bytes": dec["bytes_per_launch"],
           "hbm_bytes_per_launch": round(float(np.mean([hbm[i] for i in el]))),
           "algorithmic_bytes_per_launch": round(float(np.mean([dec["bytes_per_launch"][i] for i in el])))}
    if "native" in dec["kernels"]:
        i = dec["kernels"].index("native")
        out["native"] = {"hbm_bytes_per_launch": round(hbm[i]), "algorithmic_bytes_per_launch": dec["bytes_per_launch"][i],
                         "hbm_over_algorithmic": round(hbm[i] / dec["bytes_per_launch"][i], 4)}
    out["hbm_over_algorithmic"] = round(out["hbm_bytes_per_launch"] / out["algorithmic_bytes_per_launch"], 4)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out))


def copy_calibration():
    import torch
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n, "launches": 5}))


def build_decode(torch, kvpool, workloads, steps, warmup):
    rng = np.random.default_rng(SEED)
    seq_lens = workloads.seq_lens_uniform(rng, B, 2048, 8192)
    spare = TRANSITION_PAIRS * (steps + warmup + 2) + 64
    base = workloads.make_decode_case_torch(seq_lens, HQ, HKV, seed=SEED, outlier_channels=10,
                                            spare_blocks=spare)
    host = workloads.extract_sequences(base["pool"], base["block_table"], seq_lens, list(range(B)))
    host_q = base["q"].view(torch.int16).cpu().numpy().view(np.uint16)
    pools, pairs_by_f, modes = [], [], []
    for k, f in enumerate(FRACTIONS):
        pairs = workloads.choose_pairs(np.random.default_rng(SEED * 1000 + k), seq_lens, f, "random")
        kv = kvpool.PagedKV(base["pool"].clone(), base["block_table"], seq_lens, base["free"], HKV)
        if len(pairs):
            kv.demote(pairs, emit_lo=False)
            kv.commit()
        modes.append(kv.relower())
        pools.append(kv)
        pairs_by_f.append(pairs)
    # the newest token of each sequence, to be rewritten with its own values
    appends = []
    for kv in pools:
        sl = np.array([int(kv.mirror.bt[s, (int(l) - 1) // PAGE]) * PAGE + (int(l) - 1) % PAGE
                       for s, l in enumerate(seq_lens)], dtype=np.int32)
        view = kv.kv.view(-1, 2, HKV, PAGE, D)
        blk = torch.from_numpy(sl // PAGE).long().cuda()
        off = torch.from_numpy(sl % PAGE).long().cuda()
        appends.append((torch.from_numpy(sl).cuda(), view[blk, 0, :, off, :].contiguous(),
                        view[blk, 1, :, off, :].contiguous()))
    return dict(seq_lens=seq_lens, q=base["q"], pools=pools, pairs=pairs_by_f, modes=modes,
                appends=appends, host=host, host_q=host_q)


def build_prefill(torch, kvpool, workloads):
    c = workloads.make_prefill_case([PF_PREFIX] * PF_SEQS, [PF_CHUNK] * PF_SEQS, HQ, HKV, seed=PF_SEED,
                                    base_fraction=0.5, spare_blocks=2)
    kv = kvpool.PagedKV(c["pool"], c["block_table"], c["seq_lens"], c["free"], HKV)

    def to_bf16(w):
        return torch.from_numpy(np.ascontiguousarray(w).view(np.int16)).cuda().view(torch.bfloat16)

    slots = torch.from_numpy(c["slots"]).cuda()
    k_new, v_new = to_bf16(c["k_new"]), to_bf16(c["v_new"])
    kv.append(slots, k_new, v_new)
    if len(c["pairs"]):
        kv.demote(c["pairs"], emit_lo=False)
        kv.commit()
    kv.relower()
    return dict(case=c, kv=kv, slots=slots, k_new=k_new, v_new=v_new, q=to_bf16(c["q"]),
                cu=torch.from_numpy(c["cu_q"]).cuda(),
                out=torch.empty((PF_SEQS * PF_CHUNK, HQ, D), dtype=torch.bfloat16, device="cuda"))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(sharding across GPUs is not built)", file=sys.stderr)
        return 2
    if args.reduce_pmc:
        reduce_pmc(args.reduce_pmc)
        return 0
    import torch
    if args.copy_calibration:
        copy_calibration()
        return 0
    from __graft_entry__ import _ensure_built
    from paper_2609_33536_amd import ekv, kvpool, workloads
    if args.timeline:
        from paper_2609_33536_amd import build as _build
        ekv.LIB_PATH = _build.TIMELINE_LIB   # the instrumented variant, never the default
    else:
        _ensure_built()
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    scale = 1.0 / math.sqrt(D)

    if args.timeline:
        print(json.dumps(decode_timeline(torch, ekv, kvpool, workloads, stream, scale)))
        return 0
    if args.pressure_only:
        print(json.dumps({"pressure_mix": pressure_mix(torch, ekv, kvpool, workloads, stream, scale,
                                                       steps=max(1, args.steps))}))
        return 0
    if args.decode_8bit_only:
        lens = workloads.seq_lens_uniform(np.random.default_rng(SEED), B, 2048, 8192)
        print(json.dumps({"decode_8bit": decode_8bit(torch, ekv, kvpool, workloads, stream, lens, scale,
                                                     reps=max(1, args.steps))}))
        return 0
    if args.decode_70b_only:
        print(json.dumps({"decode_70b": decode_70b(torch, ekv, kvpool, workloads, stream, scale,
                                                   reps=max(1, args.steps))}))
        return 0

    if args.prefill_only:
        pf = build_prefill(torch, kvpool, workloads)
        pf_batch = pf["kv"].batch(HQ)
        for _ in range(args.warmup + args.steps):
            ekv.attn_prefill(pf["kv"].pool, pf_batch, pf["q"], pf["cu"], PF_CHUNK, pf["out"], scale)
        torch.cuda.synchronize()
        print(json.dumps({"prefill_only_launches": args.warmup + args.steps,
                          "flops_per_launch": prefill_flops(PF_PREFIX, PF_CHUNK, PF_SEQS, HQ)}))
        return 0

    print(f"[bench] building {WORKLOAD}: B={B} Hq={HQ} Hkv={HKV}", file=sys.stderr, flush=True)
    dec = build_decode(torch, kvpool, workloads, args.steps, args.warmup)
    seq_lens, q, pools = dec["seq_lens"], dec["q"], dec["pools"]
    outs = [torch.empty((B, HQ, D), dtype=torch.bfloat16, device="cuda") for _ in FRACTIONS]
    batches = [kv.batch(HQ) for kv in pools]
    ws = torch.zeros(max(ekv.decode_workspace_bytes(kv.pool, bt) for kv, bt in zip(pools, batches)),
                     dtype=torch.uint8, device="cuda")

    if args.decode_only:   # (counter runs: every fraction in rotation, the native launch included)
        for _ in range(args.warmup + args.steps):
            for k in range(len(FRACTIONS)):
                ekv.attn_decode(pools[k].pool, batches[k], q, outs[k], scale, ws)
        torch.cuda.synchronize()
        print(json.dumps({"decode_only_rounds": args.warmup + args.steps,
                          "base_fractions": list(FRACTIONS),
                          "kernels": ["elastic" if k in ELASTIC else "native" for k in range(len(FRACTIONS))],
                          "bytes_per_launch": [decode_bytes(seq_lens, pools[k].mirror.tags, HQ, HKV,
                                                            dec["modes"][k]) for k in range(len(FRACTIONS))]}))
        return 0

    print("[bench] building the prefill workload", file=sys.stderr, flush=True)
    pf = build_prefill(torch, kvpool, workloads)
    pf_batch = pf["kv"].batch(HQ)

    # transition candidates: TARGET pairs of the f=0.5 pool, newest block excluded
    tpool = pools[FRACTIONS.index(0.5)]
    trng = np.random.default_rng(SEED * 7 + 3)
    cand = []
    for s, l in enumerate(seq_lens):
        nblk = -(-int(l) // PAGE)
        for j in range(int(l) // (2 * PAGE)):
            if 2 * j + 1 < nblk - 1 and tpool.mirror.tags[s, 2 * j] == 0:
                cand.append((s, j))
    cand = np.array(cand, dtype=np.int32)

    block_bytes = 2 * HKV * PAGE * D * 2
    decode_bytes_f = [decode_bytes(seq_lens, kv.mirror.tags, HQ, HKV, m) for kv, m in zip(pools, dec["modes"])]
    pfc = pf["case"]
    pf_bytes = (kv_bytes(pfc["seq_lens"], pf["kv"].mirror.tags, HKV)
                + 2 * PF_SEQS * PF_CHUNK * HQ * D * 2 + PF_SEQS * (PF_PREFIX + PF_CHUNK) // PAGE * 4)
    step_bytes = {
        "decode": sum(decode_bytes_f),
        "append": len(FRACTIONS) * (B * 2 * HKV * D * 2 * 2 + B * 4)
                  + PF_SEQS * PF_CHUNK * (2 * HKV * D * 2 * 2 + 4),
        "prefill": pf_bytes,
        "transition": TRANSITION_PAIRS * 4 * block_bytes * 2,
    }
    total_step_bytes = sum(step_bytes.values())
    pf_flops = prefill_flops(PF_PREFIX, PF_CHUNK, PF_SEQS, HQ)
    pf_pool_bytes = pf["kv"].kv.numel() * pf["kv"].kv.element_size()

    events = []

    def step(timed):
        rec = []
        # every pool's append and re-lowering first, then the decodes back to
        # back: the host's work between a decode's start event and its launch
        # would otherwise let the queue run dry and count in the event time
        for k, kv in enumerate(pools):
            slots, kn, vn = dec["appends"][k]
            kv.append(slots, kn, vn)
            kv.relower()
        for k, kv in enumerate(pools):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            ekv.attn_decode(kv.pool, batches[k], q, outs[k], scale, ws)
            e1.record(stream)
            rec.append((e0, e1))
        pf["kv"].append(pf["slots"], pf["k_new"], pf["v_new"])
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        ekv.attn_prefill(pf["kv"].pool, pf_batch, pf["q"], pf["cu"], PF_CHUNK, pf["out"], scale)
        e1.record(stream)
        rec.append((e0, e1))
        sel = cand[trng.choice(len(cand), TRANSITION_PAIRS, replace=False)]
        sel = sel[np.lexsort((sel[:, 1], sel[:, 0]))]
        tpool.commit(wait=False)
        _, lo, _ = tpool.demote(sel)
        tpool.refine(sel, lo)
        if timed:
            events.append(rec)

    print(f"[bench] warmup {args.warmup} steps", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(True)
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps

    nf = len(FRACTIONS)
    per_ms = [float(np.mean([rec[k][0].elapsed_time(rec[k][1]) for rec in events])) for k in range(nf + 1)]
    dec_ms, pf_ms = per_ms[:nf], per_ms[nf]
    dec_gbs = step_bytes["decode"] / (sum(dec_ms) * 1e-3) / 1e9
    el_ms = [dec_ms[k] for k in ELASTIC]
    achieved = sum(decode_bytes_f[k] for k in ELASTIC) / (sum(el_ms) * 1e-3) / 1e9
    traffic = measured_traffic()
    result = {
        "metric": "mixed-fidelity decode attention: achieved HBM GB/s + tokens/s per layer",
        "value": round(dec_gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOAD, "batch": B, "num_q_heads": HQ, "num_kv_heads": HKV,
                   "head_dim": D, "page_size": PAGE, "context": "uniform[2048,8192] seed 1",
                   "sum_context_tokens": int(seq_lens.sum()), "base_fractions": list(FRACTIONS),
                   "prefill": f"{PF_SEQS} x ({PF_PREFIX} prefix, 50% BASE pairs, + {PF_CHUNK} chunk)",
                   "transition_pairs_per_step": TRANSITION_PAIRS, "parallelism": "single-gpu"},
        "tokens_per_s_per_layer": round(B * nf / (sum(dec_ms) * 1e-3), 1),
        "step_GB_per_s": round(total_step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
        "step_bytes": step_bytes,
        "decode": [{"base_fraction": f, "mode": ["native", "structured", "general"][dec["modes"][k]],
                    "ms": round(dec_ms[k], 5),
                    "GB_per_s": round(decode_bytes_f[k] / (dec_ms[k] * 1e-3) / 1e9, 1),
                    "tokens_per_s": round(B / (dec_ms[k] * 1e-3), 1),
                    "kv_tokens_per_s": round(float(np.sum(seq_lens)) / (dec_ms[k] * 1e-3), 1),
                    "realized_base_block_fraction": round(
                        float(sum(pools[k].mirror.tags[s, :-(-int(l) // PAGE)].sum()
                                  for s, l in enumerate(seq_lens))
                              / sum(-(-int(l) // PAGE) for l in seq_lens)), 4)}
                   for k, f in enumerate(FRACTIONS)],
        "prefill": {"ms": round(pf_ms, 5), "TFLOP_per_s": round(pf_flops / (pf_ms * 1e-3) / 1e12, 1),
                    "mfma_peak_frac": round(pf_flops / (pf_ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
                    "new_tokens_per_s": round(PF_SEQS * PF_CHUNK / (pf_ms * 1e-3), 1),
                    "pool_MiB": round(pf_pool_bytes / 2**20, 1),
                    "cache_resident": pf_pool_bytes < 256e6,
                    "note": "a pool under 256 MB fits the last-level cache; the kernel is bound by instruction "
                            "issue, not by memory"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": (traffic["hbm_bytes_per_launch"] if traffic else None),
                     "kernel": "decode_kernel<Bf16, 4, true, 4, false, false> (ekv_attn_decode, 16-bit elastic path)",
                     "algorithmic_bytes_per_launch": round(sum(decode_bytes_f[k] for k in ELASTIC) / len(ELASTIC)),
                     "avg_launch_ms": round(sum(el_ms) / len(el_ms), 5)},
    }
    if traffic:
        result["roofline"]["traffic_note"] = (
            "mean over the f=0.25/0.5/1 launches of PMC FETCH_SIZE and WRITE_SIZE, each scaled by "
            "what it reads for a 1 GiB device copy")
    result["native_dispatch"] = native_dispatch(torch, ekv, pools[FRACTIONS.index(0.0)], q, outs[0], scale, stream)
    result["decode_append"] = decode_append(torch, ekv, pools[FRACTIONS.index(0.5)], q, scale, stream)
    print("[bench] 70B-shaped decode layer", file=sys.stderr, flush=True)
    result["decode_70b"] = decode_70b(torch, ekv, kvpool, workloads, stream, scale)
    result["controller"] = controller_cost(ekv, tpool.mirror)
    print("[bench] 8-bit TARGET / 4-bit BASE decode", file=sys.stderr, flush=True)
    result["decode_8bit"] = decode_8bit(torch, ekv, kvpool, workloads, stream, seq_lens, scale)
    print("[bench] 8-bit TARGET / 4-bit BASE prefill", file=sys.stderr, flush=True)
    result["prefill_8bit"] = prefill_8bit(torch, ekv, kvpool, workloads, stream, scale)
    print("[bench] asynchronous promotion", file=sys.stderr, flush=True)
    result["async_promotion"] = async_promotion_cost(torch, kvpool, tpool, cand, stream)
    print("[bench] multi-layer transitions", file=sys.stderr, flush=True)
    result["transitions_all_layers"] = transitions_all_layers(torch, ekv, stream)
    print("[bench] pressure-transition mix", file=sys.stderr, flush=True)
    result["pressure_mix"] = pressure_mix(torch, ekv, kvpool, workloads, stream, scale)
    if not args.no_cpu_baseline:
        print("[bench] cpu_baseline: float64 oracle on the sample", file=sys.stderr, flush=True)
        result["cpu_baseline"], result["parity"] = cpu_baseline(dec, outs, pf)
    print(json.dumps(result), flush=True)
    return 0


def native_dispatch(torch, ekv, kv, q, out, scale, stream, reps=30):
    """The f=0 decode launch as dispatched (native path: no tag or range is
    read) against the same launch forced through the elastic kernel
    (general mode, every tag read), alternating; median event times.  The
    native path is meant to cost nothing: native <= 1.02 x forced."""
    native = kv.batch(HQ)
    forced = kv.batch(HQ, mode=ekv.MODE_GENERAL, use_boundaries=False)
    ws = torch.zeros(max(ekv.decode_workspace_bytes(kv.pool, b) for b in (native, forced)), dtype=torch.uint8,
                     device="cuda")
    times = {"native": [], "elastic": []}
    for r in range(reps + 3):
        for name, b in (("native", native), ("elastic", forced)):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            ekv.attn_decode(kv.pool, b, q, out, scale, ws)
            e1.record(stream)
            if r >= 3:
                times[name].append((e0, e1))
    torch.cuda.synchronize()
    med = {k: float(np.median([a.elapsed_time(b) for a, b in v])) for k, v in times.items()}
    return {"native_ms": round(med["native"], 5), "elastic_forced_ms": round(med["elastic"], 5),
            "ratio": round(med["native"] / med["elastic"], 4), "acceptance": "ratio <= 1.02"}


def decode_append(torch, ekv, kv, q, scale, stream, reps=30):
    """Append each sequence's newest token and decode, on the 8B layer at BASE
    fraction 0.5: ekv_append_kv then ekv_attn_decode, against the one launch
    of ekv_attn_decode_append (alternating; median event times around each).
    Both write the same rows, so the pool's contents do not change between
    repetitions."""
    gen = torch.Generator(device="cuda")
    gen.manual_seed(SEED + 11)
    k_new = torch.randn((B, HKV, D), generator=gen, device="cuda").to(torch.bfloat16)
    v_new = torch.randn((B, HKV, D), generator=gen, device="cuda").to(torch.bfloat16)
    lens = kv.mirror.seq_lens
    slots = torch.tensor([int(kv.mirror.bt[s, (int(l) - 1) // PAGE]) * PAGE + (int(l) - 1) % PAGE
                          for s, l in enumerate(lens)], dtype=torch.int32, device="cuda")
    batch = kv.batch(HQ)
    ws = ekv.decode_workspace(kv.pool, batch)
    out = torch.empty((B, HQ, D), dtype=torch.bfloat16, device="cuda")
    two, one = [], []
    for r in range(reps + 3):
        for fused in (False, True):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            busy_queue(torch, stream)
            e0.record(stream)
            if fused:
                ekv.attn_decode_append(kv.pool, batch, q, k_new, v_new, out, scale, ws)
            else:
                ekv.append_kv(kv.pool, slots, k_new, v_new)
                ekv.attn_decode(kv.pool, batch, q, out, scale, ws)
            e1.record(stream)
            e1.synchronize()
            if r >= 3:
                (one if fused else two).append(e0.elapsed_time(e1))
    return {"workload": "8B decode layer at BASE fraction 0.5 (general), newest token of each of the 64 "
                        "sequences appended",
            "append_then_decode_ms": round(float(np.median(two)), 5),
            "fused_ms": round(float(np.median(one)), 5),
            "saved_ms": round(float(np.median(two)) - float(np.median(one)), 5)}


def _timeline_stats(torch, lib, launch, stream, reps, first_slot):
    """Median over `reps` launches of the per-workgroup timeline statistics
    (after two warm-up launches); first_slot: workgroups below this index
    hold the first wave slot of their SIMD (0: no split reported)."""
    rows = []
    for rep in range(reps + 2):
        lib.ekv_timeline_clear()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        busy_queue(torch, stream)
        e0.record(stream)
        launch()
        e1.record(stream)
        torch.cuda.synchronize()
        host = np.zeros(8 * 8192, dtype=np.uint64)
        lib.ekv_timeline_read(host.ctypes.data, host.size)
        t = host.reshape(-1, 8).astype(np.int64)
        idx = np.nonzero(t[:, 7] == 1)[0]   # record w belongs to workgroup w
        t = t[idx]
        t0 = t[:, 0].min()
        start, first, stream_end, end = ((t[:, c] - t0) / 100.0 for c in range(4))
        xcc = t[:, 6] & 0xF
        merged = t[:, 5] > 0
        if rep >= 2:
            r = {"event_us": e0.elapsed_time(e1) * 1e3, "workgroups": len(t),
                 "start_skew_us": float(start.max()),
                 "first_slot_after_start_us": float(np.median(first - start)),
                 "first_slot_after_start_max_us": float((first - start).max()),
                 "stream_end_p50_us": float(np.median(stream_end)),
                 "stream_end_p90_us": float(np.percentile(stream_end, 90)),
                 "stream_end_max_us": float(stream_end.max()),
                 "end_max_us": float(end.max()),
                 "merge_us_p50": float(np.median((end - stream_end)[merged])) if merged.any() else 0.0,
                 "merge_us_max": float((end - stream_end)[merged].max()) if merged.any() else 0.0,
                 "xcd_mean_stream_end_us": [float(stream_end[xcc == x].mean()) for x in range(8)]}
            if first_slot:
                lo = idx < first_slot
                r["stream_end_p50_first_slot_us"] = float(np.median(stream_end[lo]))
                r["stream_end_p50_second_slot_us"] = float(np.median(stream_end[~lo]))
                r["pairs_first_slot"] = int(np.median(t[lo, 4]))
                r["pairs_second_slot"] = int(np.median(t[~lo, 4]))
            rows.append(r)
    med = {key: (round(float(np.median([r[key] for r in rows])), 1) if not isinstance(rows[0][key], list)
                 else [round(float(np.median([r[key][x] for r in rows])), 1) for x in range(8)])
           for key in rows[0]}
    med["outside_workgroups_us"] = round(med["event_us"] - med["end_max_us"], 1)
    return med


def decode_timeline(torch, ekv, kvpool, workloads, stream, scale, reps=5):
    """Where the time of one 8B decode launch goes, per BASE fraction, from
    the instrumented library's per-workgroup timestamps (100 MHz constant
    clock, relative to the first workgroup's start): workgroup start skew,
    first K/V slot after start, end of each workgroup's stream, end of its
    merges, and the mean stream end per XCD; next to the launch's HIP-event
    time.  Median over `reps` launches of each statistic.  Also the same
    layer over an 8-bit pool at BASE fraction 0.5 and 1 (two waves per
    SIMD: the stream ends of the first-slot and second-slot workgroups)."""
    import ctypes
    lib = ekv.lib()
    lib.ekv_timeline_read.argtypes = [ctypes.c_void_p, ctypes.c_int]
    dec = build_decode(torch, kvpool, workloads, 2, 2)
    q = dec["q"]
    out = torch.empty((B, HQ, D), dtype=torch.bfloat16, device="cuda")
    res = []
    for k, kv in enumerate(dec["pools"]):
        b = kv.batch(HQ)
        ws = ekv.decode_workspace(kv.pool, b)
        med = _timeline_stats(torch, lib, lambda: ekv.attn_decode(kv.pool, b, q, out, scale, ws), stream, reps, 0)
        res.append({"base_fraction": FRACTIONS[k], "mode": ["native", "structured", "general"][dec["modes"][k]],
                    "algorithmic_bytes": decode_bytes(dec["seq_lens"], kv.mirror.tags, HQ, HKV, dec["modes"][k]),
                    **med})
        del ws
    seq_lens = dec["seq_lens"]
    del dec
    torch.cuda.empty_cache()
    # the 8-bit pool of the decode_8bit leg (same inputs)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    base = workloads.make_decode_case_torch(seq_lens, HQ, HKV, seed=SEED + 5, outlier_channels=10,
                                            spare_blocks=64, dtype="e5m2")
    out8 = torch.empty((B, HQ, D), dtype=torch.float16, device="cuda")
    res8 = []
    for k, f in ((1, 0.5), (2, 1.0)):
        kv = kvpool.PagedKV(base["pool"].clone(), base["block_table"], seq_lens, base["free"], HKV, "e5m2")
        pairs = workloads.choose_pairs(np.random.default_rng(SEED * 2000 + k), seq_lens, f, "random")
        kv.demote(pairs, emit_lo=False)
        kv.commit()
        mode = kv.relower()
        b = kv.batch(HQ)
        ws = ekv.decode_workspace(kv.pool, b)
        med = _timeline_stats(torch, lib, lambda: ekv.attn_decode(kv.pool, b, base["q"], out8, scale, ws), stream,
                              reps, 4 * cus)
        res8.append({"base_fraction": f, "mode": ["native", "structured", "general"][mode], **med})
        del ws, kv
    return {"decode_timeline": res, "decode_timeline_8bit": res8,
            "library": "libekv_timeline.so (timestamps in the decode kernel)"}


def decode_70b(torch, ekv, kvpool, workloads, stream, scale, reps=20):
    """A Llama-3-70B-shaped decode layer: 256 sequences of 4096 tokens, 64
    query / 8 KV heads, the oldest half of every sequence's pairs BASE
    (structured), and the same launch forced through general mode (per-block
    tags); median event times, algorithmic bytes as for the 8B layer."""
    bsz, hq, length = 256, 64, 4096
    seq_lens = np.full(bsz, length, dtype=np.int32)
    case = workloads.make_decode_case_torch(seq_lens, hq, HKV, seed=2, spare_blocks=64)
    pairs = workloads.choose_pairs(np.random.default_rng(2), seq_lens, 0.5, "oldest")
    kv = kvpool.PagedKV(case["pool"], case["block_table"], seq_lens, case["free"], HKV)
    kv.demote(pairs, emit_lo=False)
    kv.commit()
    mode = kv.relower()
    out = torch.empty((bsz, hq, D), dtype=torch.bfloat16, device="cuda")
    res = {"workload": f"{bsz} x {length} tokens, {hq}/{HKV} heads, oldest half of the pairs BASE"}
    for name, b in (("structured", kv.batch(hq)), ("general", kv.batch(hq, mode=ekv.MODE_GENERAL,
                                                                        use_boundaries=False))):
        ws = ekv.decode_workspace(kv.pool, b)
        times = []
        for r in range(reps + 3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            ekv.attn_decode(kv.pool, b, case["q"], out, scale, ws)
            e1.record(stream)
            if r >= 3:
                times.append((e0, e1))
        torch.cuda.synchronize()
        ms = float(np.median([a.elapsed_time(c) for a, c in times]))
        nbytes = decode_bytes(seq_lens, kv.mirror.tags, hq, HKV, 2 if name == "general" else mode)
        res[name] = {"ms": round(ms, 5), "GB_per_s": round(nbytes / (ms * 1e-3) / 1e9, 1),
                     "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4), "bytes": nbytes,
                     "tokens_per_s": round(bsz / (ms * 1e-3), 1),
                     "kv_tokens_per_s": round(float(np.sum(seq_lens)) / (ms * 1e-3), 1)}
        del ws
    del kv, case
    torch.cuda.empty_cache()
    return res


def decode_8bit(torch, ekv, kvpool, workloads, stream, seq_lens, scale, reps=20):
    """The same 8B decode layer over an 8-bit TARGET (FP8 E5M2) / 4-bit BASE
    pool at BASE fraction 0, 0.5 and 1 (random pairs): median event time of
    the decode launch; algorithmic bytes count 1 B per TARGET and 0.5 B per
    BASE element of every visible token, fp16 Q and O, and the metadata."""
    base = workloads.make_decode_case_torch(seq_lens, HQ, HKV, seed=SEED + 5, outlier_channels=10,
                                            spare_blocks=64, dtype="e5m2")
    q = base["q"]
    out = torch.empty((B, HQ, D), dtype=torch.float16, device="cuda")
    res = []
    for k, f in enumerate((0.0, 0.5, 1.0)):
        kv = kvpool.PagedKV(base["pool"].clone(), base["block_table"], seq_lens, base["free"], HKV, "e5m2")
        pairs = workloads.choose_pairs(np.random.default_rng(SEED * 2000 + k), seq_lens, f, "random")
        if len(pairs):
            kv.demote(pairs, emit_lo=False)
            kv.commit()
        mode = kv.relower()
        batch = kv.batch(HQ)
        ws = torch.zeros(ekv.decode_workspace_bytes(kv.pool, batch), dtype=torch.uint8, device="cuda")
        times = []
        for r in range(reps + 3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            busy_queue(torch, stream)
            e0.record(stream)
            ekv.attn_decode(kv.pool, batch, q, out, scale, ws)
            e1.record(stream)
            e1.synchronize()
            if r >= 3:
                times.append(e0.elapsed_time(e1))
        ms = float(np.median(times))
        tags = kv.mirror.tags
        nbytes = 0
        for s, length in enumerate(seq_lens):
            nblk = -(-int(length) // PAGE)
            per_tok = np.where(tags[s, :nblk] == 1, 0.5, 1.0) * (2 * HKV * D)
            full = int(length) // PAGE
            nbytes += int((per_tok[:full] * PAGE).sum()) + (
                int(per_tok[full] * (int(length) - full * PAGE)) if nblk > full else 0)
        blocks = sum(-(-int(l) // PAGE) for l in seq_lens)
        nbytes += 2 * B * HQ * D * 2 + blocks * 4 + (blocks if mode == 2 else 0) + B * 4
        res.append({"base_fraction": f, "mode": ["native", "structured", "general"][mode], "ms": round(ms, 5),
                    "GB_per_s": round(nbytes / (ms * 1e-3) / 1e9, 1), "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                    "tokens_per_s": round(B / (ms * 1e-3), 1),
                    "kv_tokens_per_s": round(float(np.sum(seq_lens)) / (ms * 1e-3), 1), "bytes": nbytes})
        del kv, ws
    del base
    torch.cuda.empty_cache()
    return res


def prefill_8bit(torch, ekv, kvpool, workloads, stream, scale, reps=20):
    """The prefill workload of the main step (16 x (2048-token prefix, half of
    its pairs BASE, + 512-token chunk), 32 query / 8 KV heads) over an 8-bit
    TARGET (FP8 E5M2) / 4-bit BASE pool with FP16 queries and outputs: median
    event time of the prefill launch; its products run on FP16 matrix cores,
    so the peak is the dense FP16 one."""
    c = workloads.make_prefill_case([PF_PREFIX] * PF_SEQS, [PF_CHUNK] * PF_SEQS, HQ, HKV, dtype="e5m2",
                                    seed=PF_SEED, base_fraction=0.5, spare_blocks=2)
    kv = kvpool.PagedKV(c["pool"], c["block_table"], c["seq_lens"], c["free"], HKV, "e5m2")
    kv.append(torch.from_numpy(c["slots"]).cuda(), torch.from_numpy(np.ascontiguousarray(c["k_new"])).cuda(),
              torch.from_numpy(np.ascontiguousarray(c["v_new"])).cuda())
    if len(c["pairs"]):
        kv.demote(c["pairs"], emit_lo=False)
        kv.commit()
    kv.relower()
    batch = kv.batch(HQ)
    q = torch.from_numpy(np.ascontiguousarray(c["q"]).view(np.int16)).cuda().view(torch.float16)
    cu = torch.from_numpy(c["cu_q"]).cuda()
    out = torch.empty((PF_SEQS * PF_CHUNK, HQ, D), dtype=torch.float16, device="cuda")
    times = []
    for r in range(reps + 3):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        busy_queue(torch, stream)
        e0.record(stream)
        ekv.attn_prefill(kv.pool, batch, q, cu, PF_CHUNK, out, scale)
        e1.record(stream)
        e1.synchronize()
        if r >= 3:
            times.append(e0.elapsed_time(e1))
    ms = float(np.median(times))
    flops = prefill_flops(PF_PREFIX, PF_CHUNK, PF_SEQS, HQ)
    del kv, q, out
    torch.cuda.empty_cache()
    return {"ms": round(ms, 5), "TFLOP_per_s": round(flops / (ms * 1e-3) / 1e12, 1),
            "mfma_peak_frac": round(flops / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
            "new_tokens_per_s": round(PF_SEQS * PF_CHUNK / (ms * 1e-3), 1),
            "base_pairs": int(len(c["pairs"])), "dtype": "e5m2 KV, fp16 q/out"}


def async_promotion_cost(torch, kvpool, kv, cand, stream, pairs=256):
    """Asynchronous promotion (App. B.2) of 256 pairs of the f=0.5 8B pool:
    their refinement bytes (one 64 KiB block each, 16 MiB in all) are backed
    up to pinned host memory at demotion; promotion then reserves the new
    blocks and copies the backing into them on the copy stream (one kernel
    reading the pinned memory over the host link), and the staged
    refinement publishes them.  Reported: host time to issue the promotion
    (address checks included), the copy kernel's duration on the copy stream
    (events just around it), and the host time of the publication after the
    copy."""
    eng = kvpool.AsyncPromotion(kv)
    rng = np.random.default_rng(SEED * 13)
    kv.commit(wait=True)
    sel = cand[np.sort(rng.choice(len(cand), pairs, replace=False))]
    sel = sel[np.lexsort((sel[:, 1], sel[:, 0]))]
    eng.demote(sel, stream)
    torch.cuda.synchronize()
    kv.commit(wait=True)
    t0 = time.perf_counter()
    eng.promote(sel)
    t1 = time.perf_counter()
    c0, c1 = eng.last_copy
    c1.synchronize()
    t2 = time.perf_counter()
    eng.publish(wait=True, stream=stream)
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    assert int(kv.mirror.tags[sel[:, 0], 2 * sel[:, 1]].sum()) == 0
    copy_ms = c0.elapsed_time(c1)
    nbytes = pairs * kv.block_bytes
    return {"pairs": pairs, "bytes": nbytes, "issue_ms": round((t1 - t0) * 1e3, 3),
            "copy_ms": round(copy_ms, 3), "copy_GB_per_s": round(nbytes / (copy_ms * 1e-3) / 1e9, 1),
            "publish_ms": round((t3 - t2) * 1e3, 3)}


def transitions_all_layers(torch, ekv, stream, layers=32, pairs=TRANSITION_PAIRS, reps=20):
    """One demotion batch of the paper's size (16 pairs, App. B.1) across all
    32 layers of the 8B model in one launch, then its refinement: 32 pools of
    1024 blocks (2 GiB in all, so successive batches miss the caches), pairs
    drawn at random from 16 sequences x 64 blocks.  Per pair and layer both
    directions move 4 block-equivalents (256 KiB at 8 KV heads)."""
    nb, nseq = 1024, 16
    block_bytes = 2 * HKV * PAGE * D * 2
    pools = [torch.empty(nb * block_bytes // 2, dtype=torch.int16, device="cuda") for _ in range(layers)]
    layer_kv = torch.tensor([p.data_ptr() for p in pools], dtype=torch.int64, device="cuda")
    pool = ekv.make_pool(pools[0], HKV, "bf16")
    bt_h = np.arange(nb, dtype=np.int32).reshape(nseq, nb // nseq)
    bt = torch.from_numpy(bt_h.copy()).cuda()
    tags = torch.zeros(bt_h.shape, dtype=torch.uint8, device="cuda")
    freed = torch.empty(pairs, dtype=torch.int32, device="cuda")
    lo = torch.empty((pairs, layers, block_bytes), dtype=torch.uint8, device="cuda")
    rng = np.random.default_rng(SEED * 11)
    all_pairs = np.array([(s, j) for s in range(nseq) for j in range(nb // nseq // 2)], dtype=np.int32)
    times = []
    for r in range(reps + 2):
        sel = all_pairs[np.sort(rng.choice(len(all_pairs), pairs, replace=False))]
        pairs_d = torch.from_numpy(sel).cuda()
        member1 = torch.from_numpy(bt_h[sel[:, 0], 2 * sel[:, 1] + 1].copy()).cuda()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ev[0].record(stream)
        ekv.demote_layers(pool, layer_kv, pairs_d, bt, tags, freed, lo)
        ev[1].record(stream)
        ekv.refine_layers(pool, layer_kv, pairs_d, member1, bt, tags, lo)
        ev[2].record(stream)
        torch.cuda.synchronize()
        if r >= 2:
            times.append((ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2])))
    assert np.array_equal(bt.cpu().numpy(), bt_h) and int(tags.sum()) == 0
    d_ms, r_ms = (float(np.median([t[k] for t in times])) for k in range(2))
    moved = 4 * block_bytes * pairs * layers
    del pools, lo
    return {"layers": layers, "pairs": pairs, "bytes_each_way": moved,
            "demote_ms": round(d_ms, 4), "demote_GB_per_s": round(moved / (d_ms * 1e-3) / 1e9, 1),
            "refine_ms": round(r_ms, 4), "refine_GB_per_s": round(moved / (r_ms * 1e-3) / 1e9, 1),
            "paper_sync_demotion_ms": 25.44}


def pressure_mix(torch, ekv, kvpool, workloads, stream, scale, steps=20):
    """The pressure-transition mix: an 8B-shaped pool of 200,000 blocks
    (13.1 GB), 128 sequences with context uniform in [1024, 16384] (seed 4).
    Each step demotes a random 10 % of the TARGET pairs (with their
    refinement bytes, kept in device memory), then refines a random 5 % of
    the BASE pairs (sampled after that demotion; new blocks from the free
    FIFO), then decodes the whole batch.  Host planning and uploads are
    outside the timed regions; each launch is timed with HIP events on the
    launch stream, queued behind a short GPU spin (busy_queue).  Algorithmic bytes: 4 block-equivalents per demoted pair
    (2 blocks read, the packed block and the low bytes written) and per
    refined pair (packed block and low bytes read, 2 blocks written), plus
    the lists and table updates; decode as for the 8B layer."""
    nb, bsz, hq = 200_000, 128, 32
    rng = np.random.default_rng(4)
    seq_lens = workloads.seq_lens_uniform(rng, bsz, 1024, 16384)
    used = sum(-(-int(l) // PAGE) for l in seq_lens)
    case = workloads.make_decode_case_torch(seq_lens, hq, HKV, seed=4, spare_blocks=nb - used)
    kv = kvpool.PagedKV(case["pool"], case["block_table"], seq_lens, case["free"], HKV)
    del case["pool"]
    q = case["q"]
    out = torch.empty((bsz, hq, D), dtype=torch.bfloat16, device="cuda")
    block_bytes = kv.block_bytes
    full_pairs = [int(l) // (2 * PAGE) for l in seq_lens]
    pair_s = np.concatenate([np.full(n, s, dtype=np.int32) for s, n in enumerate(full_pairs)])
    pair_j = np.concatenate([np.arange(n, dtype=np.int32) for n in full_pairs])
    lo_store = {}
    srng = np.random.default_rng(44)
    ws = None

    def upload(a):
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()

    def timed(fn):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        busy_queue(torch, stream)
        e0.record(stream)
        fn()
        e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1)

    rows = []
    for step in range(steps):
        tg = kv.mirror.tags[pair_s, 2 * pair_j]
        tp = np.nonzero(tg == 0)[0]
        nd = int(0.1 * len(tp))
        dsel = np.sort(srng.choice(tp, nd, replace=False))
        dp = np.stack([pair_s[dsel], pair_j[dsel]], axis=1).astype(np.int32)
        host_freed = kv.mirror.plan_demote(dp)
        pairs_d, freed = upload(dp), torch.empty(nd, dtype=torch.int32, device="cuda")
        lo = torch.empty((nd, block_bytes), dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        d_ms = timed(lambda: ekv.demote(kv.pool, pairs_d, kv.bt, kv.tags, freed, lo))
        kv.mirror.commit_freed(host_freed)
        for i, k in enumerate(dsel.tolist()):
            lo_store[k] = (lo, i)
        tg = kv.mirror.tags[pair_s, 2 * pair_j]
        bp = np.nonzero(tg == 1)[0]
        nr = int(0.05 * len(bp))
        rsel = np.sort(srng.choice(bp, nr, replace=False))
        rp = np.stack([pair_s[rsel], pair_j[rsel]], axis=1).astype(np.int32)
        new = kv.mirror.plan_refine(rp)
        lo_in = torch.stack([lo_store[k][0][lo_store[k][1]] for k in rsel.tolist()])
        for k in rsel.tolist():
            del lo_store[k]
        rpairs_d, new_d = upload(rp), upload(new)
        torch.cuda.synchronize()
        r_ms = timed(lambda: ekv.refine(kv.pool, rpairs_d, new_d, kv.bt, kv.tags, lo_in))
        mode = kv.relower()
        batch = kv.batch(hq)
        if ws is None:
            ws = torch.zeros(ekv.decode_workspace_bytes(kv.pool, batch), dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        c_ms = timed(lambda: ekv.attn_decode(kv.pool, batch, q, out, scale, ws))
        dbytes = nd * (4 * block_bytes + 8 + 8 + 2 + 4)
        rbytes = nr * (4 * block_bytes + 8 + 4 + 4 + 2)
        cbytes = decode_bytes(seq_lens, kv.mirror.tags, hq, HKV, mode)
        rows.append({"step": step, "demoted_pairs": nd, "refined_pairs": nr,
                     "base_block_fraction": round(float(kv.mirror.tags[pair_s, 2 * pair_j].mean()), 4),
                     "mode": ["native", "structured", "general"][mode],
                     "demote_ms": round(d_ms, 4), "demote_GB_per_s": round(dbytes / (d_ms * 1e-3) / 1e9, 1),
                     "demote_pairs_per_s": round(nd / (d_ms * 1e-3), 1),
                     "refine_ms": round(r_ms, 4), "refine_GB_per_s": round(rbytes / (r_ms * 1e-3) / 1e9, 1),
                     "refine_pairs_per_s": round(nr / (r_ms * 1e-3), 1),
                     "decode_ms": round(c_ms, 4), "decode_GB_per_s": round(cbytes / (c_ms * 1e-3) / 1e9, 1)})
    del kv, lo_store, ws
    torch.cuda.empty_cache()
    med = {k: round(float(np.median([r[k] for r in rows])), 1)
           for k in ("demote_GB_per_s", "refine_GB_per_s", "decode_GB_per_s")}
    return {"workload": f"{nb} blocks (13.1 GB), {bsz} sequences with context uniform[1024,16384] seed 4, "
                        f"{hq}/{HKV} heads; per step: demote 10% of TARGET pairs (with refinement bytes), "
                        "refine 5% of BASE pairs, decode the batch",
            "steps": steps, "median": med, "per_step": rows}


def controller_cost(ekv, mirror, reps=200):
    """Host time of one control step (ekv_ctrl_demotion + ekv_ctrl_promotion,
    Alg. 1) over the 8B workload's host mirror at f=0.5: a shortage of 2
    blocks (so B_min = 16 pairs are demoted) and a promotion budget of 16;
    and of the dispatch-metadata lowering (ekv_lower) of that mirror.
    Arrays are marshalled once; the figures are the library's own work."""
    import ctypes
    cfg = ekv.ctrl_config(min_batch=16, decay=2, sink_pairs=1, recent_pairs=2)
    tags = np.ascontiguousarray(mirror.tags, dtype=np.uint8)
    lens = np.ascontiguousarray(mirror.seq_lens, dtype=np.int32)
    bsz, max_blocks = tags.shape
    cap = bsz * (max_blocks // 2)
    out = np.zeros((cap, 2), dtype=np.int32)
    tp, lp, op = (x.ctypes.data_as(ctypes.c_void_p) for x in (tags, lens, out))
    n_d, n_p = ctypes.c_int32(0), ctypes.c_int32(0)
    lib = ekv.lib()
    t0 = time.perf_counter()
    for _ in range(reps):
        st = ekv.CtrlState()
        lib.ekv_ctrl_demotion(ctypes.byref(cfg), ctypes.byref(st), 10, 8, tp, lp, None, bsz, max_blocks, PAGE,
                              op, cap, ctypes.byref(n_d))
        lib.ekv_ctrl_promotion(ctypes.byref(cfg), ctypes.byref(st), st.surplus + 16, 64, tp, lp, bsz,
                               max_blocks, PAGE, op, cap, ctypes.byref(n_p))
    us = (time.perf_counter() - t0) * 1e6 / reps
    # the dispatch-metadata lowering of the same mirror (ekv_lower: mode and boundaries)
    bounds = np.zeros((bsz, 2), dtype=np.int32)
    bp = bounds.ctypes.data_as(ctypes.c_void_p)
    mode = ctypes.c_int32(-1)
    t0 = time.perf_counter()
    for _ in range(reps):
        lib.ekv_lower(tp, lp, bsz, max_blocks, PAGE, ctypes.byref(mode), bp)
    lower_us = (time.perf_counter() - t0) * 1e6 / reps
    return {"host_us_per_step": round(us, 1), "demoted_pairs": n_d.value, "promoted_pairs": n_p.value,
            "sequences": int(bsz), "lowering_us_per_step": round(lower_us, 2),
            "note": "shortage 2 blocks, B_min 16, lambda 2, budget 16; lowering = ekv_lower of the same mirror"}


def cpu_baseline(dec, outs, pf):
    from threadpoolctl import threadpool_limits

    from oracle import attention as oatt
    from oracle import transitions as otr
    host_pool, host_bt, host_lens = dec["host"]
    tags0 = np.zeros(host_bt.shape, dtype=np.uint8)
    seconds, nbytes, worst = 0.0, 0, 0.0

    def excess(got, ref):
        return float((np.abs(got - ref) - (2e-3 + 1e-2 * np.abs(ref))).max())

    with threadpool_limits(limits=1):
        for k, f in enumerate(FRACTIONS):
            pairs = dec["pairs"][k]
            t0 = time.perf_counter()
            pool, bt, tg = host_pool, host_bt, tags0
            if len(pairs):
                pool, bt, tg, _, _ = otr.demote(pool, bt, tg, pairs, host_lens)
            ref = oatt.decode(dec["host_q"], pool, bt, tg, host_lens)
            seconds += time.perf_counter() - t0
            nbytes += decode_bytes(host_lens, tg, HQ, HKV, 2 if len(pairs) else 0)
            got = outs[k].float().cpu().numpy()
            worst = max(worst, excess(got, ref))
            print(f"[bench] parity decode f={f}: max|gpu-oracle| = {np.abs(got - ref).max():.3e}",
                  file=sys.stderr, flush=True)
        c = pf["case"]
        rows = PF_SAMPLE * PF_CHUNK
        sub_pairs = c["pairs"][c["pairs"][:, 0] < PF_SAMPLE]
        t0 = time.perf_counter()
        pool = otr.append(c["pool"], c["slots"][:rows], c["k_new"][:rows], c["v_new"][:rows])
        bt, tg = c["block_table"], c["tags"]
        if len(sub_pairs):
            pool, bt, tg, _, _ = otr.demote(pool, bt, tg, sub_pairs, c["seq_lens"])
        ref = oatt.prefill(c["q"][:rows], c["cu_q"][:PF_SAMPLE + 1], pool, bt[:PF_SAMPLE], tg[:PF_SAMPLE],
                           c["seq_lens"][:PF_SAMPLE])
        seconds += time.perf_counter() - t0
        nbytes += kv_bytes(c["seq_lens"][:PF_SAMPLE], tg[:PF_SAMPLE], HKV) + 2 * rows * HQ * D * 2
        got = pf["out"][:rows].float().cpu().numpy()
        worst = max(worst, excess(got, ref))
        print(f"[bench] parity prefill: max|gpu-oracle| = {np.abs(got - ref).max():.3e}", file=sys.stderr,
              flush=True)
    # the same oracle with every host core available to BLAS, on the f=0.5 decode
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    k = FRACTIONS.index(0.5)
    with threadpool_limits(limits=cores):
        t0 = time.perf_counter()
        pool, bt, tg, _, _ = otr.demote(host_pool, host_bt, tags0, dec["pairs"][k], host_lens)
        oatt.decode(dec["host_q"], pool, bt, tg, host_lens)
        all_s = time.perf_counter() - t0
    all_cores = {"value": round(decode_bytes(host_lens, tg, HQ, HKV, 2) / all_s / 1e9, 4), "unit": "GB/s",
                 "cores": cores, "sample": f"decode of all {B} sequences at BASE fraction 0.5",
                 "seconds": round(all_s, 2)}
    cb = {"value": round(nbytes / seconds / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
          "sample": f"decode: all {B} sequences at each BASE fraction {list(FRACTIONS)}; prefill: "
                    f"{PF_SAMPLE} of {PF_SEQS} sequences (oracle append/demote/attention, float64, "
                    f"1 BLAS thread)",
          "seconds": round(seconds, 2), "all_cores": all_cores}
    parity = {"ok": worst <= 0.0, "tolerance": "abs 2e-3 + 1e-2*|ref| (bf16 output)",
              "checked": f"all decode outputs; prefill outputs of {PF_SAMPLE} sequences"}
    return cb, parity


if __name__ == "__main__":
    sys.exit(main())
