"""Seeded synthetic inputs for the mixed-fidelity paged-attention path.

This module only makes inputs: random 16-bit K/V/Q words (or FP8 E5M2 K/V
bytes, rounded by torch), block tables that
scatter each sequence over a shuffled physical pool, sequence lengths, and
the lists of pairs a caller chooses to demote.  It performs none of the
method's arithmetic (no encoding, no attention, no transitions), so both
the HIP path and the CPU oracle can consume what it returns.

Shapes follow the paper's models (§4.1): Llama-3.1-8B (32 query / 8 KV
heads, head dim 128) and Llama-3.1-70B (64 / 8), with 16-token pages.
Values are N(0, 1) rounded to the 16-bit type, optionally with a small set
of outlier channels scaled by 10; the paper's datasets (LongBench, ShareGPT,
Mooncake traces) are not available, and these seeded inputs stand in for
them.
"""

import math

import numpy as np

HEAD_DIM = 128
PAGE = 16


def f32_to_bf16_words(x):
    """Round float32 to bfloat16 words (round to nearest even), bit by bit."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    out = rounded.astype(np.uint16)
    out[nan] = 0x7FC0
    return out


def f32_to_fp16_words(x):
    return np.asarray(x, dtype=np.float32).astype(np.float16).view(np.uint16)


def f32_to_e5m2_bytes(x):
    """Round float32 to FP8 E5M2 bytes with torch's own conversion."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.float8_e5m2)
    return t.view(torch.uint8).numpy().copy()


def to_words(x, dtype):
    """16-bit words (bf16, fp16) or bytes (e5m2) of float32 values."""
    if dtype == "bf16":
        return f32_to_bf16_words(x)
    if dtype == "fp16":
        return f32_to_fp16_words(x)
    if dtype == "e5m2":
        return f32_to_e5m2_bytes(x)
    raise ValueError(dtype)


def query_dtype(dtype):
    """Queries of an 8-bit (e5m2) pool are fp16; otherwise the pool dtype."""
    return "fp16" if dtype == "e5m2" else dtype


def complete_pairs(seq_len, page=PAGE):
    """Number of pairs (2j, 2j+1) whose two blocks are full."""
    return int(seq_len) // (2 * page)


def choose_pairs(rng, seq_lens, fraction, placement="random", page=PAGE):
    """Pick the (s, j) pairs to hold in BASE.

    Per sequence ``floor(fraction * n_complete + 0.5)`` complete pairs are
    taken: uniformly without replacement ("random") or the oldest ones
    ("oldest").  Returns int32 [n][2] in (s, j) order.
    """
    out = []
    for s, length in enumerate(seq_lens):
        n = complete_pairs(length, page)
        k = int(math.floor(fraction * n + 0.5))
        if k == 0:
            continue
        if placement == "random":
            js = np.sort(rng.permutation(n)[:k])
        elif placement == "oldest":
            js = np.arange(k)
        else:
            raise ValueError(placement)
        out.extend((s, int(j)) for j in js)
    return np.array(out, dtype=np.int32).reshape(-1, 2)


def make_decode_case(seq_lens, num_q_heads, num_kv_heads, *, head_dim=HEAD_DIM,
                     page=PAGE, dtype="bf16", seed=0, base_fraction=0.0,
                     placement="random", outlier_channels=0, spare_blocks=0,
                     max_blocks=None, garbage_tail=True):
    """A TARGET pool holding ``len(seq_lens)`` sequences plus one decode query
    per sequence, and the pairs to demote for the requested BASE fraction.

    Physical blocks are a seeded permutation of the pool; ``spare_blocks``
    extra blocks stay free.  Slots past a sequence's end, and free blocks,
    hold random 16-bit words (NaN patterns included) when ``garbage_tail``,
    so a kernel that reads them shows up in the result.
    """
    rng = np.random.default_rng(seed)
    seq_lens = np.asarray(seq_lens, dtype=np.int32)
    bsz = len(seq_lens)
    nblk = [-(-int(l) // page) for l in seq_lens]
    used = int(sum(nblk))
    nb = used + int(spare_blocks)
    if max_blocks is None:
        max_blocks = max(2, max(nblk) + (max(nblk) % 2))
    perm = rng.permutation(nb).astype(np.int32)
    bt = np.zeros((bsz, max_blocks), dtype=np.int32)
    pos = 0
    for s in range(bsz):
        bt[s, :nblk[s]] = perm[pos:pos + nblk[s]]
        pos += nblk[s]
    free = np.sort(perm[used:])

    vals = rng.standard_normal((nb, 2, num_kv_heads, page, head_dim), dtype=np.float32)
    if outlier_channels:
        for plane in range(2):
            idx = rng.choice(num_kv_heads * head_dim, size=outlier_channels, replace=False)
            for c in idx:
                vals[:, plane, c // head_dim, :, c % head_dim] *= 10.0
    pool = to_words(vals, dtype)
    if garbage_tail:
        junk = lambda shape: rng.integers(0, np.iinfo(pool.dtype).max + 1, size=shape, dtype=pool.dtype)
        for s in range(bsz):
            rem = int(seq_lens[s]) % page
            if rem:
                last = bt[s, nblk[s] - 1]
                pool[last, :, :, rem:, :] = junk(pool[last, :, :, rem:, :].shape)
        if len(free):
            pool[free] = junk(pool[free].shape)
    q = to_words(rng.standard_normal((bsz, num_q_heads, head_dim), dtype=np.float32), query_dtype(dtype))
    pairs = choose_pairs(rng, seq_lens, base_fraction, placement, page)
    return {
        "pool": pool, "block_table": bt, "tags": np.zeros((bsz, max_blocks), dtype=np.uint8),
        "seq_lens": seq_lens, "q": q, "pairs": pairs, "free": free.astype(np.int32),
        "dtype": dtype, "num_kv_heads": num_kv_heads, "page": page,
    }


def make_prefill_case(prefix_lens, chunk_lens, num_q_heads, num_kv_heads, *,
                      head_dim=HEAD_DIM, page=PAGE, dtype="bf16", seed=0,
                      base_fraction=0.0, placement="random", spare_blocks=0,
                      aligned_keys=0, aligned_factor=4.0):
    """A pool holding each sequence's prefix, the new chunk's Q/K/V rows and
    the slots the chunk's K/V are to be written to (after the prefix).

    ``aligned_keys`` > 0 plants, per sequence with a chunk and a prefix of at
    least 64 tokens, that many prefix keys in the second half of the prefix
    whose K row (for one KV head) is ``aligned_factor`` times one chunk
    query's row (a random row and a random head of that KV head's group),
    rounded like every other value: that query's score jumps far above the
    scores of the first keys, which a streaming softmax has to absorb
    after it has already accumulated output."""
    prefix_lens = np.asarray(prefix_lens, dtype=np.int32)
    chunk_lens = np.asarray(chunk_lens, dtype=np.int32)
    total = prefix_lens + chunk_lens
    case = make_decode_case(total, num_q_heads, num_kv_heads, head_dim=head_dim,
                            page=page, dtype=dtype, seed=seed, base_fraction=0.0,
                            spare_blocks=spare_blocks)
    rng = np.random.default_rng(seed + 7919)
    n = int(chunk_lens.sum())
    cu = np.zeros(len(total) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(chunk_lens)
    slots = np.empty(n, dtype=np.int64)
    for s in range(len(total)):
        for i in range(int(chunk_lens[s])):
            t = int(prefix_lens[s]) + i
            slots[cu[s] + i] = int(case["block_table"][s, t // page]) * page + t % page
    # BASE pairs only inside the prefix (new KV stays TARGET)
    case["pairs"] = choose_pairs(rng, prefix_lens, base_fraction, placement, page)
    qf = rng.standard_normal((n, num_q_heads, head_dim), dtype=np.float32)
    case["q"] = to_words(qf, query_dtype(dtype))
    planted = []
    group = num_q_heads // num_kv_heads
    for s in range(len(total) if aligned_keys else 0):
        if chunk_lens[s] == 0 or prefix_lens[s] < 64:
            continue
        for _ in range(aligned_keys):
            t = int(rng.integers(prefix_lens[s] // 2, prefix_lens[s]))
            row = int(cu[s] + rng.integers(0, chunk_lens[s]))
            kvh = int(rng.integers(0, num_kv_heads))
            head = kvh * group + int(rng.integers(0, group))
            blk = int(case["block_table"][s, t // page])
            case["pool"][blk, 0, kvh, t % page, :] = to_words(aligned_factor * qf[row, head], dtype)
            planted.append((s, t, row, head))
    case["aligned"] = np.array(planted, dtype=np.int64).reshape(-1, 4)
    case["k_new"] = to_words(rng.standard_normal((n, num_kv_heads, head_dim), dtype=np.float32), dtype)
    case["v_new"] = to_words(rng.standard_normal((n, num_kv_heads, head_dim), dtype=np.float32), dtype)
    case["cu_q"] = cu
    case["slots"] = slots.astype(np.int32)
    case["prefix_lens"] = prefix_lens
    return case


# The workloads the benchmark and the parity tests run, by what they are.
WORKLOADS = {
    "tiny-decode": dict(batch=4, num_q_heads=8, num_kv_heads=2, seq_lens=[64, 128, 192, 256],
                        base_fraction=0.5, placement="random", seed=0),
    "llama3-8b-decode": dict(batch=64, num_q_heads=32, num_kv_heads=8, len_range=(2048, 8192),
                             base_fractions=(0.0, 0.25, 0.5, 1.0), placement="random",
                             outlier_channels=10, seed=1),
    "llama3-70b-decode": dict(batch=256, num_q_heads=64, num_kv_heads=8, seq_len=4096,
                              base_fraction=0.5, placement="oldest", seed=2),
    "llama3-8b-chunked-prefill": dict(batch=16, num_q_heads=32, num_kv_heads=8, prefix=2048,
                                      chunk=512, base_fraction=0.5, placement="random", seed=3),
    "pressure-transition-mix": dict(num_blocks=200_000, batch=128, num_q_heads=32, num_kv_heads=8,
                                    len_range=(1024, 16384), demote_frac=0.10, refine_frac=0.05,
                                    seed=4),
}


def seq_lens_uniform(rng, batch, lo, hi):
    return rng.integers(lo, hi + 1, size=batch).astype(np.int32)


def make_decode_case_torch(seq_lens, num_q_heads, num_kv_heads, *, seed, outlier_channels=0,
                           spare_blocks=0, dtype="bf16", device="cuda", max_blocks=None):
    """Large-workload variant of :func:`make_decode_case` that draws the
    values on the GPU with a seeded torch generator.  Block placement and
    lengths come from NumPy as before.  Returns device tensors for the pool
    (16-bit words as int16, or e5m2 bytes as uint8, [NB][2][Hkv][16][128])
    and the query (fp16 for e5m2 pools), NumPy arrays for the rest."""
    import torch
    rng = np.random.default_rng(seed)
    seq_lens = np.asarray(seq_lens, dtype=np.int32)
    bsz = len(seq_lens)
    nblk = [-(-int(l) // PAGE) for l in seq_lens]
    used = int(sum(nblk))
    nb = used + int(spare_blocks)
    if max_blocks is None:
        max_blocks = max(2, max(nblk) + (max(nblk) % 2))
    perm = rng.permutation(nb).astype(np.int32)
    bt = np.zeros((bsz, max_blocks), dtype=np.int32)
    pos = 0
    for s in range(bsz):
        bt[s, :nblk[s]] = perm[pos:pos + nblk[s]]
        pos += nblk[s]
    free = np.sort(perm[used:]).astype(np.int32)
    tdtype = {"bf16": torch.bfloat16, "fp16": torch.float16, "e5m2": torch.float8_e5m2}[dtype]
    qdtype = torch.float16 if dtype == "e5m2" else tdtype
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    pool = torch.empty((nb, 2, num_kv_heads, PAGE, HEAD_DIM), dtype=tdtype, device=device)
    scale = torch.ones((2, num_kv_heads, 1, HEAD_DIM), dtype=torch.float32, device=device)
    for plane in range(2):
        if outlier_channels:
            idx = rng.choice(num_kv_heads * HEAD_DIM, size=outlier_channels, replace=False)
            for c in idx:
                scale[plane, c // HEAD_DIM, 0, c % HEAD_DIM] = 10.0
    chunk = 4096
    for b0 in range(0, nb, chunk):
        b1 = min(nb, b0 + chunk)
        x = torch.randn((b1 - b0, 2, num_kv_heads, PAGE, HEAD_DIM), generator=gen, device=device,
                        dtype=torch.float32)
        pool[b0:b1] = (x * scale).to(tdtype)
    q = torch.randn((bsz, num_q_heads, HEAD_DIM), generator=gen, device=device,
                    dtype=torch.float32).to(qdtype)
    words = pool.view(torch.uint8) if dtype == "e5m2" else pool.view(torch.int16)
    return {"pool": words, "q": q, "block_table": bt, "seq_lens": seq_lens,
            "free": free, "dtype": dtype, "num_kv_heads": num_kv_heads}


def extract_sequences(pool_dev, block_table, seq_lens, seq_ids):
    """Host copy of just the blocks of ``seq_ids``, renumbered densely:
    returns (pool [n][2][Hkv][16][128] of uint16 words, or uint8 bytes for a
    1-byte pool, block_table, seq_lens)."""
    import torch
    page = PAGE
    blocks = []
    bt = np.zeros((len(seq_ids), block_table.shape[1]), dtype=np.int32)
    for r, s in enumerate(seq_ids):
        nblk = -(-int(seq_lens[s]) // page)
        bt[r, :nblk] = np.arange(len(blocks), len(blocks) + nblk)
        blocks.extend(int(b) for b in block_table[s, :nblk])
    idx = torch.as_tensor(np.array(blocks, dtype=np.int64), device=pool_dev.device)
    if pool_dev.element_size() == 1:
        host = pool_dev.view(torch.uint8).index_select(0, idx).cpu().numpy()
    else:
        host = pool_dev.index_select(0, idx).cpu().numpy().view(np.uint16)
    return host, bt, np.asarray(seq_lens, dtype=np.int32)[list(seq_ids)]
