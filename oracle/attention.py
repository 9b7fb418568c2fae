"""Softmax attention over a mixed-fidelity paged sequence (oracle, float64).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's backend computes ordinary attention; only the load of each KV
block differs with its mode, and the output interface is the same for both
modes (§3.2; App. B.3).  So the oracle is the textbook definition applied to
the dense K/V that :func:`oracle.paged.gather_sequence` produces:

    S[t]  = scale * <q, K[t]>
    P     = exp(S - max S) / sum exp(S - max S)
    out   = sum_t P[t] V[t]

Readings where the paper is silent:

* ``scale`` is an argument, default ``1/sqrt(d)``;
* grouped-query attention maps query head ``h`` to KV head ``h // G`` with
  ``G = Hq / Hkv`` (contiguous groups);
* a decode query sees every cached token of its sequence, its own included
  (its K/V were appended beforehand, §3.2: new KV is written as TARGET);
* chunked prefill row ``i`` of a chunk of ``n`` new tokens, in a sequence of
  total length ``L``, sees keys ``0 .. L - n + i`` inclusive (causal).

All arithmetic is float64; the 16-bit inputs widen exactly.
"""

import math

import numpy as np

from . import encoding, paged


def _softmax_weighted(scores, values):
    m = np.max(scores, axis=-1, keepdims=True)
    e = np.exp(scores - m)
    return (e / np.sum(e, axis=-1, keepdims=True)) @ values


def decode(q, pool, block_table, tags, seq_lens, dtype="bf16", scale=None):
    """Decode attention: one query token per sequence.

    q: uint16 [B][Hq][d]; pool: uint16 [NB][2][Hkv][page][d];
    block_table: int [B][max_blocks]; tags: uint8 [B][max_blocks];
    seq_lens: int [B].  Returns float64 [B][Hq][d].
    """
    q = np.asarray(q, dtype=np.uint16)
    bsz, hq, d = q.shape
    hkv = pool.shape[2]
    if hq % hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    group = hq // hkv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    qf = encoding.words_to_f64(q, dtype)
    out = np.zeros((bsz, hq, d), dtype=np.float64)
    for s in range(bsz):
        length = int(seq_lens[s])
        if length == 0:
            continue
        k, v = paged.gather_sequence(pool, block_table[s], tags[s], length, dtype)
        for h in range(hq):
            kh = h // group
            scores = scale * (k[:, kh, :] @ qf[s, h])
            out[s, h] = _softmax_weighted(scores, v[:, kh, :])
    return out


def prefill(q, cu_q, pool, block_table, tags, seq_lens, dtype="bf16", scale=None):
    """Chunked-prefill attention for new tokens whose K/V are already in the pool.

    q: uint16 [total_new][Hq][d] with sequence s's rows at cu_q[s]..cu_q[s+1];
    seq_lens[s] counts the whole context including the chunk.
    Returns float64 [total_new][Hq][d].
    """
    q = np.asarray(q, dtype=np.uint16)
    total, hq, d = q.shape
    hkv = pool.shape[2]
    group = hq // hkv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    qf = encoding.words_to_f64(q, dtype)
    out = np.zeros((total, hq, d), dtype=np.float64)
    for s in range(len(seq_lens)):
        r0, r1 = int(cu_q[s]), int(cu_q[s + 1])
        n = r1 - r0
        length = int(seq_lens[s])
        if n == 0:
            continue
        if n > length:
            raise ValueError("chunk longer than the sequence")
        k, v = paged.gather_sequence(pool, block_table[s], tags[s], length, dtype)
        first = length - n
        visible = np.arange(length)[None, :] <= (first + np.arange(n))[:, None]
        for h in range(hq):
            kh = h // group
            scores = scale * (qf[r0:r1, h] @ k[:, kh, :].T)
            scores = np.where(visible, scores, -np.inf)
            out[r0:r1, h] = _softmax_weighted(scores, v[:, kh, :])
    return out
