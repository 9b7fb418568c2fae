"""Host-side state of a mixed-fidelity paged KV pool and its device arrays.

``HostMirror`` is the host copy of the per-block state the paper keeps in
its block-state table (App. B.1): block table, fidelity tags, sequence
lengths and the free-block pool.  It validates transition lists through
``ekv_check_transition``, applies the same table updates the device
kernels make, and returns freed blocks to the pool only when the caller
says the GPU work has completed (App. B.2: commit after completion).

Free-pool order (the paper fixes none): unused ids start in ascending
order; freed blocks are appended in list order at commit; refinement takes
new blocks from the head.

``PagedKV`` couples a mirror with the device tensors and drives the C ABI
through :mod:`ekv`.
"""

from collections import deque

import numpy as np

from . import ekv


class HostMirror:
    def __init__(self, block_table, seq_lens, num_blocks, free_ids, tags=None, page=ekv.PAGE):
        self.bt = np.array(block_table, dtype=np.int32, copy=True)
        self.seq_lens = np.array(seq_lens, dtype=np.int32, copy=True)
        self.tags = (np.zeros_like(self.bt, dtype=np.uint8) if tags is None
                     else np.array(tags, dtype=np.uint8, copy=True))
        self.num_blocks = int(num_blocks)
        self.page = page
        self.free = deque(int(b) for b in sorted(free_ids))
        self.reserved = set()   # pairs whose promotion is in flight

    def _validate(self, kind, pairs, new_blocks=None):
        ok, msg = ekv.check_transition(kind, pairs, self.bt, self.tags, self.seq_lens,
                                       self.num_blocks, new_blocks, self.page)
        if not ok:
            raise ekv.EkvError(ekv.ERR_INVALID, msg)

    def plan_demote(self, pairs):
        """Validate and apply a demotion list; returns the blocks it frees
        (not yet back in the free pool)."""
        pairs = np.asarray(pairs, dtype=np.int32).reshape(-1, 2)
        self._validate(0, pairs)
        s, j = pairs[:, 0], pairs[:, 1]   # distinct pairs (validated): one write per entry
        freed = self.bt[s, 2 * j + 1].copy()
        self.bt[s, 2 * j + 1] = self.bt[s, 2 * j]
        self.tags[s, 2 * j] = 1
        self.tags[s, 2 * j + 1] = 1
        return freed

    def commit_freed(self, freed):
        """Return demoted pairs' released blocks once the GPU has finished."""
        self.free.extend(int(b) for b in freed)

    def reserve_refine(self, pairs):
        """Validate a refinement list and take one block per pair from the
        free pool, leaving the table as it is (the pairs stay BASE until
        :meth:`publish_refine`); returns the new blocks."""
        pairs = np.asarray(pairs, dtype=np.int32).reshape(-1, 2)
        n = len(pairs)
        if n > len(self.free):
            raise ekv.EkvError(ekv.ERR_INVALID, "not enough free blocks for refinement")
        new = np.array([self.free.popleft() for _ in range(n)], dtype=np.int32)
        keys = list(zip(pairs[:, 0].tolist(), pairs[:, 1].tolist()))
        try:
            self._validate(1, pairs, new)
            busy = [k for k in keys if k in self.reserved]
            if busy:
                raise ekv.EkvError(ekv.ERR_INVALID, f"pair {busy[0]} is already being promoted")
        except ekv.EkvError:
            self.free.extendleft(reversed(new.tolist()))
            raise
        self.reserved.update(keys)
        return new

    def cancel_refine(self, pairs, new):
        """Undo :meth:`reserve_refine`: the blocks go back to the head of the
        free pool in their order and the pairs are no longer reserved."""
        self.free.extendleft(reversed(np.asarray(new, dtype=np.int32).tolist()))
        p = np.asarray(pairs, dtype=np.int32).reshape(-1, 2)
        self.reserved.difference_update(zip(p[:, 0].tolist(), p[:, 1].tolist()))

    def publish_refine(self, pairs, new):
        """Apply the table update of a refinement (after its device work)."""
        p = np.asarray(pairs, dtype=np.int32).reshape(-1, 2)
        s, j = p[:, 0], p[:, 1]   # distinct pairs (validated at reservation)
        self.bt[s, 2 * j + 1] = np.asarray(new, dtype=np.int32)
        self.tags[s, 2 * j] = 0
        self.tags[s, 2 * j + 1] = 0
        self.reserved.difference_update(zip(s.tolist(), j.tolist()))

    def plan_refine(self, pairs):
        """Validate a refinement list, take one block per pair from the free
        pool and apply the table update; returns the new blocks."""
        new = self.reserve_refine(pairs)
        self.publish_refine(pairs, new)
        return new

    def lower(self):
        return ekv.lower(self.tags, self.seq_lens, self.page)


class PagedKV:
    """Device pool + block table + tags + lengths, with a HostMirror."""

    def __init__(self, pool_words, block_table, seq_lens, free_ids, num_kv_heads, dtype="bf16",
                 device="cuda"):
        import torch
        elem = np.uint8 if dtype == "e5m2" else np.int16
        kv = pool_words if isinstance(pool_words, torch.Tensor) else torch.from_numpy(
            np.ascontiguousarray(pool_words).view(elem))
        self.kv = kv.to(device).contiguous()
        self.num_kv_heads = num_kv_heads
        self.dtype = dtype
        nb = self.kv.numel() // (2 * num_kv_heads * ekv.PAGE * ekv.HEAD_DIM)
        self.mirror = HostMirror(block_table, seq_lens, nb, free_ids)
        self.bt = torch.from_numpy(self.mirror.bt.copy()).to(device)
        self.tags = torch.from_numpy(self.mirror.tags.copy()).to(device)
        self.seq_lens = torch.from_numpy(self.mirror.seq_lens.copy()).to(device)
        self.bounds = torch.zeros((len(self.mirror.seq_lens), 2), dtype=torch.int32, device=device)
        self.pool = ekv.make_pool(self.kv, num_kv_heads, dtype)
        self.device = device
        self.mode = ekv.MODE_NATIVE

    @property
    def block_bytes(self):
        elem = 1 if self.dtype == "e5m2" else 2
        return 2 * self.num_kv_heads * ekv.PAGE * ekv.HEAD_DIM * elem

    def _upload(self, arr):
        """Host array -> device through a fresh pinned buffer (stream-ordered,
        does not block the host on earlier GPU work)."""
        import torch
        return torch.from_numpy(np.ascontiguousarray(arr)).pin_memory().to(self.device, non_blocking=True)

    def relower(self):
        """Recompute the dispatch metadata from the host mirror and upload it."""
        import torch
        self.mode, bounds = self.mirror.lower()
        self.bounds.copy_(torch.from_numpy(bounds).pin_memory(), non_blocking=True)
        return self.mode

    def batch(self, num_q_heads, mode=None, use_boundaries=True, max_seq_len=None):
        mode = self.mode if mode is None else mode
        if max_seq_len is None:
            max_seq_len = int(self.mirror.seq_lens.max()) if len(self.mirror.seq_lens) else 0
        return ekv.make_batch(self.seq_lens, self.bt, self.tags,
                              self.bounds if use_boundaries else None, num_q_heads, mode, max_seq_len)

    def demote(self, pairs, emit_lo=True, stream=None):
        """Enqueue a demotion; returns (freed ids on device, lo bytes, host freed ids).
        The freed ids return to the free pool at :meth:`commit`."""
        import torch
        host_freed = self.mirror.plan_demote(pairs)
        n = len(host_freed)
        pairs_d = self._upload(np.asarray(pairs, dtype=np.int32).reshape(-1, 2))
        freed = torch.empty(n, dtype=torch.int32, device=self.device)
        lo = torch.empty((n, self.block_bytes), dtype=torch.uint8, device=self.device) if emit_lo else None
        ekv.demote(self.pool, pairs_d, self.bt, self.tags, freed, lo, stream)
        ev = torch.cuda.Event()
        ev.record(stream)
        self._pending = getattr(self, "_pending", []) + [(ev, host_freed)]
        return freed, lo, host_freed

    def commit(self, wait=True):
        """Return blocks freed by completed demotions to the free pool.  With
        wait=False only demotions whose GPU work has already finished are
        committed."""
        keep = []
        for ev, ids in getattr(self, "_pending", []):
            if wait:
                ev.synchronize()
            if wait or ev.query():
                self.mirror.commit_freed(ids)
            else:
                keep.append((ev, ids))
        self._pending = keep

    def refine(self, pairs, lo, stream=None):
        """Enqueue a refinement of BASE pairs from their refinement bytes."""
        import torch
        new = self.mirror.plan_refine(pairs)
        pairs_d = self._upload(np.asarray(pairs, dtype=np.int32).reshape(-1, 2))
        new_d = self._upload(new)
        ekv.refine(self.pool, pairs_d, new_d, self.bt, self.tags, lo, stream)
        return new

    def append(self, slots, k, v, stream=None):
        ekv.append_kv(self.pool, slots, k, v, stream)


class AsyncPromotion:
    """CPU backing and asynchronous promotion (App. B.2).

    Demotion runs on the compute stream and emits the pair's refinement
    bytes; a copy stream moves them into pinned host memory (the CPU
    backing).  Promotion reserves one free block Q per pair and copies the
    backing into Q on the copy stream, with one kernel that reads the pinned
    memory directly; the pair stays BASE and executable meanwhile.  :meth:`publish` orders the compute stream after a finished
    copy and runs the staged refinement, which rebuilds the pair and
    publishes the mapping.  Both streams have the default priority.
    """

    def __init__(self, kv, copy_stream=None):
        import torch
        self.kv = kv
        self.copy = copy_stream if copy_stream is not None else torch.cuda.Stream()
        self.backing = {}     # (s, j) -> (pinned uint8 [block bytes], event: backing complete)
        self.inflight = []    # (copy-done event, pairs, new blocks, pinned sources)
        self.last_copy = None  # (start, end) events of the last promotion's copy on the copy stream

    def demote(self, pairs, stream=None):
        """Demote on ``stream`` and back the refinement bytes up to the host.
        Returns (freed ids on device, host freed ids)."""
        import torch
        stream = stream if stream is not None else torch.cuda.current_stream()
        pairs = np.asarray(pairs, dtype=np.int32).reshape(-1, 2)
        freed, lo, host_freed = self.kv.demote(pairs, emit_lo=True, stream=stream)
        if len(pairs) == 0:
            return freed, host_freed
        ready = torch.cuda.Event()
        ready.record(stream)
        host = torch.empty(lo.shape, dtype=torch.uint8, pin_memory=True)
        with torch.cuda.stream(self.copy):
            self.copy.wait_event(ready)
            host.copy_(lo, non_blocking=True)
            lo.record_stream(self.copy)
        done = torch.cuda.Event()
        done.record(self.copy)
        for key, row in zip(zip(pairs[:, 0].tolist(), pairs[:, 1].tolist()), host.unbind(0)):
            self.backing[key] = (row, done)
        return freed, host_freed

    def promote(self, pairs):
        """Reserve a block per pair and start restoring it from the backing;
        returns the reserved blocks.  The pairs stay BASE until published."""
        import torch
        pairs = np.asarray(pairs, dtype=np.int32).reshape(-1, 2)
        keys = list(zip(pairs[:, 0].tolist(), pairs[:, 1].tolist()))
        missing = [k for k in keys if k not in self.backing]
        if missing:
            raise ekv.EkvError(ekv.ERR_INVALID, f"no CPU backing for pairs {missing[:4]}")
        new = self.kv.mirror.reserve_refine(pairs)
        sources = [self.backing[k][0] for k in keys]
        for done in {id(self.backing[k][1]): self.backing[k][1] for k in keys}.values():
            self.copy.wait_event(done)
        # one copy kernel reads every pair's backing over the host link;
        # the library records `ev` after it (ekv_promote_begin)
        start = torch.cuda.Event(enable_timing=True)
        start.record(self.copy)
        ev = torch.cuda.Event(enable_timing=True)
        try:
            ekv.promote_begin(self.kv.pool, [h.data_ptr() for h in sources], new, ev, self.copy)
        except ekv.EkvError:
            self.kv.mirror.cancel_refine(pairs, new)
            raise
        for k in keys:
            del self.backing[k]
        self.last_copy = (start, ev)
        self.inflight.append((ev, pairs, new, sources))
        return new

    def publish(self, wait=False, stream=None):
        """Publish every promotion whose copy has finished (all, with
        ``wait``); returns the number of pairs published."""
        import torch
        stream = stream if stream is not None else torch.cuda.current_stream()
        keep, count = [], 0
        for ev, pairs, new, sources in self.inflight:
            if not (wait or ev.query()):
                keep.append((ev, pairs, new, sources))
                continue
            with torch.cuda.stream(stream):
                pairs_d = self.kv._upload(pairs)
                new_d = self.kv._upload(new)
            # the stream waits for the copy, then the staged refinement publishes
            ekv.promote_publish(self.kv.pool, pairs_d, new_d, self.kv.bt, self.kv.tags, ev, stream)
            self.kv.mirror.publish_refine(pairs, new)
            count += len(pairs)
        self.inflight = keep
        return count
