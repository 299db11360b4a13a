"""Oracle: prefix cache whose blocks have a lifecycle (test infrastructure).

What is computed (InferLog, section 2.1.2 "KV Cache and Prefix Caching"): KV
of a shared prompt prefix is reused across requests at block granularity, and
because GPU memory is bounded, cached blocks are evicted least recently used
first.  Matching and registration are those of ``oracle.prefix_ref`` (chained
16-token block keys, frozen snapshot per batch, cap so one token is
recomputed, first registration wins); what changes is where block ids come
from and when they can be taken back.

A physical block is in exactly one of three states:

* in use: held by at least one unfinished request (reference count > 0);
* cached: no request holds it, but its key is registered, so a later request
  can still hit it; these blocks form the LRU list, least recently used first;
* free: no request holds it and no key names it.

Readings taken where the paper is silent:

* a batch first pins every block its requests hit (in the frozen snapshot), in
  request order; only then are new blocks taken, request by request, block by
  block: from the front of the free queue while it is non-empty (initially
  0, 1, ..., num_blocks - 1, so without frees ids come out as from a bump
  allocator), otherwise by evicting the head of the LRU list (its key is
  unregistered and the block reused);
* a batch that needs more new blocks than free + cached-and-not-hit blocks is
  refused (ENOSPC) with no state change;
* when a request finishes, its blocks are released from its last logical block
  to its first; a block whose count drops to 0 goes to the tail of the LRU list
  if its key is registered, else to the back of the free queue.  Releasing the
  tail first makes a prompt's later blocks older than its earlier ones, so a
  prefix loses its end before its start;
* touching a cached block moves it to the LRU tail; touching a block in use or
  free changes nothing;
* the key table never limits the cache: each registered key names one block,
  so there are never more keys than blocks.

Plain dicts, a deque and an OrderedDict, no shortcuts.
"""
from __future__ import annotations

from collections import OrderedDict, deque

import numpy as np

from .prefix_ref import BLOCK, OracleError, chain_keys


class LruPrefixCacheRef:
    """The block states above; every refused call leaves the state untouched."""

    def __init__(self, num_blocks: int):
        if num_blocks < 0:
            raise OracleError("EINVAL", "num_blocks < 0")
        self.num_blocks = int(num_blocks)
        self.table: dict[int, int] = {}      # key -> block
        self.key_of: dict[int, int] = {}     # block -> key, registered blocks only
        self.ref = [0] * self.num_blocks
        self.free = deque(range(self.num_blocks))
        self.lru: OrderedDict[int, None] = OrderedDict()
        self.evictions = 0

    # -- queries ---------------------------------------------------------------
    def usage(self):
        """(blocks in use, cached blocks, free blocks, evictions so far)."""
        in_use = sum(1 for c in self.ref if c > 0)
        return in_use, len(self.lru), len(self.free), self.evictions

    def lru_order(self):
        """Cached blocks, least recently used first."""
        return list(self.lru)

    # -- matching --------------------------------------------------------------
    def match(self, prompts, reserve=None, max_blocks=None, no_lookup=False, no_register=False):
        """Returns (cached_len int32[B], block_tables int32[B, max_blocks], keys uint64)."""
        B = len(prompts)
        reserve = [0] * B if reserve is None else [int(x) for x in reserve]
        if max_blocks is None:
            max_blocks = max([-(-(len(p) + reserve[r]) // BLOCK) for r, p in enumerate(prompts)] + [1])
        plans = []
        for r, p in enumerate(prompts):
            L = len(p)
            if L <= 0:
                raise OracleError("EINVAL", f"request {r} has no tokens")
            if reserve[r] < 0:
                raise OracleError("EINVAL", f"request {r} has a negative reserve")
            n_total = -(-(L + reserve[r]) // BLOCK)
            if n_total > max_blocks:
                raise OracleError("EINVAL", f"request {r} needs {n_total} blocks > max_blocks")
            keys = chain_keys(p)
            m = 0
            if not no_lookup:
                while m < (L - 1) // BLOCK and keys[m] in self.table:
                    m += 1
            hits = [self.table[keys[b]] for b in range(m)]
            plans.append((keys, m, L // BLOCK, n_total, hits))

        need = sum(n_total - m for (_, m, _, n_total, _) in plans)
        hit_cached = {b for (_, _, _, _, hits) in plans for b in hits if self.ref[b] == 0}
        if need > len(self.free) + len(self.lru) - len(hit_cached):
            raise OracleError("ENOSPC", f"batch needs {need} new blocks")

        # pin every hit first, so no allocation below can take a block a request reuses
        for (_, _, _, _, hits) in plans:
            for b in hits:
                if self.ref[b] == 0:
                    del self.lru[b]
                self.ref[b] += 1
        cached = np.zeros(B, dtype=np.int32)
        tables = np.full((B, max_blocks), -1, dtype=np.int32)
        keys_out = np.zeros((B, max_blocks), dtype=np.uint64)
        for r, (keys, m, n_full, n_total, hits) in enumerate(plans):
            ids = list(hits)
            for _ in range(n_total - m):
                ids.append(self._take())
            cached[r] = BLOCK * m
            tables[r, :n_total] = ids
            keys_out[r, :n_full] = np.array(keys, dtype=np.uint64)
            plans[r] = (keys, m, n_full, ids)
        if not no_register:
            for keys, m, n_full, ids in plans:
                for b in range(m, n_full):
                    if keys[b] not in self.table:
                        self.table[keys[b]] = ids[b]
                        self.key_of[ids[b]] = keys[b]
        return cached, tables, keys_out

    def _take(self) -> int:
        if self.free:
            b = self.free.popleft()
        else:
            b, _ = self.lru.popitem(last=False)
            del self.table[self.key_of.pop(b)]
            self.evictions += 1
        self.ref[b] = 1
        return b

    # -- lifecycle ---------------------------------------------------------------
    def release(self, block_tables):
        """Requests finished: release each row's blocks (up to its first -1), last first."""
        rows = [[int(x) for x in row] for row in block_tables]
        rows = [row[:row.index(-1)] if -1 in row else row for row in rows]
        count: dict[int, int] = {}
        for row in rows:
            for b in row:
                if not 0 <= b < self.num_blocks:
                    raise OracleError("EINVAL", f"block id {b} out of range")
                count[b] = count.get(b, 0) + 1
        for b, c in count.items():
            if c > self.ref[b]:
                raise OracleError("EINVAL", f"block {b} released {c} times, held {self.ref[b]}")
        for row in rows:
            for b in reversed(row):
                self.ref[b] -= 1
                if self.ref[b] == 0:
                    if b in self.key_of:
                        self.lru[b] = None
                    else:
                        self.free.append(b)

    def touch(self, block_ids):
        """Mark cached blocks as just used (LRU tail); -1 entries are skipped."""
        ids = [int(b) for b in block_ids]
        for b in ids:
            if b != -1 and not 0 <= b < self.num_blocks:
                raise OracleError("EINVAL", f"block id {b} out of range")
        for b in ids:
            if b in self.lru:
                self.lru.move_to_end(b)
