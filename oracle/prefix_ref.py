"""Oracle: block-level prefix caching with chained block keys (test infrastructure).

What is computed (InferLog, section 2.1.2 "KV Cache and Prefix Caching", with
its figure of three requests): a prompt is cut into fixed-size token blocks; a
block's KV can be reused by a later request only if that request has the same
tokens in that block AND in every block before it -- req3 may reuse b1..b3 of
req1, but not req2's b7, b8, because its predecessor b3 differs from req2's b6.
The cached prefix of a request is therefore the longest run of leading blocks
whose whole token prefix was registered before.  KV for the cache-missing
tokens is then computed and stored (section 3.2.2).

Readings taken where the paper is silent:

* block size 16 tokens; only full blocks are keyed and registered, so the
  cached-prefix length P is a multiple of 16;
* a block is identified by a 64-bit chained key (defined below); the exact
  token prefix is the ground truth, the key is its compact stand-in;
* frozen snapshot: every request of a batch is matched against the table as it
  stood before the batch; the batch's new full blocks are registered after all
  requests were matched, first registration wins (lower request index);
* at least one token is always recomputed: the match is capped at
  floor((L - 1) / 16) blocks, so S = L - P >= 1;
* blocks are handed out by a bump allocator, request by request, block by
  block: cached blocks reuse the registered id, every other block of the
  request (including the reserve for later decode tokens) gets the next id.

The key (a design of this project, frozen here; the paper names none):

* fmix64 is the 64-bit finaliser of MurmurHash3 (Appleby, public domain);
* a block of 16 int32 tokens t_0..t_15 is read as eight 64-bit words
  w_i = u32(t_{2i}) | u32(t_{2i+1}) << 32;
  its digest is d = fmix64( sum_i fmix64(w_i XOR K_i) mod 2^64 ),
  K_i = (i + 1) * 0x9E3779B97F4A7C15 mod 2^64;
* keys chain: c_{-1} = 0x243F6A8885A308D3, c_b = fmix64(c_{b-1} XOR d_b),
  and a key equal to 0 (the empty-slot marker) is replaced by 1 before it is
  used as the next chain input.

Plain Python integers / numpy uint64 arithmetic, no blocking or reordering.
"""
from __future__ import annotations

import numpy as np

BLOCK = 16
MASK64 = (1 << 64) - 1
_FMIX_M1 = 0xFF51AFD7ED558CCD
_FMIX_M2 = 0xC4CEB9FE1A85EC53
_WORD_KEY = 0x9E3779B97F4A7C15
_CHAIN_SEED = 0x243F6A8885A308D3


class OracleError(Exception):
    """Raised where the C-ABI returns an error code; ``code`` names it."""

    def __init__(self, code: str, msg: str):
        super().__init__(f"{code}: {msg}")
        self.code = code


def fmix64(x: int) -> int:
    """MurmurHash3 64-bit finaliser on one Python int (mod 2^64)."""
    x &= MASK64
    x ^= x >> 33
    x = (x * _FMIX_M1) & MASK64
    x ^= x >> 33
    x = (x * _FMIX_M2) & MASK64
    x ^= x >> 33
    return x


def _fmix64_np(x: np.ndarray) -> np.ndarray:
    """The same finaliser element-wise on a uint64 array (wrap-around mod 2^64)."""
    x = x.astype(np.uint64, copy=True)
    x ^= x >> np.uint64(33)
    x *= np.uint64(_FMIX_M1)
    x ^= x >> np.uint64(33)
    x *= np.uint64(_FMIX_M2)
    x ^= x >> np.uint64(33)
    return x


def block_digest(block_tokens) -> int:
    """Digest of one block of 16 token ids (scalar reference form)."""
    toks = [int(t) & 0xFFFFFFFF for t in block_tokens]
    assert len(toks) == BLOCK
    acc = 0
    for i in range(BLOCK // 2):
        w = toks[2 * i] | (toks[2 * i + 1] << 32)
        k = ((i + 1) * _WORD_KEY) & MASK64
        acc = (acc + fmix64(w ^ k)) & MASK64
    return fmix64(acc)


def block_digests(tokens: np.ndarray) -> np.ndarray:
    """Digests of every full block of ``tokens`` (int32, 1-D) as uint64[n_full].

    Vectorised over blocks only; per block it is exactly ``block_digest``.
    """
    tokens = np.asarray(tokens, dtype=np.int32)
    n_full = tokens.shape[0] // BLOCK
    if n_full == 0:
        return np.zeros(0, dtype=np.uint64)
    u = tokens[: n_full * BLOCK].view(np.uint32).astype(np.uint64).reshape(n_full, BLOCK // 2, 2)
    w = u[:, :, 0] | (u[:, :, 1] << np.uint64(32))
    k = (np.arange(1, BLOCK // 2 + 1, dtype=np.uint64) * np.uint64(_WORD_KEY))
    acc = _fmix64_np(w ^ k[None, :]).sum(axis=1, dtype=np.uint64)
    return _fmix64_np(acc)


def chain_keys(tokens: np.ndarray) -> list[int]:
    """Chained keys c_0..c_{n_full-1} of the full blocks of one prompt."""
    keys = []
    c = _CHAIN_SEED
    for d in block_digests(tokens).tolist():
        c = fmix64(c ^ int(d))
        if c == 0:
            c = 1
        keys.append(c)
    return keys


class PrefixCacheRef:
    """Dictionary model of the prefix cache: chained key -> physical block id.

    ``max_entries`` models the table's capacity: a batch is refused (ETABLE)
    when the entries already held plus an upper bound on what it may register
    (its new full blocks) would exceed it.  ``num_blocks`` is the pool size.
    Every refused call leaves the state untouched.
    """

    def __init__(self, num_blocks: int, max_entries: int):
        self.num_blocks = int(num_blocks)
        self.max_entries = int(max_entries)
        self.table: dict[int, int] = {}
        self.next_block = 0

    def match(self, prompts, reserve=None, max_blocks=None, no_lookup=False, no_register=False):
        """Match a batch against the frozen table, allocate, then register.

        Returns (cached_len int32[B], block_tables int32[B, max_blocks] padded
        with -1, block_keys uint64[B, max_blocks] with 0 past the full blocks).
        """
        B = len(prompts)
        reserve = [0] * B if reserve is None else [int(x) for x in reserve]
        if max_blocks is None:
            max_blocks = max([-(-(len(p) + reserve[r]) // BLOCK) for r, p in enumerate(prompts)] + [1])
        snapshot = self.table  # not modified until every request is matched
        cached = np.zeros(B, dtype=np.int32)
        tables = np.full((B, max_blocks), -1, dtype=np.int32)
        keys_out = np.zeros((B, max_blocks), dtype=np.uint64)
        plans = []
        next_block = self.next_block
        for r, p in enumerate(prompts):
            L = len(p)
            if L <= 0:
                raise OracleError("EINVAL", f"request {r} has no tokens")
            if reserve[r] < 0:
                raise OracleError("EINVAL", f"request {r} has a negative reserve")
            n_full = L // BLOCK
            n_match_cap = (L - 1) // BLOCK
            n_total = -(-(L + reserve[r]) // BLOCK)
            if n_total > max_blocks:
                raise OracleError("EINVAL", f"request {r} needs {n_total} blocks > max_blocks")
            keys = chain_keys(p)
            m = 0
            if not no_lookup:
                while m < n_match_cap and keys[m] in snapshot:
                    m += 1
            ids = [snapshot[keys[b]] for b in range(m)]
            ids += list(range(next_block, next_block + n_total - m))
            next_block += n_total - m
            cached[r] = BLOCK * m
            tables[r, :n_total] = ids
            keys_out[r, :n_full] = np.array(keys, dtype=np.uint64)
            plans.append((keys, m, n_full, ids))
        if next_block > self.num_blocks:
            raise OracleError("ENOSPC", f"batch needs blocks up to {next_block} > pool {self.num_blocks}")
        if not no_register:
            bound = sum(n_full - m for (_, m, n_full, _) in plans)
            if len(self.table) + bound > self.max_entries:
                raise OracleError("ETABLE", "block table would exceed its capacity")
        # commit: state changes only after every check passed
        self.next_block = next_block
        if not no_register:
            for keys, m, n_full, ids in plans:
                for b in range(m, n_full):
                    self.table.setdefault(keys[b], ids[b])
        return cached, tables, keys_out
