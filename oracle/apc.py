"""Prefix-cache bookkeeping oracle (test infrastructure only).

Follows the paper's description of the reuse plane: KV memory is managed in
fixed-size blocks addressed through a per-request block table (Section 2,
PagedAttention's virtual-memory-inspired KV layout), and Automatic Prefix
Caching lets a request reuse the KV blocks of a matching prefix (Section 2;
Section 3: shared policy prefixes should not be recomputed; Section 5.4: the
system prompt, policy text and schema stay identical across many requests).
The paper states no procedure, so the rules below are the readings recorded in
the design notes:

* a block is shareable only when it is full; its identity is the *whole* token
  prefix up to and including it.  Cached blocks live in a trie of nested
  dicts, one level per block, keyed by that block's token tuple, so a path
  from the root spells out the full prefix (no hashing of ids, no parent
  pointers);
* admission walks full blocks from the start and stops at the first prefix not
  in the trie; at most ``(L - 1) // bs`` blocks are taken from the cache so at
  least one token is computed;
* new blocks come from the front of a caller-ordered free list;
* a prompt's full blocks are registered at admission, a sequence's other full
  blocks when it is released, each only if the block before it is registered
  and its prefix is not registered yet (the first registration wins; a
  duplicate stays private);
* released blocks that are registered stay cached with refcount 0 (idle);
  unregistered ones return to the back of the free list;
* with eviction enabled, an allocation that the free list cannot serve evicts
  idle cached blocks one at a time: only trie leaves (no cached block
  continues them), the least recently released first, where one release
  stamps its newly idle blocks last block first; an evicted block leaves the
  trie and goes straight to the request.  Without eviction such a request
  fails.  Capacity is checked before anything changes;
* truncation (rolling back draft or chunk tokens) may only drop unregistered
  blocks; they return to the *front* of the free list, so ``extend`` followed
  by ``truncate`` restores the pool exactly.
"""
from __future__ import annotations

from collections import deque

import numpy as np


class OracleError(Exception):
    code = "error"


class ArgError(OracleError):
    code = "arg"


class NoBlocksError(OracleError):
    code = "no_blocks"


class UnknownSeqError(OracleError):
    code = "unknown_seq"


class PrefixCacheOracle:
    def __init__(self, num_blocks: int, block_size: int, free_order):
        free_order = [int(b) for b in free_order]
        if num_blocks <= 0 or block_size <= 0:
            raise ArgError("pool sizes must be positive")
        if sorted(free_order) != list(range(num_blocks)):
            raise ArgError("free_order must be a permutation of the block ids")
        self.bs = block_size
        self.num_blocks = num_blocks
        self.free = deque(free_order)
        self.root = {}           # tuple(block tokens) -> [physical block, children dict]
        self.registered = set()  # physical blocks present in the trie
        self.ref = [0] * num_blocks
        self.seqs = {}           # seq_id -> {"tokens": list, "blocks": list, "n_reg": int}
        self.evict = False
        self.node = {}           # registered block -> (trie level holding it, its key)
        self.stamp = {}          # idle registered block -> release stamp
        self.clock = 0
        self.evictions = 0

    # -- helpers -----------------------------------------------------------
    def _seq(self, seq_id):
        if seq_id not in self.seqs:
            raise UnknownSeqError(f"unknown sequence {seq_id}")
        return self.seqs[seq_id]

    def _children(self, toks, depth):
        """Trie level below the first ``depth`` blocks of ``toks``."""
        level = self.root
        for j in range(depth):
            level = level[tuple(toks[j * self.bs:(j + 1) * self.bs])][1]
        return level

    def _register_run(self, st):
        """Register full blocks after the sequence's registered leading run,
        in logical order, while the chain is unbroken and the prefix is new."""
        bs, toks, blocks = self.bs, st["tokens"], st["blocks"]
        j = st["n_reg"]
        level = self._children(toks, j)
        while (j + 1) * bs <= len(toks):
            key = tuple(toks[j * bs:(j + 1) * bs])
            if key in level:
                break
            level[key] = [blocks[j], {}]
            self.registered.add(blocks[j])
            self.node[blocks[j]] = (level, key)
            level = level[key][1]
            j += 1
        st["n_reg"] = j

    def _obtainable(self, held_idle=0):
        return len(self.free) + (len(self.stamp) - held_idle if self.evict else 0)

    def _take(self):
        """Next block of an allocation: the free list's front, else evict the
        least recently released idle trie leaf."""
        if self.free:
            return self.free.popleft()
        leaves = [b for b in self.stamp if not self.node[b][0][self.node[b][1]][1]]
        b = min(leaves, key=lambda x: self.stamp[x])
        level, key = self.node.pop(b)
        del level[key]
        self.registered.discard(b)
        del self.stamp[b]
        self.evictions += 1
        return b

    # -- operations ----------------------------------------------------------
    def add(self, seq_id, tokens) -> int:
        """Admit a sequence; return the number of tokens whose KV is reused."""
        toks = [int(t) for t in tokens]
        L, bs = len(toks), self.bs
        if seq_id in self.seqs:
            raise ArgError(f"sequence {seq_id} already exists")
        if L < 1:
            raise ArgError("a sequence needs at least one token")
        hits = []
        level = self.root
        while (len(hits) + 1) * bs <= L - 1:
            key = tuple(toks[len(hits) * bs:(len(hits) + 1) * bs])
            if key not in level:
                break
            hits.append(level[key][0])
            level = level[key][1]
        need = -(-L // bs) - len(hits)
        idle_hits = sum(1 for b in hits if self.ref[b] == 0)
        if need > self._obtainable(idle_hits):
            raise NoBlocksError(f"need {need} blocks, {self._obtainable(idle_hits)} obtainable")
        for b in hits:
            if self.ref[b] == 0:
                del self.stamp[b]
            self.ref[b] += 1
        new = [self._take() for _ in range(need)]
        for b in new:
            self.ref[b] = 1
        st = {"tokens": toks, "blocks": hits + new, "n_reg": len(hits)}
        self.seqs[seq_id] = st
        self._register_run(st)
        return len(hits) * bs

    def extend(self, seq_id, tokens):
        st = self._seq(seq_id)
        toks = [int(t) for t in tokens]
        newL = len(st["tokens"]) + len(toks)
        need = -(-newL // self.bs) - len(st["blocks"])
        if need > self._obtainable():
            raise NoBlocksError(f"need {need} blocks, {self._obtainable()} obtainable")
        for _ in range(need):
            b = self._take()
            self.ref[b] = 1
            st["blocks"].append(b)
        st["tokens"].extend(toks)

    def truncate(self, seq_id, new_len: int):
        st = self._seq(seq_id)
        L = len(st["tokens"])
        if new_len < 1 or new_len > L or new_len < st["n_reg"] * self.bs:
            raise ArgError(f"cannot truncate to {new_len} (length {L}, "
                           f"registered {st['n_reg'] * self.bs})")
        keep = -(-new_len // self.bs)
        dropped = st["blocks"][keep:]
        for b in reversed(dropped):
            self.ref[b] -= 1
            assert self.ref[b] == 0 and b not in self.registered
            self.free.appendleft(b)
        del st["blocks"][keep:]
        del st["tokens"][new_len:]

    def free_seq(self, seq_id):
        st = self._seq(seq_id)
        self._register_run(st)
        for b in st["blocks"]:
            self.ref[b] -= 1
            if self.ref[b] == 0 and b not in self.registered:
                self.free.append(b)
        for b in reversed(st["blocks"]):
            if self.ref[b] == 0 and b in self.registered:
                self.clock += 1
                self.stamp[b] = self.clock
        del self.seqs[seq_id]

    def seq_len(self, seq_id) -> int:
        return len(self._seq(seq_id)["tokens"])

    def metadata(self, seq_ids, q_lens, max_blocks_per_seq: int):
        """Block table (padded with -1), lengths, query offsets and the slot of
        every query token (the last ``q_lens[r]`` positions of sequence r)."""
        seq_ids = list(seq_ids)
        q_lens = [int(x) for x in q_lens]
        if len(seq_ids) != len(q_lens):
            raise ArgError("seq_ids and q_lens differ in length")
        if len(set(seq_ids)) != len(seq_ids):
            raise ArgError("a sequence appears twice in one batch")
        n, bs = len(seq_ids), self.bs
        bt = np.full((n, max_blocks_per_seq), -1, dtype=np.int32)
        seq_lens = np.zeros(n, dtype=np.int32)
        cu = np.zeros(n + 1, dtype=np.int32)
        slots = []
        for r, (sid, ql) in enumerate(zip(seq_ids, q_lens)):
            st = self._seq(sid)
            L = len(st["tokens"])
            if ql < 0 or ql > L:
                raise ArgError(f"q_len {ql} outside [0, {L}]")
            if len(st["blocks"]) > max_blocks_per_seq:
                raise ArgError("max_blocks_per_seq too small")
            bt[r, :len(st["blocks"])] = st["blocks"]
            seq_lens[r] = L
            cu[r + 1] = cu[r] + ql
            for t in range(L - ql, L):
                slots.append(st["blocks"][t // bs] * bs + t % bs)
        return {"block_table": bt, "seq_lens": seq_lens, "cu_seqlens_q": cu,
                "slot_mapping": np.asarray(slots, dtype=np.int32)}

    # -- introspection used by invariant tests --------------------------------
    def free_list(self):
        return list(self.free)

    def stats(self):
        held = {b for st in self.seqs.values() for b in st["blocks"]}
        return {"num_blocks": self.num_blocks, "free_blocks": len(self.free),
                "cached_blocks": len(self.registered), "idle_cached_blocks": len(self.stamp),
                "evictions": self.evictions, "live_seqs": len(self.seqs),
                "live_tokens": sum(len(st["tokens"]) for st in self.seqs.values()),
                "logical_blocks": sum(len(st["blocks"]) for st in self.seqs.values()),
                "physical_blocks": len(held)}

    def kv_waste(self, max_seq_len: int):
        """Slots allocated in blocks versus a contiguous max-length reservation
        per live sequence (Section 2, paged KV memory)."""
        if any(len(st["tokens"]) > max_seq_len for st in self.seqs.values()):
            raise ArgError("max_seq_len below the longest live sequence")
        s = self.stats()
        tokens = s["live_tokens"]
        paged = s["logical_blocks"] * self.bs
        phys = s["physical_blocks"] * self.bs
        contig = s["live_seqs"] * max_seq_len
        return {"tokens": tokens, "paged_slots": paged, "physical_slots": phys,
                "contiguous_slots": contig,
                "paged_waste": 1 - tokens / paged if paged else 0.0,
                "contiguous_waste": 1 - tokens / contig if contig else 0.0,
                "sharing_factor": paged / phys if phys else 1.0}

    def blocks_of(self, seq_id):
        return list(self._seq(seq_id)["blocks"])
