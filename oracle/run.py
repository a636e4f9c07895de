"""Replay a synthetic workload script through the oracle (test infrastructure only).

The script (admissions, extensions, K/V writes, releases, truncations and
attention launches) is plain data from the seeded generator; this module
interprets it with the oracle's own prefix cache and its own float32 paged
store (values are exactly representable: they are the generator's fp32 or
bf16-rounded draws), and computes every launch's attention in float64.
"""
from __future__ import annotations

import numpy as np

from .apc import PrefixCacheOracle
from .attention import kv_append, new_cache, paged_attention


class OracleReplay:
    def __init__(self, wl, store_values: bool = True):
        cfg = wl.cfg
        self.wl = wl
        self.pool = PrefixCacheOracle(wl.num_blocks, cfg.block_size, wl.free_order)
        self.pool.evict = wl.evict
        self.store_values = store_values
        if store_values:
            self.k_cache, self.v_cache = new_cache(wl.num_blocks, cfg.num_kv_heads,
                                                   cfg.head_dim, cfg.block_size)
            self.k_cache = self.k_cache.astype(np.float32)
            self.v_cache = self.v_cache.astype(np.float32)
        self.n_cached = {}

    def _apply(self, op):
        p = self.pool
        if op.kind == "add":
            self.n_cached[op.seq_id] = p.add(op.seq_id, op.tokens)
        elif op.kind == "extend":
            p.extend(op.seq_id, op.tokens)
        elif op.kind == "free":
            p.free_seq(op.seq_id)
        elif op.kind == "truncate":
            p.truncate(op.seq_id, op.n)
        elif op.kind == "write_kv":
            if self.store_values:
                k, v = op.k.get(), op.v.get()
                md = p.metadata([op.seq_id], [len(k)], self.wl.max_blocks_per_seq)
                kv_append(self.k_cache, self.v_cache, md["slot_mapping"], k, v)
        else:
            raise ValueError(op.kind)

    def setup(self):
        for op in self.wl.setup:
            self._apply(op)
        return self

    def launch(self, launch, rows=None, attend=True):
        """Run one launch; returns its metadata, the prefix-hit token counts of
        the sequences it admitted, and (optionally) out / lse in float64."""
        self.n_cached = {}
        for op in launch.pre:
            self._apply(op)
        md = self.pool.metadata(launch.seq_ids, launch.q_lens, self.wl.max_blocks_per_seq)
        res = {"meta": md, "n_cached": dict(self.n_cached)}
        if self.store_values:
            k_new, v_new = launch.k_new.get(), launch.v_new.get()
            kv_append(self.k_cache, self.v_cache, md["slot_mapping"], k_new, v_new)
            if attend:
                q = launch.q.get()
                out, lse = paged_attention(q, self.k_cache, self.v_cache, md["block_table"],
                                           md["seq_lens"], md["cu_seqlens_q"],
                                           self.wl.cfg.num_kv_heads, rows=rows)
                res["out"], res["lse"] = out, lse
        return res

    def finish(self, launch):
        for op in launch.post:
            self._apply(op)
