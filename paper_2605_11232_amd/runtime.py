"""Drive a synthetic workload through libpa on the GPU.

Host bookkeeping (prefix-hit lookup, allocation, metadata, launch plan) runs in
the library's C++ block manager and planner; K/V appends and attention run in
its HIP kernels.  torch provides device memory, pinned staging buffers and the
stream -- nothing else.
"""
from __future__ import annotations

import numpy as np
import torch

from . import binding as B

KIND = {"prefill": B.KIND_PREFILL, "decode": B.KIND_DECODE, "verify": B.KIND_VERIFY}


def torch_dtype(name: str):
    return {"bf16": torch.bfloat16, "f32": torch.float32}[name]


class Prepared:
    """Device-resident inputs of one launch (metadata, plan, q, new K/V)."""

    def __init__(self, **kw):
        self.__dict__.update(kw)


_OPCODE = {"add": B.OP_ADD, "extend": B.OP_EXTEND, "truncate": B.OP_TRUNCATE, "free": B.OP_FREE}


def batch_ops(ops) -> B.PackedOps:
    """Pack a list of pool ops into the arrays of one pa_pool_apply call
    (write_kv ops, which only occur in setup, are kept apart)."""
    pool_ops = [op for op in ops if op.kind != "write_kv"]
    if len(pool_ops) != len(ops):
        raise ValueError("write_kv ops cannot be batched")
    n = len(pool_ops)
    codes = np.array([_OPCODE[op.kind] for op in pool_ops], dtype=np.int32)
    ids = np.array([op.seq_id for op in pool_ops], dtype=np.int64)
    lens = np.array([len(op.tokens) if op.tokens is not None else 0 for op in pool_ops],
                    dtype=np.int64)
    off = np.zeros(n + 1, dtype=np.int32)
    np.cumsum(lens, out=off[1:])
    toks = [op.tokens for op in pool_ops if op.tokens is not None and len(op.tokens)]
    toks = np.concatenate(toks).astype(np.int32) if toks else np.zeros(0, np.int32)
    new_lens = np.array([op.n if op.kind == "truncate" else 0 for op in pool_ops], dtype=np.int32)
    return B.PackedOps(codes, ids, off, toks, new_lens)


def marshal_launch(launch):
    """Pack a launch's pool operations and its (seq_ids, q_lens) once, as
    the staged path passes them to the library (cached on the launch)."""
    d = launch.__dict__
    if "_batched" not in d:
        d["_batched"] = {"pre": batch_ops(launch.pre), "post": batch_ops(launch.post)}
    if "_inputs" not in d:
        d["_inputs"] = B.LaunchInputs(launch.seq_ids, launch.q_lens)
    return d["_batched"], d["_inputs"]


def plan_words_bound(cfg, n_seqs: int, total_q: int, max_blocks_per_seq: int) -> int:
    """Upper bound on the plan size of a launch of n_seqs sequences and
    total_q query tokens (tile items, key-split items of at least 256 keys,
    merge groups, cascade member tables, per-XCD padding)."""
    max_keys = max_blocks_per_seq * cfg.block_size
    return 32 + 8 * (cfg.num_kv_heads * (total_q * cfg.group // 128 + n_seqs)
                     + 2 * cfg.num_kv_heads * n_seqs * (max_keys // 256 + 2) + 64)


class Staging:
    """One pinned host buffer and one device buffer holding a launch's
    metadata and plan ([seq_lens | cu_seqlens_q | block_table | slot_mapping |
    plan], int32), uploaded in one piece on the compute stream (by the
    library's upload kernel, or a copy-engine copy), so stream order puts it
    after the kernels of the launch that used the device buffer before.  The host fills the pinned buffer while the GPU
    still works on an earlier launch; ``guard``, an event recorded after the
    upload (``ready``, or one the caller hands to ``prepare_staged``), guards
    reuse of the host buffer."""

    def __init__(self, device, n_seqs, max_blocks, max_tokens, plan_words):
        self.n_seqs, self.max_blocks = n_seqs, max_blocks
        sizes = [("sl", n_seqs), ("cu", n_seqs + 1), ("bt", n_seqs * max_blocks),
                 ("slots", max_tokens), ("plan", plan_words)]
        total = sum(max(1, n) for _, n in sizes)
        self.host = torch.empty(total, dtype=torch.int32, pin_memory=True)
        self.dev = torch.empty(total, dtype=torch.int32, device=device)
        off = 0
        for name, n in sizes:
            m = max(1, n)
            setattr(self, name, (self.host[off:off + m], self.dev[off:off + m]))
            setattr(self, name + "_off", off)
            off += m
        self.ready = B.StreamEvent()
        self.guard = self.ready
        self.used = False
        # host views the library writes into, and device views by launch shape
        self.buffers = B.LaunchBuffers(self.bt[0].numpy().reshape(n_seqs, max_blocks),
                                       self.sl[0].numpy(), self.cu[0].numpy(),
                                       self.slots[0].numpy(), self.plan[0].numpy())
        self.info = B.PlanInfo()
        self._views = {}

    def device_views(self, n, total_q):
        """(block_table [n, max_blocks], seq_lens, cu_seqlens_q, slot_mapping)
        views of the device buffer for a launch of n sequences."""
        key = (n, total_q)
        v = self._views.get(key)
        if v is None:
            v = self._views[key] = (self.bt[1][:n * self.max_blocks].view(n, self.max_blocks),
                                    self.sl[1][:n], self.cu[1][:n + 1], self.slots[1][:total_q])
        return v

    def wait(self):
        if self.used:
            self.guard.synchronize()


class DeviceReplay:
    def __init__(self, wl, device: str = "cuda", kind: str | None = None, num_cus: int = 0,
                 cascade: bool = True, stage_kernel: bool = True):
        cfg = wl.cfg
        self.wl, self.cfg, self.device = wl, cfg, torch.device(device)
        self.tdtype = torch_dtype(cfg.dtype)
        self.dcode = B.PA_BF16 if cfg.dtype == "bf16" else B.PA_F32
        self.pool = B.Pool(wl.num_blocks, cfg.block_size, wl.free_order, evict=wl.evict)
        # keys in the grouped layout [block][head][dim / 32][slot position][32]
        shape_k = (wl.num_blocks, cfg.num_kv_heads, cfg.head_dim // 32, cfg.block_size, 32)
        shape_v = (wl.num_blocks, cfg.num_kv_heads, cfg.head_dim, cfg.block_size)
        # Uninitialised on purpose: the kernels must never read unwritten slots.
        self.k_cache = torch.empty(shape_k, dtype=self.tdtype, device=self.device)
        self.v_cache = torch.empty(shape_v, dtype=self.tdtype, device=self.device)
        self.kind = kind
        self.num_cus = num_cus
        self.cascade = cascade
        # staged uploads by the library's kernel (else by a copy-engine copy)
        self.stage_kernel = stage_kernel
        self.n_cached = {}
        self._ws = None  # split-K workspace of staged launches (all on the current stream)

    # -- host ops ------------------------------------------------------------
    def _write_kv(self, seq_id, k: np.ndarray, v: np.ndarray):
        md = self.pool.metadata([seq_id], [len(k)], self.wl.max_blocks_per_seq)
        dev = self.device
        slots = torch.from_numpy(md["slot_mapping"]).to(dev)
        kt = torch.from_numpy(k).to(dev, self.tdtype)
        vt = torch.from_numpy(v).to(dev, self.tdtype)
        B.kv_append(kt, vt, slots, self.k_cache, self.v_cache)

    def apply(self, op):
        p = self.pool
        if op.kind == "add":
            self.n_cached[op.seq_id] = p.add(op.seq_id, op.tokens)
        elif op.kind == "extend":
            p.extend(op.seq_id, op.tokens)
        elif op.kind == "free":
            p.free(op.seq_id)
        elif op.kind == "truncate":
            p.truncate(op.seq_id, op.n)
        elif op.kind == "write_kv":
            self._write_kv(op.seq_id, op.k.get(), op.v.get())
        else:
            raise ValueError(op.kind)

    def apply_batched(self, launch, which: str):
        """Apply the launch's pre or post pool ops in one library call."""
        packed = marshal_launch(launch)[0][which]
        if packed.n == 0:
            return
        self.pool.apply_packed(packed)
        self.n_cached.update(packed.admitted())

    def setup(self):
        for op in self.wl.setup:
            self.apply(op)
        torch.cuda.synchronize()
        return self

    def launch_kind(self, launch) -> str:
        if self.kind:
            return self.kind
        ql = set(launch.q_lens)
        if ql == {1}:
            return "decode"
        if len(ql) == 1 and 1 < next(iter(ql)) <= 8:
            return "verify"
        return "prefill"

    # -- one launch ------------------------------------------------------------
    def prepare(self, launch, q=None, k_new=None, v_new=None) -> Prepared:
        """Run the launch's host ops, build metadata and plan, stage to device."""
        self.n_cached = {}
        for op in launch.pre:
            self.apply(op)
        cfg, dev = self.cfg, self.device
        md = self.pool.metadata(launch.seq_ids, launch.q_lens, self.wl.max_blocks_per_seq)
        kind = self.launch_kind(launch)
        n_q = launch.q_lens[0] if kind == "verify" else 1
        plan, info = B.plan(KIND[kind], n_q, md["seq_lens"], md["cu_seqlens_q"], cfg.num_q_heads,
                            cfg.num_kv_heads, cfg.head_dim, cfg.block_size, self.dcode, self.num_cus,
                            block_table=md["block_table"] if self.cascade else None)
        if q is None:
            q = torch.from_numpy(launch.q.get()).to(dev, self.tdtype)
        if k_new is None:
            k_new = torch.from_numpy(launch.k_new.get()).to(dev, self.tdtype)
        if v_new is None:
            v_new = torch.from_numpy(launch.v_new.get()).to(dev, self.tdtype)
        ws = None
        if info.workspace_bytes:
            ws = torch.empty(int(info.workspace_bytes), dtype=torch.uint8, device=dev)
        T = launch.total_q
        return Prepared(
            kind=kind, meta=md, info=info, plan_host=plan,
            block_table=torch.from_numpy(md["block_table"]).to(dev),
            seq_lens=torch.from_numpy(md["seq_lens"]).to(dev),
            cu=torch.from_numpy(md["cu_seqlens_q"]).to(dev),
            slots=torch.from_numpy(md["slot_mapping"]).to(dev),
            plan=torch.from_numpy(plan).to(dev), q=q, k_new=k_new, v_new=v_new, ws=ws,
            out=torch.empty((T, cfg.num_q_heads, cfg.head_dim), dtype=self.tdtype, device=dev),
            lse=torch.empty((T, cfg.num_q_heads), dtype=torch.float32, device=dev),
            n_cached=dict(self.n_cached))

    def prepare_staged(self, launch, st: Staging, q, k_new, v_new, out, lse,
                       guard=None, upload: bool = True) -> Prepared:
        """Like ``prepare`` but through a preallocated pinned/device staging
        pair: one library call applies the launch's pool operations and
        writes its metadata and plan into the pinned buffer, one
        asynchronous copy uploads them, so host bookkeeping overlaps earlier
        GPU work.  The returned host views (meta, plan_host, info) live in the
        staging buffer: valid until the buffer is used for another launch.

        The staging buffer is released for reuse by an event recorded after
        the upload: its own ``ready`` event right after it, or, when the
        caller passes ``guard`` (an event it wants on the stream anyway, such
        as the start of a timed attention call), that event, recorded by
        ``append`` after the KV append.  Each event record is a marker in the
        stream that idles the device for a few microseconds.

        With upload=False only the host side runs (the pool operations,
        metadata and plan into the pinned buffer); ``upload`` then puts the
        upload on the stream, before the launch's kernels."""
        batched, inp = marshal_launch(launch)
        cfg = self.cfg
        n, T = inp.n, inp.total_q
        kind = self.launch_kind(launch)
        n_q = launch.q_lens[0] if kind == "verify" else 1
        st.wait()
        info = self.pool.prepare_launch(batched["pre"], inp, st.buffers, KIND[kind], n_q,
                                        cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim,
                                        self.dcode, self.num_cus, self.cascade, info=st.info)
        self.n_cached = batched["pre"].admitted()
        ws = None
        if info.workspace_bytes:
            if self._ws is None or self._ws.numel() < int(info.workspace_bytes):
                self._ws = torch.empty(int(info.workspace_bytes), dtype=torch.uint8,
                                       device=self.device)
            ws = self._ws
        bt, sl, cu, slots = st.device_views(n, T)
        p = Prepared(
            kind=kind, meta=st.buffers.meta(n, T), info=info,
            plan_host=st.buffers.plan[:int(info.plan_words)], block_table=bt, seq_lens=sl,
            cu=cu, slots=slots, plan=st.plan[1], q=q, k_new=k_new, v_new=v_new, ws=ws, out=out,
            lse=lse, n_cached=self.n_cached, guard=guard, staging=st)
        if upload:
            self.upload(p)
        return p

    def upload(self, p: Prepared):
        """Put the upload of a staged launch's metadata and plan on the
        stream (one copy, everything up to the end of the plan)."""
        st = p.staging
        used = st.plan_off + int(p.info.plan_words)
        if self.stage_kernel:
            B.stage_upload(st.dev, st.host, 4 * used)
        else:
            st.dev[:used].copy_(st.host[:used], non_blocking=True)
        if p.guard is None:
            st.ready.record()
            st.guard = st.ready
        else:
            st.guard = p.guard
        st.used = True

    def append(self, p: Prepared, stream=None, record_guard: bool = True):
        """KV append of the launch; records the caller's staging guard after
        it unless record_guard is False (the guard is then the start event the
        caller hands to ``attend``)."""
        B.kv_append(p.k_new, p.v_new, p.slots, self.k_cache, self.v_cache, stream)
        guard = getattr(p, "guard", None)
        if guard is not None and record_guard:
            guard.record(stream)

    def attend(self, p: Prepared, stream=None, events=None):
        """The attention call; events = (start, stop) ride on its first and
        last kernel dispatches (pa_set_launch_events)."""
        if events is not None:
            B.set_launch_events(*events)
        B.attention(KIND[p.kind], p.q, self.k_cache, self.v_cache, p.block_table, p.seq_lens, p.cu,
                    p.plan, p.info, p.ws, p.out, p.lse, stream=stream)

    def run(self, launch) -> Prepared:
        p = self.prepare(launch)
        self.append(p)
        self.attend(p)
        return p

    def finish(self, launch, batched: bool = False):
        if batched:
            self.apply_batched(launch, "post")
            return
        for op in launch.post:
            self.apply(op)
