"""ctypes binding of libpa (include/pa.h): argument marshalling only.

Every computation runs in the C++/HIP library; this module converts numpy
arrays and torch tensors to pointers and return codes to exceptions.  If the
library is missing it raises -- there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpa.so")

PA_OK, PA_ERR_ARG, PA_ERR_UNSUPPORTED, PA_ERR_NO_BLOCKS, PA_ERR_UNKNOWN_SEQ, PA_ERR_LAUNCH = (
    0, -1, -2, -3, -4, -5)
PA_F32, PA_BF16 = 0, 1
OP_ADD, OP_EXTEND, OP_TRUNCATE, OP_FREE = 0, 1, 2, 3
KIND_PREFILL, KIND_DECODE, KIND_VERIFY = 0, 1, 2
_CODES = {PA_ERR_ARG: "arg", PA_ERR_UNSUPPORTED: "unsupported", PA_ERR_NO_BLOCKS: "no_blocks",
          PA_ERR_UNKNOWN_SEQ: "unknown_seq", PA_ERR_LAUNCH: "launch"}

# Every symbol include/pa.h declares.
EXPORTS = ["pa_last_error", "pa_abi_version", "pa_pool_create", "pa_pool_destroy", "pa_seq_add",
           "pa_seq_extend", "pa_seq_truncate", "pa_seq_free", "pa_seqs_add", "pa_seqs_extend",
           "pa_seqs_truncate", "pa_seqs_free", "pa_pool_apply", "pa_seq_len", "pa_seq_blocks",
           "pa_pool_free_list", "pa_build_metadata", "pa_attn_plan", "pa_kv_append",
           "pa_attn_prefill", "pa_attn_decode", "pa_attn_verify", "pa_pool_set_eviction",
           "pa_pool_get_stats", "pa_pool_kv_waste", "pa_form_batches", "pa_prepare_launch",
           "pa_stage_upload", "pa_attn_workspace_size", "pa_attn_decode_workspace_size",
           "pa_attn_decode_noalloc", "pa_set_launch_events"]


class PaError(RuntimeError):
    def __init__(self, rc: int, msg: str):
        super().__init__(f"[{_CODES.get(rc, rc)}] {msg}")
        self.rc = rc
        self.code = _CODES.get(rc, str(rc))


class PoolStats(C.Structure):
    _fields_ = [(n, C.c_int64) for n in ("num_blocks", "free_blocks", "cached_blocks",
                                         "idle_cached_blocks", "evictions", "live_seqs",
                                         "live_tokens", "logical_blocks", "physical_blocks")]


class KvWaste(C.Structure):
    _fields_ = [("tokens", C.c_int64), ("paged_slots", C.c_int64), ("physical_slots", C.c_int64),
                ("contiguous_slots", C.c_int64), ("paged_waste", C.c_double),
                ("contiguous_waste", C.c_double), ("sharing_factor", C.c_double)]


class PlanInfo(C.Structure):
    _fields_ = [("kind", C.c_int32), ("n_q", C.c_int32), ("n_shared_items", C.c_int32),
                ("n_tile_items", C.c_int32), ("n_row_items", C.c_int32), ("n_groups", C.c_int32),
                ("n_merge_rows", C.c_int32), ("grid", C.c_int32), ("variant", C.c_int32),
                ("reserved", C.c_int32), ("plan_words", C.c_int64), ("workspace_bytes", C.c_int64),
                ("n_seqs", C.c_int32), ("total_q", C.c_int32), ("num_q_heads", C.c_int32),
                ("num_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("dtype", C.c_int32),
                ("partial_rows", C.c_int64)]


_lib = None
_P = C.c_void_p
_I32P = C.POINTER(C.c_int32)
_I64P = C.POINTER(C.c_int64)


def lib():
    """Load libpa.so (built in-tree by ``paper_2605_11232_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2605_11232_amd.build` (no fallback exists)")
    L = C.CDLL(LIB_PATH)
    i32, i64, f32 = C.c_int32, C.c_int64, C.c_float
    sig = {
        "pa_last_error": (C.c_char_p, []),
        "pa_abi_version": (i32, []),
        "pa_pool_create": (C.c_int, [i32, i32, _I32P, C.POINTER(_P)]),
        "pa_pool_destroy": (None, [_P]),
        "pa_seq_add": (C.c_int, [_P, i64, _I32P, i32, _I32P]),
        "pa_seq_extend": (C.c_int, [_P, i64, _I32P, i32]),
        "pa_seq_truncate": (C.c_int, [_P, i64, i32]),
        "pa_seq_free": (C.c_int, [_P, i64]),
        "pa_seqs_add": (C.c_int, [_P, i32, _I64P, _I32P, _I32P, _I32P, _I32P]),
        "pa_seqs_extend": (C.c_int, [_P, i32, _I64P, _I32P, _I32P, _I32P]),
        "pa_seqs_truncate": (C.c_int, [_P, i32, _I64P, _I32P, _I32P]),
        "pa_seqs_free": (C.c_int, [_P, i32, _I64P, _I32P]),
        "pa_pool_apply": (C.c_int, [_P, i32, _P, _P, _P, _P, _P, _P, _P]),
        "pa_seq_len": (C.c_int, [_P, i64, _I32P]),
        "pa_seq_blocks": (C.c_int, [_P, i64, _I32P, i32, _I32P]),
        "pa_pool_free_list": (C.c_int, [_P, _I32P, i32, _I32P]),
        "pa_build_metadata": (C.c_int, [_P, i32, _I64P, _I32P, i32, _I32P, _I32P, _I32P, _I32P, i64]),
        "pa_attn_plan": (C.c_int, [i32, i32, i32, _I32P, _I32P, _I32P, i32, i32, i32, i32, i32, i32,
                                   i32, _I32P, i64, C.POINTER(PlanInfo)]),
        "pa_kv_append": (C.c_int, [_P, _P, _P, i32, _P, _P, i32, i32, i32, i32, i32, _P]),
        "pa_stage_upload": (C.c_int, [_P, _P, i64, _P]),
        "pa_attn_workspace_size": (C.c_int, [i32, i32, i32, i32, C.POINTER(C.c_size_t)]),
        "pa_attn_decode_workspace_size": (C.c_int, [i32, i32, i32, i32, C.POINTER(C.c_size_t)]),
        "pa_pool_set_eviction": (C.c_int, [_P, i32]),
        "pa_pool_get_stats": (C.c_int, [_P, C.POINTER(PoolStats)]),
        "pa_pool_kv_waste": (C.c_int, [_P, i32, C.POINTER(KvWaste)]),
        "pa_form_batches": (C.c_int, [i32, _I32P, _I32P, i32, _I32P, _I32P, _I32P, _I32P, _I32P,
                                      _I32P, _I32P]),
        "pa_prepare_launch": (C.c_int, [_P, i32, _P, _P, _P, _P, _P, _P, i32, _P, _P, i32, _P, _P,
                                        _P, _P, i64, i32, i32, i32, i32, i32, i32, i32, i32, _P,
                                        i64, C.POINTER(PlanInfo)]),
    }
    attn = (C.c_int, [_P, _P, _P, i32, _P, i32, _P, _P, i32, i32, i32, i32, i32, i32, f32, i32, _P,
                      C.POINTER(PlanInfo), _P, C.c_size_t, _P, _P, _P])
    for name in ("pa_attn_prefill", "pa_attn_decode", "pa_attn_verify"):
        sig[name] = attn
    # decode without the workspace pair
    sig["pa_attn_decode_noalloc"] = (C.c_int, attn[1][:18] + attn[1][20:])
    sig["pa_set_launch_events"] = (C.c_int, [_P, _P])
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def _check(rc: int):
    if rc != PA_OK:
        raise PaError(rc, lib().pa_last_error().decode())


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a: np.ndarray, ctype=C.c_int32):
    return a.ctypes.data_as(C.POINTER(ctype))


def _addr(a) -> int:
    """Address of a numpy array's data (0 for None or an empty array)."""
    return 0 if a is None or a.size == 0 else a.ctypes.data


class PackedOps:
    """A step's pool operations as pa_pool_apply takes them (ops, seq_ids,
    token_offsets, tokens, new_lens), plus the n_cached output array, with
    their addresses taken once so that repeated calls marshal nothing."""

    def __init__(self, ops, seq_ids, offsets, tokens, new_lens):
        self.ops = _i32(ops)
        self.seq_ids = np.ascontiguousarray(seq_ids, dtype=np.int64)
        self.offsets = _i32(offsets)
        self.tokens = _i32(tokens)
        self.new_lens = _i32(new_lens)
        self.n = int(self.ops.size)
        if not (self.seq_ids.size == self.n and self.offsets.size == self.n + 1
                and self.new_lens.size == self.n):
            raise ValueError("PackedOps: arrays of inconsistent length")
        self.n_cached = np.zeros(max(1, self.n), np.int32)
        self.addrs = (_addr(self.ops), _addr(self.seq_ids), _addr(self.offsets),
                      _addr(self.tokens), _addr(self.new_lens), _addr(self.n_cached))
        self.add_rows = np.flatnonzero(self.ops == OP_ADD)
        self.add_ids = self.seq_ids[self.add_rows].tolist()

    def admitted(self) -> dict:
        """{seq_id: reused tokens} of the admissions of the last application."""
        return dict(zip(self.add_ids, self.n_cached[self.add_rows].tolist())) if self.add_ids else {}


class LaunchInputs:
    """One launch's sequence ids (int64) and query lengths (int32), with
    their addresses taken once."""

    def __init__(self, seq_ids, q_lens):
        self.seq_ids = np.ascontiguousarray(seq_ids, dtype=np.int64)
        self.q_lens = _i32(q_lens)
        if self.seq_ids.size != self.q_lens.size:
            raise ValueError("LaunchInputs: seq_ids and q_lens differ in length")
        self.n = int(self.seq_ids.size)
        self.total_q = int(self.q_lens.sum()) if self.n else 0
        self.addrs = (_addr(self.seq_ids), _addr(self.q_lens))


class LaunchBuffers:
    """Caller-owned host int32 arrays that launch metadata and plan are
    written to (e.g. views of one pinned staging buffer): block_table
    [rows, max_blocks], seq_lens [rows], cu_seqlens_q [rows + 1],
    slot_mapping [tokens], plan [words]; addresses taken once."""

    def __init__(self, block_table, seq_lens, cu_seqlens_q, slot_mapping, plan):
        arrs = (block_table, seq_lens, cu_seqlens_q, slot_mapping, plan)
        for a in arrs:
            if a.dtype != np.int32 or not a.flags["C_CONTIGUOUS"]:
                raise ValueError("LaunchBuffers: arrays must be contiguous int32")
        if block_table.ndim != 2 or seq_lens.size != block_table.shape[0] or \
                cu_seqlens_q.size < seq_lens.size + 1:
            raise ValueError("LaunchBuffers: inconsistent shapes")
        self.block_table, self.seq_lens, self.cu_seqlens_q, self.slot_mapping, self.plan = arrs
        self.rows, self.max_blocks = (int(x) for x in block_table.shape)
        # slot_mapping may be empty; a non-null address is passed regardless
        self.addrs = tuple(a.ctypes.data for a in arrs)

    def meta(self, n: int, total_q: int) -> dict:
        """Views of the first launch's metadata (as Pool.metadata returns)."""
        return {"block_table": self.block_table[:n], "seq_lens": self.seq_lens[:n],
                "cu_seqlens_q": self.cu_seqlens_q[:n + 1],
                "slot_mapping": self.slot_mapping[:total_q]}


class Pool:
    """Host block manager (prefix-hit lookup, allocation, tables, slots)."""

    def __init__(self, num_blocks: int, block_size: int, free_order, evict: bool = False):
        self._lib = lib()
        fo = _i32(free_order)
        h = _P()
        _check(self._lib.pa_pool_create(int(num_blocks), int(block_size),
                                        _ptr(fo) if fo.size else None, C.byref(h)))
        self._h = h
        self.num_blocks, self.block_size = int(num_blocks), int(block_size)
        if evict:
            self.set_eviction(True)

    def set_eviction(self, enabled: bool):
        _check(self._lib.pa_pool_set_eviction(self._h, int(bool(enabled))))

    def stats(self) -> dict:
        st = PoolStats()
        _check(self._lib.pa_pool_get_stats(self._h, C.byref(st)))
        return {n: int(getattr(st, n)) for n, _ in PoolStats._fields_}

    def kv_waste(self, max_seq_len: int) -> dict:
        w = KvWaste()
        _check(self._lib.pa_pool_kv_waste(self._h, int(max_seq_len), C.byref(w)))
        return {n: (float if t is C.c_double else int)(getattr(w, n)) for n, t in KvWaste._fields_}

    def close(self):
        if getattr(self, "_h", None):
            self._lib.pa_pool_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def add(self, seq_id: int, tokens) -> int:
        t = _i32(tokens)
        n = C.c_int32(0)
        _check(self._lib.pa_seq_add(self._h, int(seq_id), _ptr(t) if t.size else None, t.size,
                                    C.byref(n)))
        return n.value

    def extend(self, seq_id: int, tokens):
        t = _i32(tokens)
        _check(self._lib.pa_seq_extend(self._h, int(seq_id), _ptr(t) if t.size else None, t.size))

    def truncate(self, seq_id: int, new_len: int):
        _check(self._lib.pa_seq_truncate(self._h, int(seq_id), int(new_len)))

    def free(self, seq_id: int):
        _check(self._lib.pa_seq_free(self._h, int(seq_id)))

    # -- batched forms (one library call per serving step) --------------------
    def add_many(self, seq_ids, offsets, tokens):
        """Admit len(seq_ids) sequences; returns reused-token counts (int32)."""
        ids = np.ascontiguousarray(seq_ids, dtype=np.int64)
        off, tok = _i32(offsets), _i32(tokens)
        out = np.zeros(ids.size, np.int32)
        _check(self._lib.pa_seqs_add(self._h, ids.size, ids.ctypes.data_as(_I64P), _ptr(off),
                                     _ptr(tok) if tok.size else None, _ptr(out), None))
        return out

    def extend_many(self, seq_ids, offsets, tokens):
        ids = np.ascontiguousarray(seq_ids, dtype=np.int64)
        off, tok = _i32(offsets), _i32(tokens)
        _check(self._lib.pa_seqs_extend(self._h, ids.size, ids.ctypes.data_as(_I64P), _ptr(off),
                                        _ptr(tok) if tok.size else None, None))

    def truncate_many(self, seq_ids, new_lens):
        ids = np.ascontiguousarray(seq_ids, dtype=np.int64)
        nl = _i32(new_lens)
        _check(self._lib.pa_seqs_truncate(self._h, ids.size, ids.ctypes.data_as(_I64P), _ptr(nl),
                                          None))

    def free_many(self, seq_ids):
        ids = np.ascontiguousarray(seq_ids, dtype=np.int64)
        _check(self._lib.pa_seqs_free(self._h, ids.size, ids.ctypes.data_as(_I64P), None))

    def apply(self, ops, seq_ids, offsets, tokens, new_lens):
        """Mixed pool operations in one call (arrays as pa_pool_apply takes
        them); returns reused-token counts (int32, 0 for non-admissions)."""
        p = PackedOps(ops, seq_ids, offsets, tokens, new_lens)
        return self.apply_packed(p).copy()

    def apply_packed(self, p: PackedOps):
        """pa_pool_apply on pre-packed operations; returns p's n_cached view."""
        if p.n:
            _check(self._lib.pa_pool_apply(self._h, p.n, *p.addrs, None))
        return p.n_cached[:p.n]

    def prepare_launch(self, ops, inp: LaunchInputs, buf: LaunchBuffers, kind: int, n_q: int,
                       num_q_heads: int, num_kv_heads: int, head_dim: int, dtype: int,
                       num_cus: int = 0, shared_prefix: bool = True, info=None):
        """pa_prepare_launch: ``ops`` (PackedOps or None) applied, then the
        metadata of ``inp`` and its plan written into ``buf``; returns the
        PlanInfo (``info`` is reused when given)."""
        if inp.n > buf.rows or inp.total_q > buf.slot_mapping.size:
            raise ValueError("prepare_launch: launch larger than its buffers")
        if info is None:
            info = PlanInfo()
        if ops is not None and ops.n:
            n_ops, oa = ops.n, ops.addrs
        else:
            n_ops, oa = 0, (0, 0, 0, 0, 0, 0)
        bt, sl, cu, sm, pl = buf.addrs
        _check(self._lib.pa_prepare_launch(
            self._h, n_ops, *oa, inp.n, *inp.addrs, buf.max_blocks, bt, sl, cu, sm,
            buf.slot_mapping.size, int(kind), int(n_q), int(num_q_heads), int(num_kv_heads),
            int(head_dim), int(dtype), int(num_cus), 1 if shared_prefix else 0, pl,
            buf.plan.size, C.byref(info)))
        return info

    def seq_len(self, seq_id: int) -> int:
        n = C.c_int32(0)
        _check(self._lib.pa_seq_len(self._h, int(seq_id), C.byref(n)))
        return n.value

    def blocks_of(self, seq_id: int):
        n = C.c_int32(0)
        rc = self._lib.pa_seq_blocks(self._h, int(seq_id), None, 0, C.byref(n))
        if rc not in (PA_OK, PA_ERR_ARG):
            _check(rc)
        out = np.zeros(max(1, n.value), dtype=np.int32)
        _check(self._lib.pa_seq_blocks(self._h, int(seq_id), _ptr(out), out.size, C.byref(n)))
        return out[:n.value].tolist()

    def free_list(self):
        n = C.c_int32(0)
        out = np.zeros(self.num_blocks, dtype=np.int32)
        _check(self._lib.pa_pool_free_list(self._h, _ptr(out), out.size, C.byref(n)))
        return out[:n.value].tolist()

    def metadata(self, seq_ids, q_lens, max_blocks_per_seq: int, out=None):
        """Block table, seq_lens, cu_seqlens_q and slot_mapping (numpy int32).
        ``out`` may supply preallocated arrays (e.g. pinned) to fill."""
        ids = np.ascontiguousarray(seq_ids, dtype=np.int64)
        ql = _i32(q_lens)
        n = ids.size
        total = int(ql.sum()) if n else 0
        if out is None:
            out = {"block_table": np.empty((n, max_blocks_per_seq), np.int32),
                   "seq_lens": np.empty(n, np.int32), "cu_seqlens_q": np.empty(n + 1, np.int32),
                   "slot_mapping": np.empty(total, np.int32)}
        bt, sl, cu, sm = (out["block_table"], out["seq_lens"], out["cu_seqlens_q"],
                          out["slot_mapping"])
        _check(self._lib.pa_build_metadata(
            self._h, n, ids.ctypes.data_as(_I64P) if n else None, _ptr(ql) if n else None,
            int(max_blocks_per_seq), _ptr(bt) if n else None, _ptr(sl) if n else None, _ptr(cu),
            _ptr(sm) if sm.size else None, sm.size))
        return out


def form_batches(adapter_ids, prompt_lens, bucket_bounds):
    """pa_form_batches: returns (order, position, batches) where batches is a
    list of (adapter, bucket, original indices)."""
    a, ln, bb = _i32(adapter_ids), _i32(prompt_lens), _i32(bucket_bounds)
    n = a.size
    if ln.size != n:
        raise ValueError("adapter_ids and prompt_lens differ in length")
    order, position = np.zeros(max(n, 1), np.int32), np.zeros(max(n, 1), np.int32)
    offs = np.zeros(n + 1, np.int32)
    badp, bbuck = np.zeros(max(n, 1), np.int32), np.zeros(max(n, 1), np.int32)
    nb = C.c_int32(0)
    _check(lib().pa_form_batches(n, _ptr(a) if n else None, _ptr(ln) if n else None, bb.size,
                                 _ptr(bb) if bb.size else None, _ptr(order), _ptr(position),
                                 _ptr(offs), _ptr(badp), _ptr(bbuck), C.byref(nb)))
    batches = [(int(badp[b]), int(bbuck[b]), order[offs[b]:offs[b + 1]].tolist())
               for b in range(nb.value)]
    return order[:n].tolist(), position[:n].tolist(), batches


def plan(kind: int, n_q: int, seq_lens, cu_seqlens_q, num_q_heads: int, num_kv_heads: int,
         head_dim: int, block_size: int, dtype: int, num_cus: int = 0, out=None,
         block_table=None):
    """Build the launch plan on the host; returns (int32 plan array, PlanInfo).
    ``out`` (int32 array, e.g. a pinned staging view) is used when large
    enough.  ``block_table`` (host [n_seqs, max_blocks] int32) enables
    shared-prefix groups."""
    L = lib()
    sl, cu = _i32(seq_lens), _i32(cu_seqlens_q)
    n = sl.size
    info = PlanInfo()
    if block_table is not None and n:
        bt = _i32(block_table)
        bt_ptr, mb = _ptr(bt), int(bt.shape[1])
    else:
        bt_ptr, mb = None, 0
    args = (int(kind), int(n_q), n, _ptr(sl) if n else None, _ptr(cu), bt_ptr, mb,
            int(num_q_heads), int(num_kv_heads), int(head_dim), int(block_size), int(dtype),
            int(num_cus))
    if out is not None:
        rc = L.pa_attn_plan(*args, _ptr(out), out.size, C.byref(info))
        if rc == PA_OK:
            return out[:info.plan_words], info
        if not (rc == PA_ERR_ARG and info.plan_words > out.size):
            _check(rc)
    else:
        _check(L.pa_attn_plan(*args, None, 0, C.byref(info)))
    arr = np.zeros(max(1, info.plan_words), dtype=np.int32)
    _check(L.pa_attn_plan(*args, _ptr(arr), arr.size, C.byref(info)))
    return arr[:info.plan_words], info


def workspace_size(total_q: int, num_q_heads: int, head_dim: int, max_seq_len: int,
                   decode: bool = False) -> int:
    """Bound on the split-K workspace of any plan for such a launch
    (pa_attn_workspace_size, or pa_attn_decode_workspace_size with total_q
    the number of decode sequences)."""
    n = C.c_size_t(0)
    fn = lib().pa_attn_decode_workspace_size if decode else lib().pa_attn_workspace_size
    _check(fn(int(total_q), int(num_q_heads), int(head_dim), int(max_seq_len), C.byref(n)))
    return int(n.value)


def _dptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _stream(stream) -> int:
    if stream is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    return int(getattr(stream, "cuda_stream", stream))


_hip = None
HIP_EVENT_DISABLE_TIMING, HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x2, 0x20000000


def _hip_runtime():
    """The HIP runtime libpa links against (the process's only copy: torch
    loads the same soname)."""
    global _hip
    if _hip is None:
        lib()
        h = C.CDLL("libamdhip64.so.7")
        h.hipEventCreateWithFlags.argtypes = [C.POINTER(_P), C.c_uint]
        h.hipEventRecord.argtypes = [_P, _P]
        h.hipEventSynchronize.argtypes = [_P]
        h.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), _P, _P]
        h.hipEventDestroy.argtypes = [_P]
        for f in ("hipEventCreateWithFlags", "hipEventRecord", "hipEventSynchronize",
                  "hipEventElapsedTime", "hipEventDestroy"):
            getattr(h, f).restype = C.c_int
        _hip = h
    return _hip


class StreamEvent:
    """A HIP event recorded without a system-scope fence.

    A default event record writes back and invalidates the GPU caches at
    system scope so the host can read device results once the event
    completes; in a stream of back-to-back kernels each such record costs
    several microseconds of idle device.  Nothing waiting on these events
    reads device memory: the staging buffers use them to learn that an
    upload has finished reading pinned host memory (its loads bypass the
    caches), and the benchmark uses them for timing only."""

    def __init__(self, timing: bool = False):
        self._h = _hip_runtime()
        self._ev = _P()
        flags = HIP_EVENT_DISABLE_SYSTEM_FENCE | (0 if timing else HIP_EVENT_DISABLE_TIMING)
        self._rc("hipEventCreateWithFlags", self._h.hipEventCreateWithFlags(C.byref(self._ev), flags))

    @staticmethod
    def _rc(what: str, rc: int):
        if rc != 0:
            raise PaError(PA_ERR_LAUNCH, f"{what} returned HIP error {rc}")

    def record(self, stream=None):
        self._rc("hipEventRecord", self._h.hipEventRecord(self._ev, _stream(stream)))

    def synchronize(self):
        self._rc("hipEventSynchronize", self._h.hipEventSynchronize(self._ev))

    def elapsed_time(self, end: "StreamEvent") -> float:
        """Milliseconds from this event to end (both recorded and complete)."""
        ms = C.c_float()
        self._rc("hipEventElapsedTime", self._h.hipEventElapsedTime(C.byref(ms), self._ev, end._ev))
        return float(ms.value)

    def __del__(self):
        if getattr(self, "_ev", None) and _hip is not None:
            _hip.hipEventDestroy(self._ev)
            self._ev = None


# Per-device workspace held by pa_attn_decode_noalloc (PA_NOALLOC_WORKSPACE_BYTES).
NOALLOC_WORKSPACE_BYTES = 32 << 20


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return PA_BF16
    if t.dtype == torch.float32:
        return PA_F32
    raise PaError(PA_ERR_UNSUPPORTED, f"dtype {t.dtype}")


def stage_upload(dst, src, nbytes: int, stream=None):
    """Copy the first nbytes of pinned host tensor src into device tensor dst
    with the library's upload kernel (pa_stage_upload)."""
    _check(lib().pa_stage_upload(_dptr(dst), _dptr(src), int(nbytes), _stream(stream)))


def cache_dims(k_cache, v_cache):
    """(num_blocks, num_kv_heads, head_dim, block_size) of a paged cache: the
    value cache is [NB, Hkv, D, bs]; the key cache holds as many elements in
    the grouped layout [NB, Hkv, D / 32, bs, 32]."""
    nb, hkv, d, bs = v_cache.shape
    if k_cache.numel() != v_cache.numel() or k_cache.dtype != v_cache.dtype:
        raise PaError(PA_ERR_ARG, "key and value caches differ in size or dtype")
    return int(nb), int(hkv), int(d), int(bs)


def kv_append(k_new, v_new, slot_mapping, k_cache, v_cache, stream=None):
    """Scatter new K/V ([T, Hkv, D] device tensors) into the paged cache."""
    nb, hkv, d, bs = cache_dims(k_cache, v_cache)
    _check(lib().pa_kv_append(_dptr(k_new), _dptr(v_new), _dptr(slot_mapping),
                              int(slot_mapping.numel()), _dptr(k_cache), _dptr(v_cache), nb, hkv,
                              d, bs, _dtype_code(k_cache), _stream(stream)))


def attention(kind: int, q, k_cache, v_cache, block_table, seq_lens, cu_seqlens_q, plan_dev,
              info: PlanInfo, workspace, out, lse=None, scale=None, stream=None):
    """Paged attention (prefill / decode / verify by ``kind``) on device tensors."""
    nb, hkv, d, bs = cache_dims(k_cache, v_cache)
    total_q, hq, _ = q.shape
    n_seqs = int(seq_lens.numel())
    if scale is None:
        scale = d ** -0.5
    fn = {KIND_PREFILL: lib().pa_attn_prefill, KIND_DECODE: lib().pa_attn_decode,
          KIND_VERIFY: lib().pa_attn_verify}[kind]
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(fn(_dptr(q), _dptr(k_cache), _dptr(v_cache), nb, _dptr(block_table),
              int(block_table.shape[1]), _dptr(seq_lens), _dptr(cu_seqlens_q), n_seqs, total_q,
              hq, hkv, d, bs, float(scale), _dtype_code(q), _dptr(plan_dev), C.byref(info),
              _dptr(workspace), ws_bytes, _dptr(out), _dptr(lse), _stream(stream)))


def set_launch_events(start: "StreamEvent | None", stop: "StreamEvent | None"):
    """The next attention call on this thread records start when its first
    kernel starts and stop when its last kernel ends (events carried by the
    kernel dispatches, no event packets between kernels)."""
    _check(lib().pa_set_launch_events(start._ev if start is not None else None,
                                      stop._ev if stop is not None else None))


def attention_decode_noalloc(q, k_cache, v_cache, block_table, seq_lens, cu_seqlens_q, plan_dev,
                             info: PlanInfo, out, lse=None, scale=None, stream=None):
    """Decode through pa_attn_decode_noalloc (split-K partials in the
    library's per-device array; no workspace argument)."""
    nb, hkv, d, bs = cache_dims(k_cache, v_cache)
    total_q, hq, _ = q.shape
    n_seqs = int(seq_lens.numel())
    if scale is None:
        scale = d ** -0.5
    _check(lib().pa_attn_decode_noalloc(
        _dptr(q), _dptr(k_cache), _dptr(v_cache), nb, _dptr(block_table),
        int(block_table.shape[1]), _dptr(seq_lens), _dptr(cu_seqlens_q), n_seqs, total_q, hq, hkv,
        d, bs, float(scale), _dtype_code(q), _dptr(plan_dev), C.byref(info), _dptr(out),
        _dptr(lse), _stream(stream)))
