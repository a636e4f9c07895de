"""Algorithmic work of a launch (for throughput and roofline figures).

Counts what the computation requires, not what a kernel happens to do:

* FLOPs: 4 * D * Hq per visible (query, key) pair -- 2 * D for q.k and 2 * D
  for the weighted value sum; masked pairs and exponentials are not counted.
  Query i of a request with n queries and L keys sees L - n + i + 1 keys.
* unique bytes: every distinct KV slot the launch reads, once (a prefix block
  shared by many requests counts once), K and V, plus q, out, lse, the used
  block-table entries and the length arrays.
* logical bytes: the same with every request's keys counted separately.
* append bytes: new K and V read once and written once.
"""
from __future__ import annotations

import numpy as np

MI355X_PEAKS = {
    "hbm_gbs": 8000.0,          # HBM3E, GB/s
    "bf16_tflops": 2500.0,      # dense bf16 MFMA, TFLOP/s
    "fp32_vector_tflops": 157.3,
}
ELEM = {"bf16": 2, "f32": 4}


def attention_flops(seq_lens, cu_seqlens_q, num_q_heads, head_dim) -> float:
    L = np.asarray(seq_lens, dtype=np.float64)
    n = np.diff(np.asarray(cu_seqlens_q, dtype=np.float64))
    pairs = n * (L - n) + n * (n + 1) / 2
    return float(4.0 * head_dim * num_q_heads * pairs.sum())


def _slots(block_table, seq_lens, cu_seqlens_q, block_size):
    out = []
    n = np.diff(np.asarray(cu_seqlens_q))
    for r, L in enumerate(np.asarray(seq_lens).tolist()):
        if n[r] == 0:
            continue
        t = np.arange(L, dtype=np.int64)
        out.append(block_table[r][t // block_size].astype(np.int64) * block_size + t % block_size)
    return np.concatenate(out) if out else np.zeros(0, np.int64)


def attention_bytes(meta, cfg, unique: bool = True) -> float:
    s = ELEM[cfg.dtype]
    bt, L, cu = meta["block_table"], meta["seq_lens"], meta["cu_seqlens_q"]
    n = np.diff(cu)
    live = n > 0
    if unique:
        kv_tokens = np.unique(_slots(bt, L, cu, cfg.block_size)).size
    else:
        kv_tokens = int(np.asarray(L)[live].sum())
    T = int(cu[-1])
    kv = 2.0 * kv_tokens * cfg.num_kv_heads * cfg.head_dim * s
    qo = 2.0 * T * cfg.num_q_heads * cfg.head_dim * s + 4.0 * T * cfg.num_q_heads
    tables = 4.0 * float(np.ceil(np.asarray(L)[live] / cfg.block_size).sum()) + 8.0 * len(L) + 4.0
    return kv + qo + tables


def append_bytes(n_tokens, cfg) -> float:
    return 2.0 * 2.0 * n_tokens * cfg.num_kv_heads * cfg.head_dim * ELEM[cfg.dtype]
