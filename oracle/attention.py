"""float64 attention oracle over a paged KV store (test infrastructure only).

What the method computes has a plain definition: serving a request's suffix
against cached prefix blocks gives exactly the attention it would get if the
prefix were recomputed (paper, Section 3: shared policy prefixes should not be
recomputed; Section 2: PagedAttention stores the same keys and values in
blocks addressed through a block table).  So this oracle is that definition
written out -- causal scaled-dot-product attention over each request's logical
token sequence, which it rebuilds from its own block table and its own paged
store:

    s_t = (q . k_t) / sqrt(D)            for every key t <= a
    o   = sum_t exp(s_t - m) v_t / sum_t exp(s_t - m),  m = max_t s_t
    lse = m + log sum_t exp(s_t - m)

where a query at logical position ``a`` sees keys ``0..a`` (queries are the
last ``n`` positions of the sequence), and q-head ``h`` reads kv-head
``h // G`` with ``G = Hq / Hkv`` (grouped-query attention with contiguous
groups, the Llama/Qwen convention the configurations follow).

Cache layout (the same definition the library documents, implemented here
independently):  ``k_cache[NB, Hkv, bs, D]`` holds key ``d`` of the token in
block ``b`` at offset ``o`` at ``k_cache[b, h, o, d]``; ``v_cache[NB, Hkv, D,
bs]`` holds the value at ``v_cache[b, h, d, o]``.  A token's slot is
``block * bs + offset``.
"""
from __future__ import annotations

import numpy as np


def new_cache(num_blocks: int, num_kv_heads: int, head_dim: int, block_size: int):
    """Zero-filled float64 paged store (K in [NB,Hkv,bs,D], V in [NB,Hkv,D,bs])."""
    k = np.zeros((num_blocks, num_kv_heads, block_size, head_dim), dtype=np.float64)
    v = np.zeros((num_blocks, num_kv_heads, head_dim, block_size), dtype=np.float64)
    return k, v


def kv_append(k_cache, v_cache, slot_mapping, k_new, v_new):
    """Store token ``i``'s keys/values at slot ``slot_mapping[i]``; a negative
    slot means "skip this token"."""
    bs = k_cache.shape[2]
    for i, slot in enumerate(np.asarray(slot_mapping).tolist()):
        if slot < 0:
            continue
        b, o = divmod(slot, bs)
        k_cache[b, :, o, :] = k_new[i]
        v_cache[b, :, :, o] = v_new[i]


def gather_sequence(k_cache, v_cache, block_row, seq_len: int):
    """Rebuild the logical K, V ``[L, Hkv, D]`` of one request from its block
    table row."""
    bs = k_cache.shape[2]
    t = np.arange(seq_len)
    blocks = np.asarray(block_row)[t // bs]
    off = t % bs
    K = k_cache[blocks, :, off, :]
    V = v_cache[blocks, :, :, off]
    return K.astype(np.float64), V.astype(np.float64)


def softmax_attention(q, K, V, visible, scale):
    """One head: ``q [n, D]``, ``K, V [L, D]``, ``visible [n, L]`` bool.
    Returns ``o [n, D]``, ``lse [n]`` and the probability rows ``[n, L]``.
    A row with no visible key gives o = 0 and lse = -inf."""
    s = (q.astype(np.float64) @ K.astype(np.float64).T) * scale
    s = np.where(visible, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    m_safe = np.where(np.isfinite(m), m, 0.0)
    p = np.exp(s - m_safe)
    l = p.sum(axis=1, keepdims=True)
    l_safe = np.where(l > 0, l, 1.0)
    o = (p @ V.astype(np.float64)) / l_safe
    lse = np.where(l[:, 0] > 0, m_safe[:, 0] + np.log(l_safe[:, 0]), -np.inf)
    return o, lse, p / l_safe


def causal_visible(n: int, L: int) -> np.ndarray:
    """Bottom-right causal mask: the ``n`` queries are positions ``L-n..L-1``."""
    pos = L - n + np.arange(n)
    return np.arange(L)[None, :] <= pos[:, None]


def sequence_attention(q, K, V, scale, rows=None):
    """Attention of one request.  ``q [n, Hq, D]`` are its last ``n`` positions,
    ``K, V [L, Hkv, D]`` its logical sequence.  Returns ``o [n, Hq, D]`` and
    ``lse [n, Hq]`` (float64).  ``rows`` optionally restricts the computation
    to a list of ``(i, h)`` pairs (other entries are left as NaN)."""
    n, Hq, D = q.shape
    L, Hkv, _ = K.shape
    G = Hq // Hkv
    vis = causal_visible(n, L)
    o = np.full((n, Hq, D), np.nan)
    lse = np.full((n, Hq), np.nan)
    if rows is None:
        for h in range(Hq):
            g = h // G
            oh, lh, _ = softmax_attention(q[:, h, :], K[:, g, :], V[:, g, :], vis, scale)
            o[:, h, :], lse[:, h] = oh, lh
    else:
        for i, h in rows:
            g = h // G
            oh, lh, _ = softmax_attention(q[i:i + 1, h, :], K[:, g, :], V[:, g, :],
                                          vis[i:i + 1], scale)
            o[i, h, :], lse[i, h] = oh[0], lh[0]
    return o, lse


def paged_attention(q, k_cache, v_cache, block_table, seq_lens, cu_seqlens_q,
                    num_kv_heads, scale=None, rows=None):
    """Varlen paged attention: request ``r`` owns query rows
    ``cu_seqlens_q[r]:cu_seqlens_q[r+1]`` of ``q [T, Hq, D]``.

    ``rows`` optionally lists ``(token, head)`` pairs to compute (the others
    stay NaN) so large launches can be checked on samples."""
    T, Hq, D = q.shape
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    out = np.full((T, Hq, D), np.nan)
    lse = np.full((T, Hq), np.nan)
    want = None
    if rows is not None:
        want = {}
        for t, h in rows:
            want.setdefault(int(t), []).append(int(h))
    for r in range(len(seq_lens)):
        a, b = int(cu_seqlens_q[r]), int(cu_seqlens_q[r + 1])
        if b == a:
            continue
        if want is not None:
            sub = [(t - a, h) for t in range(a, b) for h in want.get(t, [])]
            if not sub:
                continue
        else:
            sub = None
        K, V = gather_sequence(k_cache, v_cache, block_table[r], int(seq_lens[r]))
        o, l = sequence_attention(np.asarray(q[a:b], dtype=np.float64), K, V, scale, sub)
        out[a:b], lse[a:b] = o, l
    return out, lse


def merge_partials(o_parts, lse_parts):
    """Combine attention results over disjoint key sets by their log-sum-exp:
    o = sum_i exp(lse_i - lse) o_i, lse = log sum_i exp(lse_i)."""
    lse_parts = np.stack(lse_parts)
    m = lse_parts.max(axis=0)
    w = np.exp(lse_parts - m)
    lse = m + np.log(w.sum(axis=0))
    o = sum(np.exp(lp - lse)[..., None] * op for lp, op in zip(lse_parts, o_parts))
    return o, lse
