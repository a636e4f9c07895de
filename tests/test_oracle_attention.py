"""Pins for the float64 attention oracle (CPU only).

Each pin is something other than the oracle itself:

* pure-Python brute force on tiny shapes (1e-12);
* a library routine: torch ``scaled_dot_product_attention`` in float64 with an
  explicit bottom-right causal mask and ``repeat_interleave`` GQA (1e-10);
* closed forms (zero keys, constant values, one visible key, a "needle");
* invariants: probability rows sum to 1, paged == contiguous, permuting
  physical blocks leaves the result unchanged, shared prefix == duplicated
  prefix, decode == last row of prefill, verify == sequential decodes,
  chunked == one-shot prefill, log-sum-exp merge of disjoint key sets == all.

A plausible slip in the oracle -- a missing 1/sqrt(D), an off-by-one in the
causal boundary, h % Hkv instead of h // G, a transposed K or V layout, a
wrong log-sum-exp -- fails at least one of them.
"""
import math

import numpy as np
import pytest
import torch

from oracle import brute
from oracle.apc import PrefixCacheOracle
from oracle.attention import (causal_visible, gather_sequence, kv_append, merge_partials,
                              new_cache, paged_attention, sequence_attention, softmax_attention)


def _rand(r, *shape):
    return r.standard_normal(shape)


@pytest.mark.parametrize("seed", range(12))
def test_brute_force_matches(seed):
    r = np.random.default_rng(seed)
    Hkv = int(r.integers(1, 3))
    G = int(r.integers(1, 4))
    Hq, D = Hkv * G, int(r.integers(2, 9))
    L = int(r.integers(1, 41))
    n = int(r.integers(1, L + 1))
    q, K, V = _rand(r, n, Hq, D), _rand(r, L, Hkv, D), _rand(r, L, Hkv, D)
    o, lse = sequence_attention(q, K, V, 1.0 / math.sqrt(D))
    ob, lb = brute.attention(q.tolist(), K.tolist(), V.tolist(), Hq, Hkv)
    np.testing.assert_allclose(o, np.array(ob), rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, np.array(lb), rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", range(8))
def test_torch_sdpa_float64(seed):
    r = np.random.default_rng(100 + seed)
    Hkv, G = int(r.integers(1, 5)), int(r.integers(1, 9))
    Hq, D = Hkv * G, int(r.choice([16, 64, 128]))
    L = int(r.integers(1, 300))
    n = int(r.integers(1, L + 1))
    q, K, V = _rand(r, n, Hq, D), _rand(r, L, Hkv, D), _rand(r, L, Hkv, D)
    o, _ = sequence_attention(q, K, V, 1.0 / math.sqrt(D))
    tq = torch.from_numpy(q).permute(1, 0, 2)                       # [Hq, n, D]
    tk = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(G, 0)  # [Hq, L, D]
    tv = torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(G, 0)
    mask = torch.ones(n, L, dtype=torch.bool).tril(diagonal=L - n)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask)
    np.testing.assert_allclose(o, ref.permute(1, 0, 2).numpy(), rtol=0, atol=1e-10)


def test_zero_keys_give_prefix_mean_and_log_count():
    r = np.random.default_rng(1)
    L, n, Hq, Hkv, D = 37, 9, 6, 2, 16
    q, V = _rand(r, n, Hq, D), _rand(r, L, Hkv, D)
    K = np.zeros((L, Hkv, D))
    o, lse = sequence_attention(q, K, V, 1.0 / math.sqrt(D))
    for i in range(n):
        a = L - n + i
        for h in range(Hq):
            np.testing.assert_allclose(o[i, h], V[:a + 1, h // 3].mean(0), atol=1e-13)
            assert abs(lse[i, h] - math.log(a + 1)) < 1e-13


def test_constant_values_and_single_key():
    r = np.random.default_rng(2)
    L, Hq, Hkv, D = 20, 4, 4, 8
    q, K = _rand(r, L, Hq, D), _rand(r, L, Hkv, D)
    c = _rand(r, Hkv, D)
    V = np.broadcast_to(c, (L, Hkv, D)).copy()
    o, _ = sequence_attention(q, K, V, 1.0 / math.sqrt(D))
    np.testing.assert_allclose(o, np.broadcast_to(c, (L, Hq, D)), atol=1e-13)
    # the first position sees only key 0
    V = _rand(r, L, Hkv, D)
    o, lse = sequence_attention(q, K, V, 1.0 / math.sqrt(D))
    np.testing.assert_allclose(o[0], V[0], atol=1e-14)
    np.testing.assert_allclose(lse[0], np.einsum("hd,hd->h", q[0], K[0]) / math.sqrt(D), atol=1e-13)


def test_needle():
    """Q = alpha e1, K[t*] = beta e1, other keys 0: o = (e^s v* + sum_{t!=t*} v_t) / (e^s + a)."""
    r = np.random.default_rng(3)
    L, n, Hkv, G, D = 50, 4, 2, 2, 64
    Hq = Hkv * G
    alpha, beta = 8.0, 20.0
    sigma = alpha * beta / math.sqrt(D)
    needles = [11, 30]                       # a different needle position per kv-head
    q = np.zeros((n, Hq, D)); q[:, :, 0] = alpha
    K = np.zeros((L, Hkv, D))
    for g, t in enumerate(needles):
        K[t, g, 0] = beta
    V = _rand(r, L, Hkv, D)
    o, _ = sequence_attention(q, K, V, 1.0 / math.sqrt(D))
    for i in range(n):
        a = L - n + i
        for h in range(Hq):
            g, ts = h // G, needles[h // G]
            others = V[:a + 1, g].sum(0) - V[ts, g]
            want = (math.exp(sigma) * V[ts, g] + others) / (math.exp(sigma) + a)
            np.testing.assert_allclose(o[i, h], want, rtol=1e-12, atol=1e-13)


def test_rows_sum_to_one_and_respect_mask():
    r = np.random.default_rng(4)
    n, L, D = 7, 23, 8
    vis = causal_visible(n, L)
    _, _, p = softmax_attention(_rand(r, n, D), _rand(r, L, D), _rand(r, L, D), vis, 0.3)
    np.testing.assert_allclose(p.sum(1), 1.0, atol=1e-14)
    assert np.all(p[~vis] == 0)
    assert vis.sum(1).tolist() == list(range(L - n + 1, L + 1))


def test_lse_merge_of_disjoint_keys():
    r = np.random.default_rng(5)
    n, L, D = 5, 40, 16
    q, K, V = _rand(r, n, D), _rand(r, L, D), _rand(r, L, D)
    vis = causal_visible(n, L)
    o, lse, _ = softmax_attention(q, K, V, vis, 0.25)
    cut = np.zeros_like(vis); cut[:, :17] = True
    o1, l1, _ = softmax_attention(q, K, V, vis & cut, 0.25)
    o2, l2, _ = softmax_attention(q, K, V, vis & ~cut, 0.25)
    om, lm = merge_partials([o1, o2], [l1, l2])
    np.testing.assert_allclose(om, o, atol=1e-13)
    np.testing.assert_allclose(lm, lse, atol=1e-13)


# ---------------------------------------------------------------------------
# paged-store invariants
# ---------------------------------------------------------------------------

def _paged_setup(seed, free_order, prefix_cached=True, bs=4, Hq=6, Hkv=2, D=8):
    """Three requests sharing a 12-token prefix; returns the oracle result and
    the logical K/V each request should see."""
    r = np.random.default_rng(seed)
    P, S = 12, [5, 9, 3]
    pre_tok = list(range(1000, 1000 + P))
    pre_k, pre_v = _rand(r, P, Hkv, D), _rand(r, P, Hkv, D)
    suf = [(_rand(r, s, Hkv, D), _rand(r, s, Hkv, D)) for s in S]
    q = _rand(r, sum(S), Hq, D)
    nb = len(free_order)
    pool = PrefixCacheOracle(nb, bs, free_order)
    kc, vc = new_cache(nb, Hkv, D, bs)
    if prefix_cached:
        pool.add(99, pre_tok)
        md = pool.metadata([99], [P], 16)
        kv_append(kc, vc, md["slot_mapping"], pre_k, pre_v)
        pool.free_seq(99)
    # without a cached prefix each request gets its own prefix token ids (same
    # K/V values), so nothing is shared and every request stores its own copy
    toks = [(pre_tok if prefix_cached else [t + 100 * (i + 1) for t in pre_tok])
            + list(range(10 * i, 10 * i + S[i])) for i in range(3)]
    nc = [pool.add(i, toks[i]) for i in range(3)]
    q_lens = [P + S[i] - nc[i] for i in range(3)]
    md = pool.metadata([0, 1, 2], q_lens, 16)
    k_new = np.concatenate([np.concatenate([pre_k[nc[i]:], suf[i][0]]) for i in range(3)])
    v_new = np.concatenate([np.concatenate([pre_v[nc[i]:], suf[i][1]]) for i in range(3)])
    kv_append(kc, vc, md["slot_mapping"], k_new, v_new)
    qq = np.concatenate([np.concatenate([_rand(np.random.default_rng(7 + i), q_lens[i] - S[i], Hq, D),
                                         q[sum(S[:i]):sum(S[:i + 1])]]) for i in range(3)])
    out, lse = paged_attention(qq, kc, vc, md["block_table"], md["seq_lens"], md["cu_seqlens_q"], Hkv)
    logical = [(np.concatenate([pre_k, suf[i][0]]), np.concatenate([pre_v, suf[i][1]])) for i in range(3)]
    # keep only the suffix rows (the part every variant computes)
    rows = np.concatenate([np.arange(md["cu_seqlens_q"][i + 1] - S[i], md["cu_seqlens_q"][i + 1])
                           for i in range(3)])
    return out[rows], lse[rows], md, kc, vc, logical, q, S


def test_paged_equals_contiguous():
    order = list(np.random.default_rng(0).permutation(40))
    out, lse, md, kc, vc, logical, q, S = _paged_setup(0, order)
    off = 0
    for i in range(3):
        K, V = gather_sequence(kc, vc, md["block_table"][i], int(md["seq_lens"][i]))
        np.testing.assert_array_equal(K, logical[i][0])
        np.testing.assert_array_equal(V, logical[i][1])
        o, l = sequence_attention(q[off:off + S[i]], logical[i][0], logical[i][1], 1 / math.sqrt(8))
        np.testing.assert_array_equal(out[off:off + S[i]], o)
        off += S[i]


def test_block_permutation_and_shared_vs_duplicated_prefix():
    base = _paged_setup(0, list(range(40)))
    perm = _paged_setup(0, list(np.random.default_rng(9).permutation(40)))
    dup = _paged_setup(0, list(np.random.default_rng(10).permutation(40)), prefix_cached=False)
    assert not np.array_equal(base[2]["block_table"], perm[2]["block_table"])
    # with the prefix cached, all three share their first 3 blocks; without, none do
    assert len({tuple(r[:3]) for r in perm[2]["block_table"]}) == 1
    assert len({tuple(r[:3]) for r in dup[2]["block_table"]}) == 3
    np.testing.assert_array_equal(base[0], perm[0])
    np.testing.assert_array_equal(base[0], dup[0])
    np.testing.assert_array_equal(base[1], dup[1])


def test_decode_verify_chunked_consistency():
    r = np.random.default_rng(11)
    L, Hq, Hkv, D = 61, 8, 2, 16
    q, K, V = _rand(r, L, Hq, D), _rand(r, L, Hkv, D), _rand(r, L, Hkv, D)
    sc = 1 / math.sqrt(D)
    full, full_l = sequence_attention(q, K, V, sc)                    # one-shot prefill
    dec, dec_l = sequence_attention(q[-1:], K, V, sc)                 # decode
    np.testing.assert_allclose(dec, full[-1:], atol=1e-13)
    ver, _ = sequence_attention(q[-5:], K, V, sc)                     # verify n_q = 5
    seq = np.concatenate([sequence_attention(q[L - 5 + j:L - 4 + j], K[:L - 4 + j], V[:L - 4 + j], sc)[0]
                          for j in range(5)])
    np.testing.assert_allclose(ver, seq, atol=1e-13)
    chunks = [sequence_attention(q[a:b], K[:b], V[:b], sc)[0] for a, b in ((0, 20), (20, 45), (45, 61))]
    np.testing.assert_allclose(np.concatenate(chunks), full, atol=1e-13)
