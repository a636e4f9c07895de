"""Pins for the prefix-cache bookkeeping oracle (CPU only).

* a hand-worked example (``tests/golden/apc_worked_example.json``) derived by
  hand from the block-table / prefix-reuse rules;
* invariants the problem fixes, on seeded random workloads: shared prefixes
  map to identical leading blocks, private blocks are disjoint, query slots
  are distinct and lie inside their own sequence's blocks, allocation follows
  the caller's free-list order, and blocks are conserved.
"""
import json
import os
from collections import Counter

import numpy as np
import pytest

from oracle.apc import NoBlocksError, OracleError, PrefixCacheOracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "apc_worked_example.json")


def _tokens(spec, prefix):
    if isinstance(spec, list):
        return spec
    if spec == "prefix":
        return list(prefix)
    assert spec.startswith("prefix+")
    return list(prefix) + json.loads(spec[len("prefix+"):])


def run_golden(make_pool, apply_op):
    g = json.load(open(GOLDEN))
    pool = make_pool(g["num_blocks"], g["block_size"], g["free_order"])
    for st in g["steps"]:
        res = apply_op(pool, st, _tokens(st.get("tokens", []), g["prefix"]) if "tokens" in st else None)
        if "expect_error" in st:
            assert res == ("error", st["expect_error"]), st
        if "expect_n_cached" in st:
            assert res == st["expect_n_cached"], st
        if "expect_blocks" in st:
            assert pool.blocks_of(st["seq"]) == st["expect_blocks"], st
        if "expect_free" in st:
            assert pool.free_list() == st["expect_free"], st
        if st["op"] == "metadata":
            for key in ("block_table", "seq_lens", "cu_seqlens_q", "slot_mapping"):
                assert np.asarray(res[key]).tolist() == st["expect_" + key], (st, key)


def _oracle_apply(pool, st, toks):
    try:
        if st["op"] == "add":
            return pool.add(st["seq"], toks)
        if st["op"] == "extend":
            return pool.extend(st["seq"], toks)
        if st["op"] == "free":
            return pool.free_seq(st["seq"])
        if st["op"] == "truncate":
            return pool.truncate(st["seq"], st["n"])
        if st["op"] == "metadata":
            return pool.metadata(st["seqs"], st["q_lens"], st["max_blocks"])
    except OracleError as e:
        return ("error", e.code)
    raise ValueError(st["op"])


def test_worked_example():
    run_golden(PrefixCacheOracle, _oracle_apply)


def _random_batch(seed, n_prefix=3, R=12, bs=8, vocab=5):
    """Small random workload: a few shared prefixes (some not block aligned),
    requests mixing them, a tiny vocabulary so accidental sharing occurs."""
    r = np.random.default_rng(seed)
    prefixes = [r.integers(0, vocab, size=int(r.integers(1, 5 * bs))).tolist()
                for _ in range(n_prefix)]
    reqs = []
    for i in range(R):
        p = int(r.integers(0, n_prefix))
        suf = r.integers(0, vocab, size=int(r.integers(1, 3 * bs))).tolist()
        reqs.append((p, prefixes[p] + suf))
    return prefixes, reqs


@pytest.mark.parametrize("seed", range(20))
def test_invariants_random(seed):
    bs = 8
    prefixes, reqs = _random_batch(seed, bs=bs)
    nb = 400
    order = np.random.default_rng(seed + 99).permutation(nb).tolist()
    pool = PrefixCacheOracle(nb, bs, order)
    # pre-populate the prefixes
    for p, toks in enumerate(prefixes):
        pool.add(1000 + p, toks)
        pool.free_seq(1000 + p)
    # allocation pops the caller's order; each prefix's partial tail block went
    # back to the end of the free list
    n_tail = sum(1 for toks in prefixes if len(toks) % bs)
    F = pool.free_list()
    popped = nb - len(F) + n_tail
    assert F[:nb - popped] == order[popped:]
    assert set(F[nb - popped:]) <= set(order[:popped]) and len(F) - (nb - popped) == n_tail
    n_cached = {}
    for i, (p, toks) in enumerate(reqs):
        n_cached[i] = pool.add(i, toks)
    q_lens = [len(t) - n_cached[i] for i, (_, t) in enumerate(reqs)]
    md = pool.metadata(list(range(len(reqs))), q_lens, 16)
    bt, sl, cu, slots = md["block_table"], md["seq_lens"], md["cu_seqlens_q"], md["slot_mapping"]
    # n_cached is whole blocks, leaves >= 1 token, and equals the longest
    # block-aligned prefix shared with a pre-populated prefix (capped)
    for i, (p, toks) in enumerate(reqs):
        L = len(toks)
        assert n_cached[i] % bs == 0 and n_cached[i] <= L - 1
        best = 0
        for pre in prefixes:
            k = 0
            while (k + 1) * bs <= min(len(pre), L - 1) and pre[:(k + 1) * bs] == toks[:(k + 1) * bs]:
                k += 1
            best = max(best, k)
        # earlier requests in the batch can add registered blocks, so hits are
        # at least what the prefixes alone give
        assert n_cached[i] >= best * bs
    # equal token prefixes (block aligned, within the cached run) -> equal blocks
    for i in range(len(reqs)):
        for j in range(i + 1, len(reqs)):
            ti, tj = reqs[i][1], reqs[j][1]
            k = 0
            while ((k + 1) * bs <= min(n_cached[i], n_cached[j])
                   and ti[:(k + 1) * bs] == tj[:(k + 1) * bs]):
                assert bt[i, k] == bt[j, k]
                k += 1
    # no block twice in a row; blocks used by one request only are disjoint
    use = Counter()
    for i in range(len(reqs)):
        row = [b for b in bt[i] if b >= 0]
        assert len(row) == len(set(row)) == -(-len(reqs[i][1]) // bs)
        use.update(row)
    # a block shared by two rows sits at the same logical index, is full in
    # both, and both hold the same tokens up to and including it
    where = {}
    for i in range(len(reqs)):
        for k, b in enumerate(bt[i].tolist()):
            if b >= 0:
                where.setdefault(b, []).append((i, k))
    for b, occ in where.items():
        if len(occ) > 1:
            (i0, k0) = occ[0]
            for (i1, k1) in occ[1:]:
                assert k1 == k0
                n = (k0 + 1) * bs
                assert len(reqs[i0][1]) >= n and len(reqs[i1][1]) >= n
                assert reqs[i0][1][:n] == reqs[i1][1][:n]
    # query slots: distinct, inside the sequence's own (non-cached) blocks
    assert len(set(slots.tolist())) == len(slots)
    for i in range(len(reqs)):
        for k, s in enumerate(slots[cu[i]:cu[i + 1]].tolist()):
            t = sl[i] - q_lens[i] + k
            assert s // bs == bt[i, t // bs] and s % bs == t % bs
            assert s // bs not in bt[i][:n_cached[i] // bs]
    # conservation: free + cached-idle + in use == all blocks
    in_use = set(int(b) for b in bt.ravel() if b >= 0)
    idle = {b for b in pool.registered if pool.ref[b] == 0}
    assert len(pool.free_list()) + len(idle) + len(in_use) == nb
    assert not (set(pool.free_list()) & (idle | in_use))


def test_allocation_follows_free_order():
    nb, bs = 64, 4
    order = np.random.default_rng(7).permutation(nb).tolist()
    pool = PrefixCacheOracle(nb, bs, order)
    got = []
    for i in range(5):
        pool.add(i, list(range(100 * i, 100 * i + 9)))  # 3 blocks each, distinct tokens
        got += pool.blocks_of(i)
    assert got == order[:15]


def test_extend_truncate_restores_pool():
    pool = PrefixCacheOracle(32, 4, list(range(31, -1, -1)))
    pool.add(0, list(range(10)))
    before_free, before_blocks = pool.free_list(), pool.blocks_of(0)
    pool.extend(0, list(range(50, 63)))
    assert len(pool.blocks_of(0)) == -(-23 // 4)
    pool.truncate(0, 10)
    assert pool.free_list() == before_free and pool.blocks_of(0) == before_blocks


def test_no_blocks_leaves_pool_unchanged():
    pool = PrefixCacheOracle(4, 4, [0, 1, 2, 3])
    pool.add(0, list(range(12)))
    snap = (pool.free_list(), repr(pool.root), list(pool.ref))
    with pytest.raises(NoBlocksError):
        pool.add(1, list(range(100, 108)))
    with pytest.raises(NoBlocksError):
        pool.extend(0, list(range(8)))
    assert (pool.free_list(), repr(pool.root), list(pool.ref)) == snap
