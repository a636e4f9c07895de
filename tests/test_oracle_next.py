"""Pins of the oracle's prefix-cache lifecycle additions (least-recently-used
eviction, KV memory accounting) and of the adapter/length batch former.

Expected values come from hand-derived fixtures (tests/golden/), closed forms
and definitions independent of the oracle's code (a sort for the batch order,
direct block counting for the accounting)."""
import json
import os

import numpy as np
import pytest

from oracle.apc import NoBlocksError, OracleError, PrefixCacheOracle
from oracle.batching import bucket_of, form_batches

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def eviction_tokens(name):
    return {"A": list(range(12)), "B": list(range(100, 120)),
            "C": list(range(8)) + [50, 51]}[name]


def run_eviction_golden(make_pool, apply_op, stats, blocks_of, free_list):
    """Replay tests/golden/apc_eviction_example.json on a pool implementation."""
    with open(os.path.join(GOLDEN, "apc_eviction_example.json")) as f:
        g = json.load(f)
    pool = make_pool(g["num_blocks"], g["block_size"], g["free_order"])
    for st in g["steps"]:
        res = apply_op(pool, st)
        if "error" in st:
            assert res == ("error", st["error"]), st
        elif "result" in st:
            assert res == st["result"], (st, res)
        if "blocks" in st:
            assert blocks_of(pool, st["seq"]) == st["blocks"], st
        if "free" in st:
            assert free_list(pool) == st["free"], st
        for k, v in st.get("stats", {}).items():
            assert stats(pool)[k] == v, (st, k)


def _oracle_op(pool, st):
    try:
        if st["op"] == "add":
            return pool.add(st["seq"], eviction_tokens(st["tokens"]))
        if st["op"] == "free":
            return pool.free_seq(st["seq"])
        if st["op"] == "kv_waste":
            return pool.kv_waste(st["max_seq_len"])
    except OracleError as e:
        return ("error", e.code)
    raise ValueError(st["op"])


def _oracle_pool(nb, bs, order):
    p = PrefixCacheOracle(nb, bs, order)
    p.evict = True
    return p


def test_eviction_worked_example():
    run_eviction_golden(_oracle_pool, _oracle_op, lambda p: p.stats(),
                        lambda p, s: list(p.seqs[s]["blocks"]), lambda p: p.free_list())


def _random_ops(pool, r, bs, steps=150):
    """Random admissions (sharing prefixes), extensions and releases."""
    prefixes = [r.integers(0, 3, size=int(r.integers(bs, 5 * bs))).tolist() for _ in range(3)]
    live, nid, log = [], 0, []
    for _ in range(steps):
        op = r.integers(0, 4)
        try:
            if op <= 1 or not live:
                toks = prefixes[int(r.integers(0, 3))] + r.integers(0, 3, size=int(r.integers(1, 3 * bs))).tolist()
                before = pool.evictions if hasattr(pool, "evictions") else None
                free_before = len(pool.free_list())
                n = pool.add(nid, toks)
                log.append(("add", nid, n, free_before, before))
                live.append(nid)
                nid += 1
            elif op == 2:
                sid = live[int(r.integers(0, len(live)))]
                pool.extend(sid, r.integers(0, 3, size=int(r.integers(0, 2 * bs))).tolist())
                log.append(("extend", sid))
            else:
                sid = live.pop(int(r.integers(0, len(live))))
                pool.free_seq(sid)
                log.append(("free", sid))
        except NoBlocksError:
            log.append(("no_blocks",))
    return log


@pytest.mark.parametrize("seed", range(6))
def test_eviction_is_invisible_when_the_free_list_suffices(seed):
    """With a pool large enough that nothing is ever evicted, enabling eviction
    changes nothing (same tables, hits, free list)."""
    bs = 4
    a = PrefixCacheOracle(2000, bs, list(range(2000)))
    b = PrefixCacheOracle(2000, bs, list(range(2000)))
    b.evict = True
    la = _random_ops(a, np.random.default_rng(seed), bs)
    lb = _random_ops(b, np.random.default_rng(seed), bs)
    assert [x[:3] for x in la] == [x[:3] for x in lb]
    assert a.free_list() == b.free_list() and b.evictions == 0
    assert {k: v["blocks"] for k, v in a.seqs.items()} == {k: v["blocks"] for k, v in b.seqs.items()}


@pytest.mark.parametrize("seed", range(6))
def test_eviction_only_after_the_free_list_is_used_up(seed):
    """An admission evicts only when the free list could not serve it, and it
    then uses the whole free list first."""
    bs = 4
    r = np.random.default_rng(100 + seed)
    p = PrefixCacheOracle(24, bs, r.permutation(24).tolist())
    p.evict = True
    evicted_any = False
    for step in range(200):
        toks = r.integers(0, 3, size=int(r.integers(2, 6 * bs))).tolist()
        free_before, ev_before = len(p.free_list()), p.evictions
        try:
            p.add(step, toks)
        except NoBlocksError:
            continue
        if p.evictions > ev_before:
            evicted_any = True
            assert p.free_list() == [] and free_before < len(p.seqs[step]["blocks"])
        if r.random() < 0.6:
            p.free_seq(int(r.choice(list(p.seqs))))
    assert evicted_any


def test_eviction_keeps_trie_paths_and_refcounts_consistent():
    """After random operations with eviction, every trie node's block is
    registered exactly once, idle stamps are exactly the registered blocks no
    live sequence holds, and reference counts equal the holders."""
    bs = 4
    r = np.random.default_rng(7)
    p = PrefixCacheOracle(30, bs, list(range(30)))
    p.evict = True
    _random_ops(p, r, bs, steps=300)
    seen = []

    def walk(level):
        for key, (blk, ch) in level.items():
            seen.append(blk)
            walk(ch)
    walk(p.root)
    assert sorted(seen) == sorted(p.registered) and len(set(seen)) == len(seen)
    holders = [0] * p.num_blocks
    for st in p.seqs.values():
        for b in st["blocks"]:
            holders[b] += 1
    assert holders == p.ref
    assert set(p.stamp) == {b for b in p.registered if holders[b] == 0}
    assert not set(p.free_list()) & (set(p.registered) | {b for b in range(30) if holders[b]})


def test_kv_waste_closed_forms():
    """k sequences sharing a P-token prefix plus s private tokens each, block
    size bs: paged slots k * ceil((P + s) / bs) * bs, physical slots
    (P / bs + k * ceil(s / bs)) * bs for P a multiple of bs, contiguous
    k * max_len."""
    bs, P, s, k, max_len = 16, 64, 21, 5, 200
    p = PrefixCacheOracle(200, bs, list(range(200)))
    prefix = list(range(P))
    for i in range(k):
        p.add(i, prefix + [1000 + 100 * i + j for j in range(s)])
    w = p.kv_waste(max_len)
    L = P + s
    assert w["tokens"] == k * L
    assert w["paged_slots"] == k * (-(-L // bs)) * bs
    assert w["physical_slots"] == (P // bs + k * (-(-s // bs))) * bs
    assert w["contiguous_slots"] == k * max_len
    assert w["contiguous_waste"] == pytest.approx(1 - L / max_len)
    assert w["paged_waste"] == pytest.approx(1 - L / ((-(-L // bs)) * bs))
    # per-sequence paged waste stays below block_size / length
    assert w["paged_waste"] < bs / L
    with pytest.raises(OracleError):
        p.kv_waste(L - 1)


def test_batch_former_worked_example():
    with open(os.path.join(GOLDEN, "batch_former_example.json")) as f:
        g = json.load(f)
    order, position, batches = form_batches(g["adapter_ids"], g["prompt_lens"], g["bucket_bounds"])
    assert [[a, k, idx] for a, k, idx in batches] == g["batches"]
    assert order == g["order"] and position == g["position"]


@pytest.mark.parametrize("seed", range(20))
def test_batch_former_equals_a_stable_sort(seed):
    """The execution order is the original indices sorted by (rank of the
    adapter's first appearance, length bucket, index); batches are the runs of
    equal (adapter, bucket); position inverts order."""
    r = np.random.default_rng(seed)
    n = int(r.integers(0, 60))
    ad = r.integers(0, int(r.integers(1, 8)), size=n).tolist()
    ln = r.integers(0, 5000, size=n).tolist()
    bounds = sorted(set(r.integers(1, 5000, size=int(r.integers(0, 4))).tolist()))
    order, position, batches = form_batches(ad, ln, bounds)
    first = {}
    for i, a in enumerate(ad):
        first.setdefault(a, i)
    nb = [sum(1 for b in bounds if x >= b) for x in ln]   # bucket by counting bounds passed
    expect = sorted(range(n), key=lambda i: (first[ad[i]], nb[i], i))
    assert order == expect
    assert [position[i] for i in order] == list(range(n))
    runs = []
    for i in expect:
        key = (ad[i], nb[i])
        if runs and runs[-1][0] == key:
            runs[-1][1].append(i)
        else:
            runs.append((key, [i]))
    assert [((a, k), idx) for a, k, idx in batches] == runs
    assert all(bucket_of(ln[i], bounds) == nb[i] for i in range(n))


def test_batch_former_rejects_bad_bounds():
    with pytest.raises(ValueError):
        form_batches([0], [1], [10, 10])
    with pytest.raises(ValueError):
        form_batches([0], [-1], [])
