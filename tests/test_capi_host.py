"""CPU tests of the C-ABI boundary (no GPU): the library loads, exports every
symbol include/pa.h declares, and its host block manager produces the same
block tables, slot mappings and prefix-hit counts as the oracle, bit for bit;
error paths leave the pool unchanged.  Device entry points are only called
with arguments that fail host validation (nothing is launched)."""
import ctypes
import itertools
import os
import re

import numpy as np
import pytest

from paper_2605_11232_amd import binding as B
from paper_2605_11232_amd import synth
from oracle.apc import OracleError, PrefixCacheOracle
from tests.test_oracle_apc import _random_batch, run_golden

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_symbols():
    txt = open(os.path.join(ROOT, "include", "pa.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)  # drop comments
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(pa_[a-z0-9_]+)\s*\(",
                                 txt, flags=re.M)))


def test_exports_every_declared_symbol():
    lib = B.lib()
    declared = _header_symbols()
    assert set(declared) == set(B.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name
    assert lib.pa_abi_version() == 2


def _lib_apply(pool, st, toks):
    try:
        if st["op"] == "add":
            return pool.add(st["seq"], toks)
        if st["op"] == "extend":
            return pool.extend(st["seq"], toks)
        if st["op"] == "free":
            return pool.free(st["seq"])
        if st["op"] == "truncate":
            return pool.truncate(st["seq"], st["n"])
        if st["op"] == "metadata":
            return pool.metadata(st["seqs"], st["q_lens"], st["max_blocks"])
    except B.PaError as e:
        return ("error", e.code)
    raise ValueError(st["op"])


def test_worked_example_library():
    run_golden(B.Pool, _lib_apply)


class _Both:
    """Apply every operation to the oracle and the library and compare."""

    def __init__(self, nb, bs, order, evict=False):
        self.o = PrefixCacheOracle(nb, bs, order)
        self.l = B.Pool(nb, bs, order, evict=evict)
        self.o.evict = evict

    def do(self, name, *args):
        res = []
        for impl, fn in ((self.o, {"free": "free_seq"}.get(name, name)), (self.l, name)):
            try:
                res.append(("ok", getattr(impl, fn)(*args)))
            except OracleError as e:
                res.append(("error", e.code))
            except B.PaError as e:
                res.append(("error", e.code))
        assert res[0] == res[1], (name, args, res)
        assert self.o.free_list() == self.l.free_list()
        assert self.o.stats() == self.l.stats()
        return res[0]

    def meta(self, ids, q_lens, mb):
        a = self.o.metadata(ids, q_lens, mb)
        b = self.l.metadata(ids, q_lens, mb)
        for k in a:
            np.testing.assert_array_equal(a[k], b[k], err_msg=k)
        return a


@pytest.mark.parametrize("seed", range(25))
def test_random_operation_sequences_bit_exact(seed):
    _random_operations(seed, evict=False)


@pytest.mark.parametrize("seed", range(25))
def test_random_operation_sequences_with_eviction_bit_exact(seed):
    """Small pools force least-recently-used evictions of idle cached blocks;
    tables, free lists, hit counts and counters stay identical."""
    both = _random_operations(seed, evict=True)
    assert both.o.evictions == both.l.stats()["evictions"]


def test_eviction_happens_in_random_sequences():
    assert sum(_random_operations(s, evict=True).o.evictions for s in range(6)) > 0


def _random_operations(seed, evict):
    r = np.random.default_rng(1000 + seed)
    bs = int(r.choice([2, 4, 16]))
    nb = int(r.integers(8, 40 if evict else 120))
    both = _Both(nb, bs, r.permutation(nb).tolist(), evict=evict)
    prefixes, reqs = _random_batch(seed, bs=bs, vocab=int(r.choice([2, 3, 50])))
    live = {}
    next_id = 0
    for step in range(120):
        op = r.integers(0, 6)
        if op <= 1 or not live:
            p, toks = reqs[int(r.integers(0, len(reqs)))]
            if r.random() < 0.3:
                toks = toks[:int(r.integers(1, len(toks) + 1))]
            res = both.do("add", next_id, toks)
            if res[0] == "ok":
                live[next_id] = len(toks)
            next_id += 1
        elif op == 2:
            sid = int(r.choice(list(live)))
            n = int(r.integers(0, 2 * bs + 2))
            res = both.do("extend", sid, r.integers(0, 4, size=n).tolist())
        elif op == 3:
            sid = int(r.choice(list(live)))
            L = both.o.seq_len(sid)
            both.do("truncate", sid, int(r.integers(0, L + 2)))
        elif op == 4:
            sid = int(r.choice(list(live)))
            both.do("free", sid)
            del live[sid]
        else:
            ids = list(live)
            r.shuffle(ids)
            ids = ids[:int(r.integers(1, len(ids) + 1))]
            q = [int(r.integers(0, both.o.seq_len(i) + 1)) for i in ids]
            both.meta(ids, q, 64 if bs >= 4 else 200)
        # unknown sequences and duplicate ids behave alike
        if step % 17 == 0:
            both.do("free", 10 ** 9)
            if live:
                sid = next(iter(live))
                both.do("add", sid, [1, 2, 3])
        if step % 13 == 0 and live:
            mx = max(both.o.seq_len(i) for i in live)
            for m in (mx, mx + 7, mx - 1):
                both.do("kv_waste", m)
    return both


@pytest.mark.parametrize("name", ["tiny", "prefill", "decode", "mixed", "verify", "evict"])
def test_workload_tables_bit_exact(name):
    """Setup + first launch of every workload at full size: tables, slots and
    prefix hits agree exactly (values are not drawn; tables only)."""
    wl = synth.workload(name, steps=2)
    o = PrefixCacheOracle(wl.num_blocks, wl.cfg.block_size, wl.free_order)
    o.evict = wl.evict
    l = B.Pool(wl.num_blocks, wl.cfg.block_size, wl.free_order, evict=wl.evict)

    def apply(op):
        if op.kind == "write_kv":
            return None
        fn = {"add": ("add", "add"), "extend": ("extend", "extend"), "free": ("free_seq", "free"),
              "truncate": ("truncate", "truncate")}[op.kind]
        args = (op.seq_id, op.tokens) if op.tokens is not None else (op.seq_id, op.n)
        if op.kind == "free":
            args = (op.seq_id,)
        a = getattr(o, fn[0])(*args)
        b = getattr(l, fn[1])(*args)
        assert a == b, op.kind
        return a

    for op in wl.setup:
        apply(op)
    extra = [wl.step(1)] if wl.step and name != "tiny" else []
    for li, launch in enumerate(wl.launches[:2] + extra):
        hits = [apply(op) for op in launch.pre]
        if name == "evict":   # hand-derived from the eviction rules
            assert hits == wl.notes["expected_hits"][li]
        mo = o.metadata(launch.seq_ids, launch.q_lens, wl.max_blocks_per_seq)
        ml = l.metadata(launch.seq_ids, launch.q_lens, wl.max_blocks_per_seq)
        for k in mo:
            np.testing.assert_array_equal(mo[k], ml[k], err_msg=k)
        # the configured prefix is reused in full by every admitted request
        if name in ("prefill", "tiny") and launch.pre[0].kind == "add":
            assert set(hits) == {wl.notes["prefix"]}
        for op in launch.post:
            apply(op)
        assert o.free_list() == l.free_list()
        assert o.stats() == l.stats()
    if name == "evict":
        assert o.evictions == 5


# plan layout (plan_format.h): header words, record sizes
H_N_SHARED, H_N_TILE, H_N_ROW, H_N_GROUPS, H_GRID = 2, 3, 4, 5, 6
H_SHARED_OFF, H_TILE_OFF, H_ROW_OFF, H_GROUP_OFF, H_MEMBER_OFF, H_PARTIAL_ROWS = 12, 13, 14, 15, 16, 17
H_DISPATCH_OFF, H_HEAD_PARTIAL, H_HKV = 18, 19, 8
H_N_SHARED_TMPL, H_N_TILE_TMPL, H_N_ROW_TMPL, H_N_GROUP_TMPL = 20, 21, 22, 23
H_TAIL_OFF, H_N_TAIL, H_N_WILD, H_CTR_OFF = 24, 25, 26, 27
HEADER_WORDS = 32
XCD_QUEUES, COUNTER_WORDS = 8, 32
HEAD_SHIFT = 24           # dispatch word: (kv-head << 24) | template index
WILDCARD = (1 << HEAD_SHIFT) - 1   # template index of a wildcard workgroup
STREAM_FLAG = 1           # item flags word: no other item reads the item's keys
WAVES = 4                 # wavefronts per workgroup: row items come WAVES to a workgroup
TILE_ROWS = 32 * WAVES    # rows of a tile or shared item (32 per wavefront)
ROW_ITEM_ROWS = 32        # rows of a row item (two 16-column MFMA tiles)
VARIANT_WIDE_ROWS = 2     # plan info variant bit: some row item has more than 16 rows
VARIANT_TAIL = 4          # plan info variant bit: the plan has tail lists (wildcard workgroups)


def tail_lists(plan):
    """The tail list of each XCD queue (dispatch words), from the tail table."""
    h = plan[:HEADER_WORDS]
    if not h[H_N_TAIL]:
        return [[] for _ in range(XCD_QUEUES)]
    tab = plan[h[H_TAIL_OFF]:h[H_TAIL_OFF] + 2 * XCD_QUEUES]
    return [plan[tab[q]:tab[q] + tab[XCD_QUEUES + q]].tolist() for q in range(XCD_QUEUES)]


def parse_plan(plan):
    """The plan's work per workgroup, expanded from the dispatch list and the
    kv-head-0 templates: shared items as (member table, kvh, row0, nrows,
    kv0, kv1, rows per member, block sequence, partial offset), tile and row
    items and merge groups with their kv-head and partial rows stamped."""
    h = plan[:HEADER_WORDS]
    assert h[H_DISPATCH_OFF] == HEADER_WORDS   # the dispatch list follows the header
    hp = int(h[H_HEAD_PARTIAL])
    tmpl = lambda off, n: plan[off:off + 8 * n].reshape(-1, 8).tolist()
    ts, tt = tmpl(h[H_SHARED_OFF], h[H_N_SHARED_TMPL]), tmpl(h[H_TILE_OFF], h[H_N_TILE_TMPL])
    tr, tg = tmpl(h[H_ROW_OFF], h[H_N_ROW_TMPL]), tmpl(h[H_GROUP_OFF], h[H_N_GROUP_TMPL])
    disp = plan[h[H_DISPATCH_OFF]:h[H_DISPATCH_OFF] + h[H_GRID]].tolist()
    assert all(w >= 0 for w in disp)
    # wildcard workgroups take the tail lists' tile items at run time: one
    # wildcard per tail item, the table and lists right after the dispatch
    # list, then the counters, zero
    tail = sum(tail_lists(plan), [])
    if h[H_N_TAIL]:
        assert h[H_TAIL_OFF] == h[H_DISPATCH_OFF] + h[H_GRID]
        assert h[H_CTR_OFF] == h[H_TAIL_OFF] + 2 * XCD_QUEUES + h[H_N_TAIL]
        assert not plan[h[H_CTR_OFF]:h[H_CTR_OFF] + (XCD_QUEUES + 1) * COUNTER_WORDS].any()
    assert disp.count(WILDCARD) == h[H_N_WILD] == len(tail) == h[H_N_TAIL]
    split = [(w >> HEAD_SHIFT, w & ((1 << HEAD_SHIFT) - 1)) for w in disp if w != WILDCARD]
    split += [(w >> HEAD_SHIFT, w & ((1 << HEAD_SHIFT) - 1)) for w in tail]
    # template indices run over the shared, tile and row templates in order
    n_st, n_tt = h[H_N_SHARED_TMPL], h[H_N_TILE_TMPL]
    s_split = [(g, i) for g, i in split if i < n_st]
    t_split = [(g, i - n_st) for g, i in split if n_st <= i < n_st + n_tt]
    r_split = [(g, i - n_st - n_tt) for g, i in split if i >= n_st + n_tt]
    assert len(s_split) == h[H_N_SHARED] and len(t_split) == h[H_N_TILE]
    assert all(i % WAVES == 0 and i < h[H_N_ROW_TMPL] for _, i in r_split)

    def stamp(t, g):
        t = list(t)
        assert t[1] == 0            # templates are kv-head 0's
        if t[0] >= 0:
            t[1] = g
            if t[6] >= 0:
                t[6] += g * hp
        return t
    shared = [tuple(ts[i][:1]) + (g,) + tuple(ts[i][2:]) + (g * hp,) for g, i in s_split]
    tiles = [stamp(tt[i], g) for g, i in t_split]
    rows = [stamp(tr[i + k], g) for g, i in r_split for k in range(WAVES)]
    groups = [[t[0], g, t[2], t[3], t[4], t[5] + g * hp, t[6], t[7]]
              for g in range(h[H_HKV]) for t in tg]
    assert len(groups) == h[H_N_GROUPS] and len(rows) == h[H_N_ROW]
    return h, shared, tiles, rows, groups


def check_plan(plan, info, L, cu, G, hkv, D=128):
    """Every (sequence, kv-head, row) is produced exactly once: by one item
    covering all its visible keys, or by parts whose key ranges tile [0, L)
    and whose partial rows are exactly those of its merge group."""
    h, shared, tiles, rows, groups = parse_plan(plan)
    assert h[0] == 0x31304150 and h[H_GRID] == info.grid
    assert info.grid == h[H_N_SHARED] + h[H_N_TILE] + h[H_N_ROW] // WAVES
    n = len(L)
    q = np.diff(cu)
    cover = {}      # (seq, kvh, rho) -> list of (kv0, kv1, partial row or -1)
    writes = {}     # partial row -> count
    def add(key, kv0, kv1, pr):
        cover.setdefault(key, []).append((kv0, kv1, pr))
        if pr >= 0:
            writes[pr] = writes.get(pr, 0) + 1
    assert h[H_N_ROW] % WAVES == 0
    assert bool(info.variant & VARIANT_WIDE_ROWS) == any(t[3] > 16 for t in rows if t[0] >= 0)
    assert bool(info.variant & VARIANT_TAIL) == (h[H_N_TAIL] > 0)
    assert all(0 < t[3] <= TILE_ROWS for t in tiles) and all(0 < t[3] <= TILE_ROWS for t in shared)
    assert all(t[3] <= ROW_ITEM_ROWS for t in rows if t[0] >= 0)
    # a row item's block ids are one 64-lane load: at most 64 blocks of 16 keys
    assert all(t[5] - t[4] <= 64 * 16 for t in rows if t[0] >= 0)
    for seq, kvh, row0, nrows, kv0, kv1, part, _ in tiles + rows:
        if seq < 0:
            continue
        assert kv0 % 16 == 0 and 0 <= kv0 < kv1 <= L[seq]
        for lr in range(nrows):
            add((seq, kvh, row0 + lr), kv0, kv1, -1 if part < 0 else part + lr)
    for moff, kvh, row0, nrows, kv0, kv1, rpm, bseq, poff in shared:
        assert kv0 % 64 == 0 and kv1 % 64 == 0
        for lr in range(nrows):
            rg = row0 + lr
            m, rl = divmod(rg, rpm)
            seq, base = plan[moff + 2 * m], plan[moff + 2 * m + 1] + poff
            assert kv1 <= L[seq] - q[seq]          # every shared key is visible
            add((seq, kvh, rl), kv0, kv1, base + rl)
    assert len(cover) == sum(int(q[s]) * G * hkv for s in range(n))
    expected = {}
    for seq, kvh, row0, nrows, nsplit, part, stride, _ in groups:
        for lr in range(nrows):
            expected[(seq, kvh, row0 + lr)] = {part + sp * stride + lr for sp in range(nsplit)}
    for key, ranges in cover.items():
        seq, kvh, rho = key
        ranges.sort()
        need = int(L[seq] - q[seq] + rho // G + 1)
        if len(ranges) == 1 and ranges[0][2] == -1:
            assert key not in expected and ranges[0][0] == 0 and ranges[0][1] >= need
        else:
            assert {pr for _, _, pr in ranges} == expected[key]
            assert ranges[0][0] == 0 and ranges[-1][1] == L[seq]
            assert all(ranges[i][1] == ranges[i + 1][0] for i in range(len(ranges) - 1))
    assert set(writes) == set(range(h[H_PARTIAL_ROWS])) and set(writes.values()) <= {1}
    assert int(info.workspace_bytes) == int(h[H_PARTIAL_ROWS]) * (D + 1) * 4
    assert int(info.partial_rows) == int(h[H_PARTIAL_ROWS])
    # the launch shape the attention calls check against
    assert (info.n_seqs, info.total_q, info.num_kv_heads, info.head_dim) == (n, int(cu[-1]), hkv, D)
    assert info.num_q_heads == hkv * G
    # the plan-free workspace bound covers this plan
    bound = B.workspace_size(int(cu[-1]), hkv * G, D, int(max(L)) if n else 0)
    assert bound >= int(info.workspace_bytes)


def test_plan_covers_every_row_once():
    r = np.random.default_rng(5)
    for trial in range(40):
        n = int(r.integers(1, 40))
        hkv = int(r.choice([1, 2, 4, 8]))
        G = int(r.choice([1, 4, 7, 8]))
        L = r.integers(1, 5000, size=n)
        q = np.minimum(L, r.choice([1, 2, 5, 8, 33, 300, 1000], size=n))
        if trial % 3 == 0:
            q[:] = 1
        cu = np.concatenate([[0], np.cumsum(q)])
        kind = B.KIND_DECODE if trial % 3 == 0 else B.KIND_PREFILL
        # block tables: a few prefix groups share leading blocks
        mb = int((L.max() + 15) // 16)
        bt = np.full((n, mb), -1, np.int32)
        nxt = 0
        prefixes = [r.integers(0, 200) for _ in range(3)]
        shared_blocks = {}
        for s_ in range(n):
            nb = int((L[s_] + 15) // 16)
            grp = int(r.integers(0, 4))
            if grp < 3:
                pb = min(nb - 1, int(prefixes[grp]))
                base = shared_blocks.setdefault(grp, list(range(10 ** 6 + 1000 * grp, 10 ** 6 + 1000 * grp + 300)))
                bt[s_, :pb] = base[:pb]
                bt[s_, pb:nb] = np.arange(nxt, nxt + nb - pb)
                nxt += nb - pb
            else:
                bt[s_, :nb] = np.arange(nxt, nxt + nb)
                nxt += nb
        for table in (None, bt):
            plan, info = B.plan(kind, 1, L, cu, hkv * G, hkv, 128, 16, B.PA_BF16, 256,
                                block_table=table)
            check_plan(plan, info, L, cu, G, hkv)
            if table is None:
                assert info.n_shared_items == 0


def _workload_plan(name, scale):
    wl = synth.workload(name, scale=scale)
    o = PrefixCacheOracle(wl.num_blocks, wl.cfg.block_size, wl.free_order)
    for op in wl.setup:
        if op.kind == "add":
            o.add(op.seq_id, op.tokens)
        elif op.kind == "free":
            o.free_seq(op.seq_id)
    launch = wl.step(0) if wl.step else wl.launches[0]
    for op in launch.pre:
        (o.add if op.kind == "add" else o.extend)(op.seq_id, op.tokens)
    md = o.metadata(launch.seq_ids, launch.q_lens, wl.max_blocks_per_seq)
    cfg = wl.cfg
    kind = {"decode": B.KIND_DECODE, "verify": B.KIND_VERIFY}.get(name, B.KIND_PREFILL)
    plan, info = B.plan(kind, int(max(launch.q_lens)), md["seq_lens"], md["cu_seqlens_q"],
                        cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, 16, B.PA_BF16, 256,
                        block_table=md["block_table"])
    return plan, info, md, cfg


@pytest.mark.parametrize("name", ["prefill", "decode", "mixed", "verify"])
def test_dispatch_keeps_kv_heads_on_their_xcds(name):
    """Workgroup b runs on XCD b % 8; a kv-head's work goes to the XCDs
    g (mod Hkv) only, segment after segment of the dispatch list."""
    plan, info, md, cfg = _workload_plan(name, 0.25)
    hkv = cfg.num_kv_heads
    disp = plan[HEADER_WORDS:HEADER_WORDS + info.grid]
    fixed = disp != WILDCARD   # wildcards take tail items on whichever XCD runs them
    heads = disp[fixed] >> HEAD_SHIFT
    xcd = np.arange(info.grid)[fixed] % 8
    assert np.array_equal(xcd % hkv, heads % 8 if hkv >= 8 else heads)
    check_plan(plan, info, md["seq_lens"], md["cu_seqlens_q"], cfg.group, hkv)


def test_plan_finds_shared_prefix_of_workloads():
    """The decode and verify workloads share their whole cached prefix."""
    for name, prefix in (("decode", 2048), ("verify", 16384)):
        wl = synth.workload(name, scale=0.25)
        o = PrefixCacheOracle(wl.num_blocks, wl.cfg.block_size, wl.free_order)
        for op in wl.setup:
            if op.kind == "add":
                o.add(op.seq_id, op.tokens)
            elif op.kind == "free":
                o.free_seq(op.seq_id)
        launch = wl.step(0)
        for op in launch.pre:
            o.extend(op.seq_id, op.tokens)
        md = o.metadata(launch.seq_ids, launch.q_lens, wl.max_blocks_per_seq)
        cfg = wl.cfg
        kind = B.KIND_DECODE if name == "decode" else B.KIND_VERIFY
        plan, info = B.plan(kind, launch.q_lens[0], md["seq_lens"], md["cu_seqlens_q"],
                            cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, 16, B.PA_BF16,
                            block_table=md["block_table"])
        h, shared, tiles, *_ = parse_plan(plan)
        assert info.n_shared_items > 0
        P = wl.notes["prefix"]
        assert max(s[5] for s in shared) == P // 64 * 64
        # verify's 40-row private parts are tile items marked as streamed
        # (no other item reads their keys)
        assert (len(tiles) > 0) == (name == "verify")
        assert all(t[7] == STREAM_FLAG for t in tiles)
        check_plan(plan, info, md["seq_lens"], md["cu_seqlens_q"], cfg.group, cfg.num_kv_heads)


def test_decode_tail_gets_half_length_items():
    """The sequences with the fewest private keys (about a tenth of the row
    work) are split with half the target length, so the shortest items run
    last; the rest keep the full target (576 keys at full size)."""
    plan, info, md, cfg = _workload_plan("decode", 1.0)
    _, _, _, rows, _ = parse_plan(plan)
    items = [t for t in rows if t[0] >= 0 and t[1] == 0]
    per_seq = {}
    for t in items:
        per_seq.setdefault(t[0], []).append(t[5] - t[4])
    longest = max(max(v) for v in per_seq.values())
    assert longest == 576
    private = {r: sum(v) for r, v in per_seq.items()}
    halved = [r for r, v in per_seq.items() if max(v) <= 288 and len(v) > 1]
    assert halved, "some sequence is split into several items with the half target"
    # halved sequences are among the shortest: every sequence that kept
    # full-target items is at least as long as every halved one
    full = [r for r, v in per_seq.items() if max(v) > 288]
    assert max(private[r] for r in halved) <= min(private[r] for r in full)
    tail_work = sum(private[r] for r in halved)
    assert tail_work <= 0.1 * sum(private.values())


def test_prefill_tiles_are_not_streamed():
    """Tiles of a long sequence share its keys: none carries the stream flag."""
    plan, info, md, cfg = _workload_plan("prefill", 0.25)
    _, _, tiles, _, _ = parse_plan(plan)
    assert tiles and not any(t[7] & STREAM_FLAG for t in tiles)


def test_device_calls_reject_bad_arguments_without_launching():
    lib = B.lib()
    info = B.PlanInfo()
    info.kind = B.KIND_DECODE
    # the launch shape of the call below
    info.n_seqs, info.total_q, info.num_q_heads, info.num_kv_heads = 1, 1, 8, 2
    info.head_dim, info.dtype = 128, B.PA_BF16
    args = [None, None, None, 16, None, 4, None, None, 1, 1, 8, 2, 128, 16, 0.1, B.PA_BF16, None,
            ctypes.byref(info), None, 0, None, None, None]
    # plan kind mismatch
    assert lib.pa_attn_prefill(*args) == B.PA_ERR_ARG
    assert b"kind" in lib.pa_last_error()
    # unsupported head_dim / block_size / dtype
    for idx, val, code in ((12, 96, B.PA_ERR_UNSUPPORTED), (13, 32, B.PA_ERR_UNSUPPORTED),
                           (15, 7, B.PA_ERR_UNSUPPORTED), (10, 7, B.PA_ERR_ARG),
                           (14, 0.0, B.PA_ERR_ARG)):
        a = list(args)
        a[idx] = val
        assert lib.pa_attn_decode(*a) == code, idx
    # NULL device pointers with work to do
    assert lib.pa_attn_decode(*args) == B.PA_ERR_ARG
    assert b"NULL" in lib.pa_last_error()
    # a plan built for another launch shape is refused before anything else
    for field, val in (("n_seqs", 2), ("total_q", 3), ("num_q_heads", 16), ("num_kv_heads", 1),
                       ("head_dim", 64), ("dtype", B.PA_F32)):
        bad = B.PlanInfo()
        ctypes.memmove(ctypes.byref(bad), ctypes.byref(info), ctypes.sizeof(info))
        setattr(bad, field, val)
        a = list(args)
        a[17] = ctypes.byref(bad)
        assert lib.pa_attn_decode(*a) == B.PA_ERR_ARG, field
        assert b"plan was built for" in lib.pa_last_error(), field
    assert lib.pa_kv_append(None, None, None, 3, None, None, 16, 2, 128, 16, B.PA_BF16, None) == B.PA_ERR_ARG
    assert lib.pa_kv_append(None, None, None, 0, None, None, 16, 2, 100, 16, B.PA_BF16, None) == B.PA_ERR_UNSUPPORTED
    # staged upload: size and alignment are checked before any runtime call
    assert lib.pa_stage_upload(None, None, 0, None) == B.PA_OK
    assert lib.pa_stage_upload(None, None, 8, None) == B.PA_ERR_ARG
    assert lib.pa_stage_upload(4096, 8192, 6, None) == B.PA_ERR_ARG
    assert lib.pa_stage_upload(4098, 8192, 8, None) == B.PA_ERR_ARG
    assert lib.pa_stage_upload(4096, 8192, -4, None) == B.PA_ERR_ARG


def test_stream_event_binds_the_runtime():
    """The fence-free stream events resolve in the HIP runtime libpa links;
    without a device, creating one raises instead of returning a null event."""
    h = B._hip_runtime()
    for f in ("hipEventCreateWithFlags", "hipEventRecord", "hipEventSynchronize",
              "hipEventElapsedTime", "hipEventDestroy"):
        assert getattr(h, f) is not None
    import torch
    if torch.cuda.is_available():
        pytest.skip("a device is present; the GPU tests record these events")
    with pytest.raises(B.PaError, match="hipEventCreateWithFlags"):
        B.StreamEvent(timing=True)


def test_plan_rejects_inconsistent_lengths():
    with pytest.raises(B.PaError) as e:
        B.plan(B.KIND_DECODE, 1, [10, 10], [0, 1, 3], 8, 2, 128, 16, B.PA_BF16)
    assert e.value.code == "arg"
    with pytest.raises(B.PaError):
        B.plan(B.KIND_VERIFY, 5, [10], [0, 4], 8, 2, 128, 16, B.PA_BF16)
    with pytest.raises(B.PaError):
        B.plan(B.KIND_PREFILL, 0, [3], [0, 4], 8, 2, 128, 16, B.PA_BF16)
    with pytest.raises(B.PaError) as e:
        B.plan(B.KIND_PREFILL, 0, [3], [0, 2], 8, 3, 128, 16, B.PA_BF16)
    _, info = B.plan(B.KIND_PREFILL, 0, [], [0], 8, 2, 128, 16, B.PA_BF16)
    assert info.grid == 0 and info.workspace_bytes == 0


def test_batched_pool_calls_match_single_calls():
    """pa_seqs_* apply the single-sequence operations in order; a failing
    operation stops the batch and leaves the pool as before that operation."""
    r = np.random.default_rng(9)
    bs, nb = 4, 60
    order = r.permutation(nb).tolist()
    o = PrefixCacheOracle(nb, bs, order)
    lib_pool = B.Pool(nb, bs, order)
    prefix = list(range(100, 112))
    reqs = [prefix + r.integers(0, 9, size=int(r.integers(1, 9))).tolist() for _ in range(6)]
    hits_o = [o.add(i, t) for i, t in enumerate(reqs)]
    off = np.concatenate([[0], np.cumsum([len(t) for t in reqs])])
    hits_l = lib_pool.add_many(list(range(6)), off, np.concatenate(reqs))
    assert hits_o == hits_l.tolist()
    ext = [r.integers(0, 9, size=int(r.integers(0, 6))).tolist() for _ in range(6)]
    for i, t in enumerate(ext):
        o.extend(i, t)
    off = np.concatenate([[0], np.cumsum([len(t) for t in ext])])
    lib_pool.extend_many(list(range(6)), off, np.concatenate(ext) if sum(map(len, ext)) else [])
    new_lens = [len(reqs[i]) for i in range(6)]
    for i in range(6):
        o.truncate(i, new_lens[i])
    lib_pool.truncate_many(list(range(6)), new_lens)
    assert o.free_list() == lib_pool.free_list()
    md_o = o.metadata(list(range(6)), [1] * 6, 16)
    md_l = lib_pool.metadata(list(range(6)), [1] * 6, 16)
    for k in md_o:
        np.testing.assert_array_equal(md_o[k], md_l[k])
    # a batch whose third operation fails: two applied, pool otherwise intact
    n_done = ctypes.c_int32(-1)
    ids = np.array([0, 1, 999, 2], dtype=np.int64)
    rc = B.lib().pa_seqs_free(lib_pool._h, 4, ids.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                              ctypes.byref(n_done))
    assert rc == B.PA_ERR_UNKNOWN_SEQ and n_done.value == 2
    o.free_seq(0)
    o.free_seq(1)
    assert o.free_list() == lib_pool.free_list()
    assert lib_pool.seq_len(2) == o.seq_len(2)


@pytest.mark.parametrize("name", ["mixed", "verify"])
def test_pool_apply_matches_oracle_on_steps(name):
    """pa_pool_apply (one call per step phase) against the oracle applying the
    same operations one by one, over several steps of a workload."""
    from paper_2605_11232_amd.runtime import batch_ops
    wl = synth.workload(name, scale=0.25, steps=4)
    o = PrefixCacheOracle(wl.num_blocks, wl.cfg.block_size, wl.free_order)
    lp = B.Pool(wl.num_blocks, wl.cfg.block_size, wl.free_order)
    for op in wl.setup:
        if op.kind == "add":
            assert o.add(op.seq_id, op.tokens) == lp.add(op.seq_id, op.tokens)
        elif op.kind == "free":
            o.free_seq(op.seq_id)
            lp.free(op.seq_id)
    for st in range(3):
        launch = wl.step(st)
        hits = lp.apply_packed(batch_ops(launch.pre)).copy()
        want = [o.add(op.seq_id, op.tokens) if op.kind == "add" else
                (o.extend(op.seq_id, op.tokens) or 0) for op in launch.pre]
        assert hits.tolist() == want
        mo = o.metadata(launch.seq_ids, launch.q_lens, wl.max_blocks_per_seq)
        ml = lp.metadata(launch.seq_ids, launch.q_lens, wl.max_blocks_per_seq)
        for k in mo:
            np.testing.assert_array_equal(mo[k], ml[k])
        lp.apply_packed(batch_ops(launch.post))
        for op in launch.post:
            if op.kind == "free":
                o.free_seq(op.seq_id)
            else:
                o.truncate(op.seq_id, op.n)
        assert o.free_list() == lp.free_list()


# -- prefix-cache lifecycle and batch forming (library against the oracle) ----

def _lib_evict_op(pool, st):
    from tests.test_oracle_next import eviction_tokens
    try:
        if st["op"] == "add":
            return pool.add(st["seq"], eviction_tokens(st["tokens"]))
        if st["op"] == "free":
            return pool.free(st["seq"])
        if st["op"] == "kv_waste":
            return pool.kv_waste(st["max_seq_len"])
    except B.PaError as e:
        return ("error", e.code)
    raise ValueError(st["op"])


def test_eviction_worked_example_library():
    from tests.test_oracle_next import run_eviction_golden
    run_eviction_golden(lambda nb, bs, order: B.Pool(nb, bs, order, evict=True), _lib_evict_op,
                        lambda p: p.stats(), lambda p, s: p.blocks_of(s), lambda p: p.free_list())


def test_eviction_off_by_default_fails_cleanly():
    p = B.Pool(4, 4, [0, 1, 2, 3])
    p.add(0, list(range(12)))
    p.free(0)
    with pytest.raises(B.PaError) as e:
        p.add(1, list(range(100, 116)))
    assert e.value.code == "no_blocks" and p.free_list() == [3]
    p.set_eviction(True)
    assert p.add(1, list(range(100, 116))) == 0
    assert p.stats()["evictions"] == 3


def test_batch_former_library_matches_oracle():
    import json
    from oracle.batching import form_batches
    with open(os.path.join(os.path.dirname(__file__), "golden", "batch_former_example.json")) as f:
        g = json.load(f)
    order, position, batches = B.form_batches(g["adapter_ids"], g["prompt_lens"], g["bucket_bounds"])
    assert [[a, k, idx] for a, k, idx in batches] == g["batches"]
    assert order == g["order"] and position == g["position"]
    r = np.random.default_rng(3)
    for _ in range(200):
        n = int(r.integers(0, 80))
        ad = r.integers(-3, int(r.integers(1, 10)), size=n).tolist()
        ln = r.integers(0, 6000, size=n).tolist()
        bounds = sorted(set(r.integers(0, 6000, size=int(r.integers(0, 5))).tolist()))
        assert B.form_batches(ad, ln, bounds) == form_batches(ad, ln, bounds)


def test_batch_former_rejects_bad_arguments():
    for ad, ln, bb in (([0], [1], [10, 10]), ([0], [-1], []), ([0, 1], [1, 2], [5, 3])):
        with pytest.raises(B.PaError) as e:
            B.form_batches(ad, ln, bb)
        assert e.value.code == "arg"


@pytest.mark.parametrize("name", ["decode", "verify", "mixed"])
def test_prepare_launch_matches_separate_calls(name):
    """pa_prepare_launch (pool operations, metadata and plan in one call, into
    caller buffers) against pa_pool_apply + pa_build_metadata + pa_attn_plan
    on a second pool, over several steps: identical tables, plans, infos,
    reuse counts and free lists."""
    from paper_2605_11232_amd.runtime import batch_ops
    wl = synth.workload(name, scale=0.25, steps=4)
    cfg = wl.cfg
    pools = [B.Pool(wl.num_blocks, cfg.block_size, wl.free_order) for _ in range(2)]
    for lp in pools:
        for op in wl.setup:
            if op.kind == "add":
                lp.add(op.seq_id, op.tokens)
            elif op.kind == "free":
                lp.free(op.seq_id)
    mb = wl.max_blocks_per_seq
    for st in range(3):
        launch = wl.step(st)
        n, T = len(launch.seq_ids), int(sum(launch.q_lens))
        kind = {"decode": B.KIND_DECODE, "verify": B.KIND_VERIFY}.get(name, B.KIND_PREFILL)
        n_q = launch.q_lens[0] if name == "verify" else 1
        # fused, into caller buffers
        buf = B.LaunchBuffers(np.full((n, mb), 7, np.int32), np.zeros(n, np.int32),
                              np.zeros(n + 1, np.int32), np.zeros(T, np.int32),
                              np.zeros(1 << 20, np.int32))
        pre = batch_ops(launch.pre)
        info = pools[0].prepare_launch(pre, B.LaunchInputs(launch.seq_ids, launch.q_lens), buf,
                                       kind, n_q, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim,
                                       B.PA_BF16, 256, True)
        # separate calls
        hits = pools[1].apply_packed(batch_ops(launch.pre)).copy()
        md = pools[1].metadata(launch.seq_ids, launch.q_lens, mb)
        plan, info2 = B.plan(kind, n_q, md["seq_lens"], md["cu_seqlens_q"], cfg.num_q_heads,
                             cfg.num_kv_heads, cfg.head_dim, cfg.block_size, B.PA_BF16, 256,
                             block_table=md["block_table"])
        assert pre.n_cached[:pre.n].tolist() == hits.tolist()
        for k, v in buf.meta(n, T).items():
            np.testing.assert_array_equal(v, md[k], err_msg=k)
        np.testing.assert_array_equal(buf.plan[:info.plan_words], plan)
        for f, _ in B.PlanInfo._fields_:
            assert getattr(info, f) == getattr(info2, f), f
        for lp in pools:
            lp.apply_packed(batch_ops(launch.post))
        assert pools[0].free_list() == pools[1].free_list()
    # a plan buffer that is too small: argument error, pool operations applied
    launch = wl.step(3)
    n, T = len(launch.seq_ids), int(sum(launch.q_lens))
    small = B.LaunchBuffers(np.zeros((n, mb), np.int32), np.zeros(n, np.int32),
                            np.zeros(n + 1, np.int32), np.zeros(T, np.int32),
                            np.zeros(8, np.int32))
    before = pools[0].stats()["live_tokens"]
    with pytest.raises(B.PaError) as e:
        pools[0].prepare_launch(batch_ops(launch.pre), B.LaunchInputs(launch.seq_ids, launch.q_lens),
                                small, B.KIND_PREFILL if name == "mixed" else kind, n_q,
                                cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, B.PA_BF16)
    assert e.value.rc == B.PA_ERR_ARG and b"capacity" in B.lib().pa_last_error()
    added = sum(len(op.tokens) for op in launch.pre if op.tokens is not None)
    assert pools[0].stats()["live_tokens"] == before + added


def test_workspace_size_bounds_every_plan():
    """pa_attn_workspace_size / pa_attn_decode_workspace_size bound the
    workspace of random decode, verification and mixed plans (with and
    without shared-prefix groups), grow with every argument, and reject bad
    arguments."""
    r = np.random.default_rng(11)
    for trial in range(60):
        n = int(r.integers(1, 300))
        hkv = int(r.choice([1, 2, 4, 8]))
        G = int(r.choice([1, 2, 4, 8, 16]))
        D = int(r.choice([64, 128]))
        kind = [B.KIND_DECODE, B.KIND_VERIFY, B.KIND_PREFILL][trial % 3]
        n_q = int(r.integers(1, 9)) if kind == B.KIND_VERIFY else 1
        L = r.integers(n_q, 30000, size=n)
        if kind == B.KIND_PREFILL:
            q = np.where(r.random(n) < 0.5, 1, np.minimum(L, r.integers(1, 700, size=n)))
        else:
            q = np.full(n, n_q)
        cu = np.concatenate([[0], np.cumsum(q)]).astype(np.int32)
        mb = int((L.max() + 15) // 16)
        # every sequence shares its first P blocks (cascade groups), or none
        P = int(r.integers(0, int(L.min()) // 16 + 1)) if trial % 2 else 0
        bt = np.full((n, mb), -1, np.int32)
        nxt = 10 ** 6
        for s_ in range(n):
            nb = int((L[s_] + 15) // 16)
            bt[s_, :min(P, nb)] = np.arange(min(P, nb))
            bt[s_, min(P, nb):nb] = np.arange(nxt, nxt + nb - min(P, nb))
            nxt += nb
        _, info = B.plan(kind, n_q, L, cu, hkv * G, hkv, D, 16, B.PA_BF16, 256,
                         block_table=bt if P else None)
        bound = B.workspace_size(int(cu[-1]), hkv * G, D, int(L.max()))
        assert bound >= int(info.workspace_bytes), (trial, bound, int(info.workspace_bytes))
        if kind == B.KIND_DECODE:
            assert B.workspace_size(n, hkv * G, D, int(L.max()), decode=True) == bound
    # the decode workload's own plan fits the decode bound
    wl = synth.workload("decode", scale=0.25)
    assert B.workspace_size(256, 32, 128, 4000, decode=True) >= B.workspace_size(64, 32, 128, 4000)
    assert B.workspace_size(10, 8, 128, 256) == 0   # one part per sequence: nothing split
    assert B.workspace_size(10, 8, 128, 257) > 0
    lib = B.lib()
    n_out = ctypes.c_size_t(0)
    assert lib.pa_attn_workspace_size(-1, 8, 128, 10, ctypes.byref(n_out)) == B.PA_ERR_ARG
    assert lib.pa_attn_decode_workspace_size(1, 8, 96, 10, ctypes.byref(n_out)) == B.PA_ERR_UNSUPPORTED
    assert b"pa_attn_decode_workspace_size" in lib.pa_last_error()
    assert lib.pa_attn_workspace_size(1, 8, 128, 10, None) == B.PA_ERR_ARG


def test_noalloc_decode_rejects_before_launching():
    """pa_attn_decode_noalloc checks its arguments like pa_attn_decode and
    refuses a plan whose workspace exceeds its per-device array, all before
    any runtime call."""
    lib = B.lib()
    h = open(os.path.join(ROOT, "include", "pa.h")).read()
    assert re.search(r"#define PA_NOALLOC_WORKSPACE_BYTES \(\(size_t\)32 << 20\)", h)
    assert B.NOALLOC_WORKSPACE_BYTES == 32 << 20
    info = B.PlanInfo()
    info.kind = B.KIND_DECODE
    info.n_seqs, info.total_q, info.num_q_heads, info.num_kv_heads = 1, 1, 8, 2
    info.head_dim, info.dtype, info.variant, info.grid = 128, B.PA_BF16, 1, 1
    args = [1, 2, 3, 16, 4, 4, 5, 6, 1, 1, 8, 2, 128, 16, 0.1, B.PA_BF16, 7,
            ctypes.byref(info), 8, None, None]
    # one byte too many for the per-device array
    info.partial_rows = (B.NOALLOC_WORKSPACE_BYTES // (129 * 4)) + 1
    info.workspace_bytes = info.partial_rows * 129 * 4
    assert lib.pa_attn_decode_noalloc(*args) == B.PA_ERR_ARG
    assert b"pa_attn_decode_noalloc" in lib.pa_last_error()
    assert b"workspace" in lib.pa_last_error()
    # a plan of another kind, and a shape other than the plan's
    info.partial_rows, info.workspace_bytes = 0, 0
    info.kind = B.KIND_VERIFY
    assert lib.pa_attn_decode_noalloc(*args) == B.PA_ERR_ARG
    assert b"kind" in lib.pa_last_error()
    info.kind = B.KIND_DECODE
    info.total_q = 2
    assert lib.pa_attn_decode_noalloc(*args) == B.PA_ERR_ARG
    assert b"plan was built for" in lib.pa_last_error()


@pytest.mark.parametrize("name", ["prefill", "mixed", "decode", "verify"])
def test_tail_lists_hold_last_full_tiles(name):
    """Prefill and mixed: the last plain full tiles in dispatch order, about
    5 % of the tile work, move to the tail list of their XCD queue
    (workgroup b runs on XCD b % 8), still in dispatch order (a sequence's
    tiles together), and their slots hold wildcards, as many per queue as its
    list has items; decode and verify have no such tiles, so no tail."""
    plan, info, md, cfg = _workload_plan(name, 0.25)
    h = plan[:HEADER_WORDS]
    disp = plan[HEADER_WORDS:HEADER_WORDS + info.grid]
    lists = tail_lists(plan)
    n_st = int(h[H_N_SHARED_TMPL])
    tt = plan[h[H_TILE_OFF]:h[H_TILE_OFF] + 8 * h[H_N_TILE_TMPL]].reshape(-1, 8)
    if name in ("decode", "verify"):
        assert h[H_N_TAIL] == 0 and not (disp == WILDCARD).any()
        return
    assert h[H_N_TAIL] > 0
    wild = disp == WILDCARD
    total_tail = 0
    for q, lst in enumerate(lists):
        assert len(lst) == int(wild[q::XCD_QUEUES].sum())
        if not lst:
            continue
        t = tt[(np.array(lst) & WILDCARD) - n_st]
        assert (t[:, 3] > 96).all() and (t[:, 7] == 0).all()   # full tiles, not streamed
        cost = t[:, 5].astype(np.int64) * t[:, 3]
        seqs = [k for k, _ in itertools.groupby(t[:, 0].tolist())]
        assert len(seqs) == len(set(seqs))                        # a sequence's tiles together
        # a queue's items keep their kv-heads: the XCD's own heads
        heads = np.array(lst) >> HEAD_SHIFT
        fixed_heads = disp[q::XCD_QUEUES][~wild[q::XCD_QUEUES]] >> HEAD_SHIFT
        assert set(heads.tolist()) <= set(fixed_heads.tolist())
        total_tail += int(cost.sum())
    is_full = np.array([w != WILDCARD and n_st <= (w & WILDCARD) < n_st + len(tt)
                        and tt[(w & WILDCARD) - n_st][3] > 96 and tt[(w & WILDCARD) - n_st][7] == 0
                        for w in disp])
    fixed_cost = sum(int(tt[(w & WILDCARD) - n_st][5]) * int(tt[(w & WILDCARD) - n_st][3])
                     for w in disp[is_full])
    frac = total_tail / (total_tail + fixed_cost)
    assert 0.05 <= frac < 0.06
    # every wildcard sits after the last fixed full tile of the dispatch order
    assert np.flatnonzero(wild).min() > np.flatnonzero(is_full).max()
    check_plan(plan, info, md["seq_lens"], md["cu_seqlens_q"], cfg.group, cfg.num_kv_heads)


def test_set_launch_events_without_a_gpu():
    """pa_set_launch_events only stores the two handles for the calling
    thread's next attention call: it touches no device, accepts NULLs and
    reports success."""
    L = B.lib()
    assert L.pa_set_launch_events(None, None) == B.PA_OK
    try:
        assert L.pa_set_launch_events(ctypes.c_void_p(0x1000), ctypes.c_void_p(0x2000)) == B.PA_OK
    finally:
        # clear them again, so no later call on this thread carries these handles
        assert L.pa_set_launch_events(None, None) == B.PA_OK
