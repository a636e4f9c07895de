"""GPU parity: libpa (HIP, through the C ABI) against the float64 oracle.

Reduced sizes run the whole launch element by element (several 128-row tiles,
split key ranges, ragged tails); full sizes run the exact launch the benchmark
times and compare sampled rows.  Tables, slot mappings and prefix hits are
compared bit for bit, the appended cache bit for bit, outputs within
|o - r| <= atol + rtol |r| (bf16 1e-2 / 2e-2, float32 1e-5 / 1e-5).
"""
import numpy as np
import pytest
import torch

from paper_2605_11232_amd import synth
from tests.parity import key_slot_pos, run_parity, sample_rows, say

pytestmark = pytest.mark.gpu


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def test_tiny_f32_prefill_and_decode_steps():
    _gpu()
    errs, _, _ = run_parity(synth.workload("tiny"))
    say("tiny normalized errors", errs)
    assert len(errs) == 9


def test_tiny_f32_head_dim_128():
    """The float32 kernel at head_dim 128 (the tiny recipe with D = 128):
    prefill then eight decode steps, within 1e-5."""
    _gpu()
    errs, dev, _ = run_parity(synth.workload("tiny", head_dim=128), label="tiny-f32-d128")
    say("tiny d128 normalized errors", errs)
    assert len(errs) == 9 and all(i.head_dim == 128 for i in dev.infos)


def test_verify_multi_chunk_shared_prefix_every_row():
    """Verification at the full 16384-token shared prefix and 4096-token
    private suffix, 4 requests, n_q 5, G 8: the shared prefix runs as three
    key chunks of cascade tiles (a full and a partial 128-row tile each), the
    40-row private parts (4101 keys) as one tile item each; every row
    compared."""
    _gpu()
    wl = synth.workload("verify", requests=4, steps=2)
    errs, dev, _ = run_parity(wl, steps=[1], label="verify-4req-full-length")
    say("verify multi-chunk normalized errors", errs)
    info = dev.infos[0]
    # 3 chunks x 2 tiles of gathered rows (160 rows) x 8 kv-heads
    assert info.n_shared_items == 3 * 2 * 8, info.n_shared_items
    assert info.n_tile_items == 4 * 1 * 8, info.n_tile_items


def test_prefill_long_sequences_every_row():
    """Suffix prefill of 2 requests at full length (2048 cached prefix +
    U[256,1024] suffix: more than 1024 keys, so the tile loop's window of
    block ids advances past 64 blocks), every row compared."""
    _gpu()
    wl = synth.workload("prefill", requests=2, steps=2)
    errs, dev, _ = run_parity(wl, steps=[1], label="prefill-2req-full-length")
    say("prefill long normalized errors", errs)
    assert min(wl.notes["suffix"]) + wl.notes["prefix"] > 64 * 16


def test_mixed_full_length_every_row():
    """The mixed launch at full lengths with 40 requests (5 prefill chunks of
    512 tokens over 1k-8k prefixes, 35 decode tokens, cascade groups on
    shared prefixes, the 8k prefix in two key chunks), every row compared."""
    _gpu()
    wl = synth.workload("mixed", requests=40, steps=2)
    errs, dev, _ = run_parity(wl, steps=[1], label="mixed-40req-full-length")
    say("mixed full-length normalized errors", errs)
    assert dev.infos[0].n_shared_items > 0


def test_tiny_in_bf16():
    _gpu()
    run_parity(synth.workload("tiny", dtype="bf16"), label="tiny-bf16")


def test_eviction_and_cold_miss_recompute():
    """Least-recently-used eviction shortens a cached prefix; the next request
    on it recomputes the evicted prefix tokens with the prefill kernel.  Hits,
    tables, appended cache and outputs match the oracle."""
    _gpu()
    wl = synth.workload("evict")
    errs, _, _ = run_parity(wl, label="evict")
    say("evict normalized errors", errs)
    assert len(errs) == 2


@pytest.mark.parametrize("name,scale", [("prefill", 0.125), ("decode", 0.0625),
                                        ("mixed", 0.0625), ("verify", 0.125)])
def test_reduced(name, scale):
    _gpu()
    errs, _, _ = run_parity(synth.workload(name, scale=scale, steps=3), steps=[1],
                            label=f"{name}@{scale}")
    say(name, "normalized errors", errs)


@pytest.mark.parametrize("name,scale", [("tiny", None), ("prefill", 0.125), ("decode", 0.0625),
                                        ("mixed", 0.0625), ("verify", 0.125)])
def test_staged_path(name, scale):
    """The benchmark's path: one library call per step for pool operations,
    metadata and plan into pinned staging buffers used alternately, one
    upload, the reused split workspace, batched release; four consecutive
    steps so each staging buffer is reused."""
    _gpu()
    if scale is None:  # the tiny float32 workload: its own nine launches
        wl, steps = synth.workload(name), None
    else:
        wl, steps = synth.workload(name, scale=scale, steps=5), [1, 2, 3]
    errs, _, _ = run_parity(wl, steps=steps, staged=True, label=f"staged {name}")
    say(name, "staged normalized errors", errs)
    assert len(errs) == len(wl.launches) + len(steps or [])


def test_staged_path_copy_engine_upload():
    """The staged path with a copy-engine copy instead of the upload kernel,
    reduced decode over consecutive steps."""
    _gpu()
    errs, _, _ = run_parity(synth.workload("decode", scale=0.0625, steps=5), steps=[1, 2, 3],
                            staged=True, stage_kernel=False, label="staged decode copy")
    say("staged copy-engine normalized errors", errs)


@pytest.mark.parametrize("staged", [False, True])
@pytest.mark.parametrize("name", ["prefill", "decode", "mixed", "verify"])
def test_full_size_sampled(name, staged):
    """The benchmark's exact launch (full size) on sampled rows, through the
    plain path and through the staged path bench.py times."""
    _gpu()
    wl = synth.workload(name, steps=2)
    rows = sample_rows(wl.launches[0], 48, wl.cfg.num_q_heads, seed=7)
    errs, _, _ = run_parity(wl, n_launches=1, rows=rows, staged=staged,
                            label=f"{name}-full" + (" staged" if staged else ""))
    say(name, "full-size normalized error", errs)


def test_stage_upload():
    """The upload kernel copies pinned host memory to device memory exactly,
    twice in a row (the second time fewer bytes of rewritten data: the new
    values arrive, nothing past the range changes, nothing stale is read), and
    refuses sources that are not pinned host memory before launching."""
    _gpu()
    from paper_2605_11232_amd import binding as B
    n = 1_000_003
    r = np.random.default_rng(3)
    host = torch.empty(n, dtype=torch.int32, pin_memory=True)
    dev = torch.zeros(n, dtype=torch.int32, device="cuda")
    first = r.integers(-2**31, 2**31 - 1, size=n, dtype=np.int64).astype(np.int32)
    host.numpy()[:] = first
    B.stage_upload(dev, host, 4 * n)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(dev.cpu().numpy(), first)
    m = 12_345
    second = r.integers(-2**31, 2**31 - 1, size=n, dtype=np.int64).astype(np.int32)
    host.numpy()[:] = second
    B.stage_upload(dev, host, 4 * m)
    torch.cuda.synchronize()
    got = dev.cpu().numpy()
    np.testing.assert_array_equal(got[:m], second[:m])
    np.testing.assert_array_equal(got[m:], first[m:])
    pageable = torch.ones(16, dtype=torch.int32)
    with pytest.raises(B.PaError):
        B.stage_upload(dev, pageable, 64)
    with pytest.raises(B.PaError):
        B.stage_upload(dev, dev, 64)
    torch.cuda.synchronize()


def test_stream_events():
    """Fence-free events: a timed interval around an upload is positive and
    ordered on the stream; a staging buffer released by a caller's event
    waits on that event, not its own."""
    _gpu()
    from paper_2605_11232_amd import binding as B
    from paper_2605_11232_amd.runtime import Staging
    n = 1 << 22
    host = torch.arange(n, dtype=torch.int32).pin_memory()
    dev = torch.zeros(n, dtype=torch.int32, device="cuda")
    a, b = B.StreamEvent(timing=True), B.StreamEvent(timing=True)
    a.record()
    B.stage_upload(dev, host, 4 * n)
    b.record()
    b.synchronize()
    ms = a.elapsed_time(b)
    assert 0.0 < ms < 1000.0, ms
    # the upload before b is complete once b is
    assert int(dev[n - 1].item()) == n - 1
    st = Staging("cuda", 2, 4, 8, 64)
    assert st.guard is st.ready
    g = B.StreamEvent()
    st.guard, st.used = g, True
    g.record()
    st.wait()
    torch.cuda.synchronize()


def test_bitwise_invariants():
    """Outputs are identical bit for bit when physical placement changes and
    when the shared prefix is duplicated instead of shared, and from run to run
    (reduction order follows logical key order only)."""
    _gpu()
    base = synth.workload("prefill", scale=0.125)
    wl_b = synth.workload("prefill", scale=0.125)
    wl_b.free_order = np.random.default_rng(3).permutation(wl_b.num_blocks).astype(np.int32)
    from paper_2605_11232_amd.runtime import DeviceReplay

    def outputs(wl):
        d = DeviceReplay(wl).setup()
        p = d.run(wl.launches[0])
        torch.cuda.synchronize()
        return p.out.view(torch.int16).cpu().numpy(), p.lse.cpu().numpy(), p.meta["block_table"]

    oa, la, bta = outputs(base)
    oa2, la2, _ = outputs(base)
    ob, lb, btb = outputs(wl_b)
    assert not np.array_equal(bta, btb)
    np.testing.assert_array_equal(oa, oa2)
    np.testing.assert_array_equal(oa, ob)
    np.testing.assert_array_equal(la, lb)
    # duplicated prefix: no pre-population, each request carries its own copy
    wl_c = synth.workload("prefill", scale=0.125)
    pref_ops = [op for op in wl_c.setup]
    add_op = pref_ops[0]
    k, v = pref_ops[1].k.get(), pref_ops[1].v.get()
    wl_c.setup = []
    launch = wl_c.launches[0]
    # every request now stores its own copy of the prefix
    wl_c.num_blocks = base.num_blocks + len(launch.q_lens) * (len(add_op.tokens) // 16 + 1)
    wl_c.free_order = np.arange(wl_c.num_blocks, dtype=np.int32)
    P = len(add_op.tokens)
    new_pre = []
    for i, op in enumerate(launch.pre):
        toks = op.tokens.copy()
        toks[:P] += 1 + i  # distinct token ids -> no sharing
        new_pre.append(synth.Op("add", op.seq_id, toks))
    qv = launch.q.get()
    kn, vn = launch.k_new.get(), launch.v_new.get()
    # each request now computes its prefix too: prepend prefix K/V, and
    # queries for the prefix positions (discarded), to every request
    R = len(launch.q_lens)
    cu = np.concatenate([[0], np.cumsum(launch.q_lens)])
    Hq, D = qv.shape[1], qv.shape[2]
    qs, ks, vs, ql = [], [], [], []
    for r in range(R):
        qs += [np.zeros((P, Hq, D), np.float32), qv[cu[r]:cu[r + 1]]]
        ks += [k, kn[cu[r]:cu[r + 1]]]
        vs += [v, vn[cu[r]:cu[r + 1]]]
        ql.append(P + launch.q_lens[r])

    class Fixed:
        def __init__(self, a):
            self.a = a

        def get(self):
            return self.a

    wl_c.launches = [synth.Launch(new_pre, launch.seq_ids, ql, Fixed(np.concatenate(qs)),
                                  Fixed(np.concatenate(ks)), Fixed(np.concatenate(vs)))]
    oc, lc, _ = outputs(wl_c)
    keep = np.concatenate([np.arange(cu[r] + (r + 1) * P, cu[r + 1] + (r + 1) * P) for r in range(R)])
    np.testing.assert_array_equal(oa, oc[keep])
    np.testing.assert_array_equal(la, lc[keep])


def test_needle_through_block_table():
    """Q = alpha e1, one key per kv-head = beta e1 at a chosen logical position,
    all other keys 0: o = (e^s v* + sum of the other visible v) / (e^s + a).
    A mis-mapped block moves the result by O(1)."""
    _gpu()
    from paper_2605_11232_amd import binding as B
    from paper_2605_11232_amd.runtime import DeviceReplay
    import math
    wl = synth.workload("verify", scale=0.125)
    cfg = wl.cfg
    d = DeviceReplay(wl).setup()
    launch = wl.step(0)
    p = d.prepare(launch)
    Hq, Hkv, D = cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim
    G = Hq // Hkv
    alpha, beta = 4.0, 8.0
    sigma = alpha * beta / math.sqrt(D)
    # zero every key of the launch's sequences, keep values
    bt = p.meta["block_table"]
    L = p.meta["seq_lens"]
    r = np.random.default_rng(0)
    needles = {}
    P = wl.notes["prefix"]
    for i in range(len(L)):
        blocks = torch.from_numpy(bt[i][:(L[i] + 15) // 16].astype(np.int64)).to(d.device)
        d.k_cache[blocks] = 0
    for i in range(len(L)):
        for g in range(Hkv):
            # private positions only: prefix blocks are shared by every request
            t = int(r.integers(P, L[i] - 5))
            needles[(i, g)] = t
            # dim 0 of key t: group 0, slot position of offset t % 16
            d.k_cache[int(bt[i][t // 16]), g, 0, int(key_slot_pos(t % 16)), 0] = beta
    p.k_new.zero_()
    q = torch.zeros_like(p.q)
    q[:, :, 0] = alpha
    p.q = q
    d.append(p)
    d.attend(p)
    torch.cuda.synchronize()
    out = p.out.float().cpu().numpy()
    # values: gather logical V on the host from the device cache
    vc = d.v_cache.float().cpu().numpy()
    cu = p.meta["cu_seqlens_q"]
    for i in range(len(L)):
        for j in range(cu[i + 1] - cu[i]):
            a = L[i] - (cu[i + 1] - cu[i]) + j
            tpos = np.arange(a + 1)
            V = vc[bt[i][tpos // 16], :, :, tpos % 16]  # [a+1, Hkv, D]
            for h in range(Hq):
                g = h // G
                ts = needles[(i, g)]
                want = (math.exp(sigma) * V[ts, g] + V[:, g].sum(0) - V[ts, g]) / (math.exp(sigma) + a)
                got = out[cu[i] + j, h]
                assert np.all(np.abs(got - want) <= 1e-2 + 2e-2 * np.abs(want)), (i, j, h)


class _Scaled:
    """A launch's queries multiplied by a factor, rounded back to bf16 (both
    the oracle and the library read these exact values)."""

    def __init__(self, values, factor):
        self.values, self.factor = values, factor

    def get(self):
        return synth.round_to_dtype(self.values.get() * np.float32(self.factor), "bf16")


@pytest.mark.parametrize("factor", [24.0, 1e-3])
@pytest.mark.parametrize("name,scale", [("prefill", 0.0625), ("decode", 0.0625),
                                        ("verify", 0.125), ("mixed", 0.0625)])
def test_extreme_score_scales(name, scale, factor):
    """Queries scaled by 24 (scores of standard deviation ~24 nats: nearly
    one-hot rows, the running maximum moves many times, most probabilities
    underflow) or by 1e-3 (nearly uniform rows) on every path: tile items,
    row items, shared-prefix items and their merge, against the oracle."""
    _gpu()
    wl = synth.workload(name, scale=scale, steps=2)
    launch = wl.launches[0]
    wl.launches = [synth.Launch(launch.pre, launch.seq_ids, launch.q_lens,
                                _Scaled(launch.q, factor), launch.k_new, launch.v_new, launch.post)]
    errs, dev, _ = run_parity(wl, n_launches=1, label=f"{name}@{scale} q x {factor}")
    say(f"{name} q x {factor} normalized errors", errs)


def test_edge_cases():
    """Empty launch, zero-query sequences mixed in, a one-token sequence,
    head_dim 64 in bf16, G = 1, verify with 16 to 128 rows per sequence (narrow
    and wide row items, tile items).  Each launch runs once more with timing
    events on its kernels: the same output bit for bit, and the events
    recorded also when nothing is launched."""
    _gpu()
    from oracle.run import OracleReplay
    from paper_2605_11232_amd import binding as B
    from paper_2605_11232_amd.runtime import DeviceReplay
    from tests.parity import TOL, close
    cfg = synth.AttnConfig("edge", "bf16", 4, 4, 64, 16, 77)
    Val = synth.Values
    r = np.random.default_rng(1)

    def mk(q_lens, lens, seed, cfg=cfg):
        """Sequences of length lens[i] whose last q_lens[i] tokens are queried;
        the earlier positions get their K/V written in setup."""
        setup, pre = [], []
        for i, (q, L) in enumerate(zip(q_lens, lens)):
            toks = r.integers(0, 50, size=L).astype(np.int32)
            if L - q >= 1:
                setup.append(synth.Op("add", i, toks[:L - q]))
                setup.append(synth.Op("write_kv", i,
                                      k=Val((seed, 15, i), (L - q, cfg.num_kv_heads, cfg.head_dim), "bf16"),
                                      v=Val((seed, 16, i), (L - q, cfg.num_kv_heads, cfg.head_dim), "bf16")))
                pre.append(synth.Op("extend", i, toks[L - q:]))
            else:
                pre.append(synth.Op("add", i, toks))
        T = sum(q_lens)
        return setup, synth.Launch(pre, list(range(len(lens))), q_lens,
                                   Val((seed, 4), (T, cfg.num_q_heads, cfg.head_dim), "bf16"),
                                   Val((seed, 5), (T, cfg.num_kv_heads, cfg.head_dim), "bf16"),
                                   Val((seed, 6), (T, cfg.num_kv_heads, cfg.head_dim), "bf16"))

    cases = [([0, 0], [5, 9]), ([1], [1]), ([0, 7, 0, 300, 1], [4, 7, 33, 300, 1000])]
    for ci, (ql, lens) in enumerate(cases):
        say("[edge] case", ci, ql, lens)
        setup, launch = mk(ql, lens, 50 + ci)
        wl = synth.Workload(cfg, 256, np.random.default_rng(ci).permutation(256).astype(np.int32),
                            setup, [launch], None, 80)
        o = OracleReplay(wl).setup()
        dv = DeviceReplay(wl, kind="prefill").setup()
        ro = o.launch(wl.launches[0])
        p = dv.run(wl.launches[0])
        torch.cuda.synchronize()
        if sum(ql):
            close(p.out.float().cpu().numpy(), ro["out"], *TOL["bf16"], f"edge{ci}")
        first = p.out.clone()
        ev = (B.StreamEvent(timing=True), B.StreamEvent(timing=True))
        dv.attend(p, events=ev)
        ev[1].synchronize()
        ms = ev[0].elapsed_time(ev[1])
        assert (ms > 0.0) if sum(ql) else (ms >= 0.0), ms
        assert torch.equal(p.out, first)
    # verify with n_q = 8: G = 2 gives 16 rows per sequence (one 16-row row
    # item per key range); G = 3 gives 24 rows (a row item of two 16-column
    # tiles); G = 8 gives 64 rows (tile items, two of the four wavefronts
    # idle; 4400 keys are two split ranges merged by log-sum-exp); G = 16
    # gives 128 rows (one tile item)
    for G, want_tiles, want_wide, lens in ((2, False, False, [40, 517]), (3, False, True, [40, 517]),
                                           (8, True, False, [40, 517]), (8, True, False, [40, 4400]),
                                           (16, True, False, [40, 517])):
        cfg8 = synth.AttnConfig(f"edge-g{G}", "bf16", 2 * G, 2, 128, 16, 78)
        setup, launch = mk([8, 8], lens, 9, cfg=cfg8)
        nb = sum(-(-L // 16) for L in lens) + 8
        wl = synth.Workload(cfg8, nb, np.arange(nb, dtype=np.int32), setup, [launch], None,
                            -(-max(lens) // 16))
        o = OracleReplay(wl).setup()
        dv = DeviceReplay(wl, kind="verify").setup()
        ro = o.launch(wl.launches[0])
        p = dv.run(wl.launches[0])
        torch.cuda.synchronize()
        assert (p.info.n_tile_items > 0) == want_tiles
        assert (p.info.n_row_items > 0) == (not want_tiles)
        assert bool(p.info.variant & 2) == want_wide
        if max(lens) > 4160:   # the private keys run as split tile items
            assert p.info.n_tile_items > 2 * cfg8.num_kv_heads and p.info.n_groups > 0
        close(p.out.float().cpu().numpy(), ro["out"], *TOL["bf16"], f"verify-G{G}-{max(lens)}")


@pytest.mark.parametrize("name", ["prefill", "mixed"])
def test_tail_stealing_plan_reuse(name):
    """A launch whose plan has tail lists (wildcard workgroups taking full
    tiles through counters in the plan) matches the oracle, and runs eight
    more times on the same device plan with the same output bit for bit
    (which workgroup takes which tail item changes from run to run; each
    item's result does not): the last wildcard workgroup leaves the
    counters zero, as uploaded."""
    _gpu()
    from paper_2605_11232_amd.runtime import DeviceReplay
    from tests.parity import TOL, close
    from oracle.run import OracleReplay
    wl = synth.workload(name, scale=0.125, steps=2)
    o = OracleReplay(wl).setup()
    dv = DeviceReplay(wl).setup()
    launch = wl.step(0) if wl.step else wl.launches[0]
    say(f"[tail] {name}@0.125 launch 0")
    p = dv.run(launch)
    torch.cuda.synchronize()
    h = p.plan[:32].cpu().numpy()
    n_tail, n_wild, ctr_off = int(h[25]), int(h[26]), int(h[27])
    assert n_tail > 0 and n_wild == n_tail
    ro = o.launch(launch, rows=None)
    close(p.out.float().cpu().numpy(), ro["out"], *TOL["bf16"], f"tail-stealing {name}")
    first = p.out.clone()
    for k in range(8):
        dv.attend(p)
        torch.cuda.synchronize()
        assert torch.equal(p.out, first), f"repeat {k}"
        ctr = p.plan[ctr_off:ctr_off + 9 * 32].cpu().numpy()
        assert not ctr.any(), ctr[ctr != 0]


@pytest.mark.parametrize("name,scale", [("decode", 0.125), ("verify", 0.25), ("mixed", 0.125)])
def test_shared_prefix_cascade_matches_per_sequence(name, scale):
    """With shared-prefix groups (prefix attention once for all sequences,
    merged by log-sum-exp) and without them: both match the oracle on every
    row, and agree with each other within the bf16 tolerance."""
    _gpu()
    from tests.parity import TOL, close
    outs = []
    for cascade in (True, False):
        wl = synth.workload(name, scale=scale, steps=2)
        _, dev, _ = run_parity(wl, n_launches=1, cascade=cascade,
                               label=f"{name}@{scale} cascade={cascade}")
        if cascade:
            assert dev.infos[0].n_shared_items > 0
        else:
            assert dev.infos[0].n_shared_items == 0
        outs.append(dev.outs[0])
    close(outs[0][0], outs[1][0], *TOL["bf16"], f"{name} cascade vs per-sequence")
    close(outs[0][1], outs[1][1], 2e-3, 1e-4, f"{name} lse cascade vs per-sequence")


def _random_workload(seed):
    """A random small launch: random heads, group size and head_dim; one or
    two cached prefixes (whole blocks) shared by some sequences; a launch
    kind of suffix prefill, decode, verification or a mix of prefill and
    decode sequences."""
    r = np.random.default_rng(9000 + seed)
    hkv = int(r.choice([1, 2, 4, 8]))
    G = int(r.choice([1, 2, 4, 7, 8, 16]))
    D = int(r.choice([64, 128]))
    cfg = synth.AttnConfig(f"fuzz{seed}", "bf16", hkv * G, hkv, D, 16, 5000 + seed)
    Val = synth.Values
    bs = 16
    prefixes = [r.integers(0, 1 << 17, size=16 * int(r.integers(1, 40))).astype(np.int32)
                for _ in range(int(r.integers(1, 3)))]
    setup = []
    for pi, pt in enumerate(prefixes):
        sid = synth.PREFIX_SEQ_BASE + pi
        setup += [synth.Op("add", sid, pt),
                  synth.Op("write_kv", sid, k=Val((cfg.seed, 15, 100 + pi), (len(pt), hkv, D), "bf16"),
                           v=Val((cfg.seed, 16, 100 + pi), (len(pt), hkv, D), "bf16")),
                  synth.Op("free", sid)]
    kind = ["prefill", "decode", "verify", "mixed"][seed % 4]
    n = int(r.integers(1, 9))
    n_q = int(r.integers(2, 9))
    pre, q_lens = [], []
    for i in range(n):
        pt = prefixes[int(r.integers(0, len(prefixes)))] if r.random() < 0.8 else np.zeros(0, np.int32)
        body = r.integers(0, 1 << 17, size=int(r.integers(1, 400))).astype(np.int32)
        toks = np.concatenate([pt, body])
        sk = kind if kind != "mixed" else ("prefill" if r.random() < 0.5 else "decode")
        if sk == "prefill":
            pre.append(synth.Op("add", i, toks))
            q_lens.append(len(body))
        else:
            q = 1 if sk == "decode" else n_q
            # context in the cache (prefix hits, body written), then q new tokens
            setup.append(synth.Op("add", i, toks))
            setup.append(synth.Op("write_kv", i, k=Val((cfg.seed, 15, i), (len(body), hkv, D), "bf16"),
                                  v=Val((cfg.seed, 16, i), (len(body), hkv, D), "bf16")))
            pre.append(synth.Op("extend", i, r.integers(0, 1 << 17, size=q).astype(np.int32)))
            q_lens.append(q)
    T = sum(q_lens)
    launch = synth.Launch(pre, list(range(n)), q_lens, Val((cfg.seed, 4), (T, hkv * G, D), "bf16"),
                          Val((cfg.seed, 5), (T, hkv, D), "bf16"), Val((cfg.seed, 6), (T, hkv, D), "bf16"))
    nb = 4096
    max_len = max(len(p) for p in prefixes) + 400 + 16
    return synth.Workload(cfg, nb, np.random.default_rng(seed).permutation(nb).astype(np.int32),
                          setup, [launch], None, -(-max_len // bs))


@pytest.mark.parametrize("seed", range(16))
def test_random_launches(seed):
    """Random shapes and launch kinds through the whole path (tables, cache,
    outputs, LSE against the oracle)."""
    _gpu()
    wl = _random_workload(seed)
    c = wl.cfg
    say(f"[fuzz] seed {seed}: Hq {c.num_q_heads} Hkv {c.num_kv_heads} D {c.head_dim} "
        f"q_lens {wl.launches[0].q_lens}")
    run_parity(wl, label=f"fuzz{seed}")
