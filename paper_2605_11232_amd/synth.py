"""Seeded synthetic workloads for prefix-cached paged attention.

This module only draws inputs: token ids, lengths, physical block placement and
N(0,1) query/key/value values.  It contains none of the arithmetic of the
method (no table building, no slot computation, no attention); both the HIP
path and the CPU oracle consume what it produces.

Workload shapes follow the paper's prefix-dominated compliance prompts: a long
shared policy prefix followed by per-case evidence and a short structured
output (Introduction; Section 3, Table "phenotype"; Section 5.1, Table
"publiccoverage": average inputs 1.2k-2.8k tokens, outputs 64-96 tokens).
The public AML datasets the paper renders its prompts from are not used;
seeded synthetic values with the same token-count shapes stand in for them.

A workload is a script of host operations on a prefix cache:

* ``Op("add", seq, tokens)``       admit a sequence (prefix-hit lookup + allocation)
* ``Op("extend", seq, tokens)``    append tokens to a live sequence
* ``Op("write_kv", seq, k=, v=)``  store K/V for the last ``len(k)`` positions
* ``Op("free", seq)``              release a finished sequence
* ``Op("truncate", seq, n=)``      roll a sequence back to ``n`` tokens

plus ``Launch`` records: run ``pre`` ops, build metadata for ``seq_ids`` with
``q_lens`` query tokens each (the last ``q_lens[r]`` positions), append
``k_new``/``v_new`` for those positions, run attention for ``q``, then run
``post`` ops.

Seeds: configuration ``k`` (1-based, in the order of ``CONFIG_NAMES``) uses
seed ``1000 + k``; every array has its own stream
``np.random.default_rng([seed, tag, *index])`` with tags
lengths=1, prefix tokens=2, suffix tokens=3, Q=4, K=5, V=6, free list=7,
Zipf prefix choice=8, chunk/decode split=9, decode step j -> 100 + j.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Callable, List, Optional, Sequence

import numpy as np

TOKEN_VOCAB = 1 << 17

TAG_LEN, TAG_PREFIX_TOK, TAG_SUFFIX_TOK, TAG_Q, TAG_K, TAG_V = 1, 2, 3, 4, 5, 6
TAG_FREE, TAG_ZIPF, TAG_SPLIT, TAG_STEP = 7, 8, 9, 100

# Sequence ids at or above this value are the prefix pre-population sequences.
PREFIX_SEQ_BASE = 1 << 40


@dataclass(frozen=True)
class AttnConfig:
    name: str
    dtype: str            # "f32" or "bf16": storage type of q, k, v, out
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    seed: int
    description: str = ""

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads


CONFIGS = {
    "tiny": AttnConfig("tiny", "f32", 8, 2, 64, 16, 1001,
                       "4 requests, 128-token shared prefix, suffix U[32,64], "
                       "prefill then 8 decode steps"),
    "prefill": AttnConfig("prefill", "bf16", 32, 8, 128, 16, 1002,
                          "64 requests, 2048-token shared prefix, suffix prefill U[256,1024]"),
    "decode": AttnConfig("decode", "bf16", 32, 8, 128, 16, 1003,
                         "256 sequences, context 2048 + U[256,1024] + U[1,128], 1 query each"),
    "mixed": AttnConfig("mixed", "bf16", 28, 4, 128, 16, 1004,
                        "512 requests over 4 prefixes (1k/2k/4k/8k, Zipf 1.1): "
                        "64 x 512-token chunks + 448 decode tokens in one launch"),
    "verify": AttnConfig("verify", "bf16", 64, 8, 128, 16, 1005,
                         "32 requests, 16384 shared prefix + 4096 cached suffix, "
                         "5 query tokens (4 draft + 1)"),
    "evict": AttnConfig("evict", "bf16", 8, 2, 128, 16, 1006,
                        "two cached 64-token prefixes in a 12-block pool with eviction: "
                        "requests on one prefix evict the other's tail, which a later "
                        "request recomputes (cold miss)"),
}
CONFIG_NAMES = list(CONFIGS)


def rng(seed: int, tag: int, *index: int) -> np.random.Generator:
    return np.random.default_rng([seed, tag, *index])


def round_to_dtype(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float32 values to the storage dtype (RNE for bf16) and return float32."""
    if dtype == "f32":
        return x.astype(np.float32)
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(
        torch.bfloat16).to(torch.float32).numpy()


@dataclass
class Values:
    """A lazily drawn N(0,1) array, rounded to the workload dtype."""
    seed: tuple
    shape: tuple
    dtype: str

    def get(self) -> np.ndarray:
        x = np.random.default_rng(list(self.seed)).standard_normal(self.shape, dtype=np.float32)
        return round_to_dtype(x, self.dtype)


def tokens(seed: int, tag: int, idx: Sequence[int], n: int) -> np.ndarray:
    return rng(seed, tag, *idx).integers(0, TOKEN_VOCAB, size=n, dtype=np.int64).astype(np.int32)


@dataclass
class Op:
    kind: str
    seq_id: int
    tokens: Optional[np.ndarray] = None
    n: int = 0
    k: Optional[Values] = None
    v: Optional[Values] = None


@dataclass
class Launch:
    pre: List[Op]
    seq_ids: List[int]
    q_lens: List[int]
    q: Values          # [sum q_lens, Hq, D]
    k_new: Values      # [sum q_lens, Hkv, D]
    v_new: Values
    post: List[Op] = field(default_factory=list)

    @property
    def total_q(self) -> int:
        return int(sum(self.q_lens))


@dataclass
class Workload:
    cfg: AttnConfig
    num_blocks: int
    free_order: np.ndarray
    setup: List[Op]
    launches: List[Launch]
    # Builds the launch of repeated step ``s`` (fresh token ids where requests
    # are admitted); ``launches`` holds step 0 (and, for "tiny", its decode steps).
    step: Optional[Callable[[int], Launch]] = None
    max_blocks_per_seq: int = 0
    notes: dict = field(default_factory=dict)
    evict: bool = False   # the pool evicts idle cached blocks when it runs out


def _kv_values(cfg: AttnConfig, idx: tuple, n: int):
    shp = (n, cfg.num_kv_heads, cfg.head_dim)
    return (Values((cfg.seed, TAG_K) + idx, shp, cfg.dtype),
            Values((cfg.seed, TAG_V) + idx, shp, cfg.dtype))


def _q_values(cfg: AttnConfig, idx: tuple, n: int) -> Values:
    return Values((cfg.seed, TAG_Q) + idx, (n, cfg.num_q_heads, cfg.head_dim), cfg.dtype)


def _prefix_setup(cfg: AttnConfig, prefixes: List[np.ndarray]) -> List[Op]:
    """Pre-populate every distinct prefix: admit it, store its K/V, release it
    (its full blocks stay cached for later requests)."""
    ops: List[Op] = []
    for p, toks in enumerate(prefixes):
        sid = PREFIX_SEQ_BASE + p
        k, v = _kv_values(cfg, (1, p), len(toks))
        ops += [Op("add", sid, toks), Op("write_kv", sid, k=k, v=v), Op("free", sid)]
    return ops


def _cdiv(a: int, b: int) -> int:
    return -(-a // b)


def _pool(needed: int, seed: int, extra: int = 0):
    nb = needed + max(64, needed // 4) + extra
    return nb, rng(seed, TAG_FREE).permutation(nb).astype(np.int32)


def _concat(*parts: np.ndarray) -> np.ndarray:
    return np.concatenate([np.asarray(p, dtype=np.int32) for p in parts])


# --------------------------------------------------------------------------
# Individual workloads
# --------------------------------------------------------------------------

def _tiny(cfg: AttnConfig, scale: float = 1.0, steps: int = 1) -> Workload:
    s, bs = cfg.seed, cfg.block_size
    R, P, n_dec = 4, 128, 8
    S = rng(s, TAG_LEN).integers(32, 65, size=R)
    prefix = tokens(s, TAG_PREFIX_TOK, (0,), P)
    suffix = [tokens(s, TAG_SUFFIX_TOK, (r,), int(S[r])) for r in range(R)]
    setup = _prefix_setup(cfg, [prefix])
    launches = []
    pre = [Op("add", r, _concat(prefix, suffix[r])) for r in range(R)]
    k, v = _kv_values(cfg, (2, 0), int(S.sum()))
    launches.append(Launch(pre, list(range(R)), [int(x) for x in S],
                           _q_values(cfg, (0,), int(S.sum())), k, v))
    for j in range(1, n_dec + 1):
        pre = [Op("extend", r, tokens(s, TAG_STEP + j, (r,), 1)) for r in range(R)]
        k, v = _kv_values(cfg, (2, j), R)
        launches.append(Launch(pre, list(range(R)), [1] * R, _q_values(cfg, (j,), R), k, v))
    max_len = P + int(S.max()) + n_dec
    needed = P // bs + sum(_cdiv(P + int(S[r]) + n_dec, bs) - P // bs for r in range(R))
    nb = 64
    assert needed <= nb

    def step(st: int) -> Launch:
        # repeated prefill launches (benchmarking): fresh suffix token ids per
        # step, requests released afterwards
        first = launches[0]
        pre = [Op("add", r, _concat(prefix, tokens(s, TAG_SUFFIX_TOK, (r, st + 1), int(S[r]))))
               for r in range(R)]
        return Launch(pre, first.seq_ids, first.q_lens, first.q, first.k_new, first.v_new,
                      [Op("free", r) for r in range(R)])

    if steps > 1:
        nb = max(nb, P // bs + steps * sum(_cdiv(P + int(S[r]), bs) - P // bs for r in range(R))
                 + 64)
    free_order = rng(s, TAG_FREE).permutation(nb).astype(np.int32)
    return Workload(cfg, nb, free_order, setup, launches, step, _cdiv(max_len, bs),
                    {"prefix": P, "suffix": S.tolist(), "decode_steps": n_dec})


def _prefill(cfg: AttnConfig, scale: float = 1.0, steps: int = 1,
             requests: Optional[int] = None) -> Workload:
    """Suffix prefill of per-case evidence against one cached policy prefix."""
    s, bs = cfg.seed, cfg.block_size
    R = requests or max(1, int(round(64 * scale)))
    P = max(bs, int(round(2048 * scale / bs)) * bs) if scale < 1 else 2048
    lo, hi = (256, 1024) if scale >= 1 else (max(1, int(256 * scale)), max(2, int(1024 * scale)))
    S = rng(s, TAG_LEN).integers(lo, hi + 1, size=R)
    prefix = tokens(s, TAG_PREFIX_TOK, (0,), P)
    setup = _prefix_setup(cfg, [prefix])
    T = int(S.sum())
    qv = _q_values(cfg, (0,), T)
    kn, vn = _kv_values(cfg, (2, 0), T)

    def step(st: int) -> Launch:
        pre = [Op("add", r, _concat(prefix, tokens(s, TAG_SUFFIX_TOK, (r, st), int(S[r]))))
               for r in range(R)]
        post = [Op("free", r) for r in range(R)]
        return Launch(pre, list(range(R)), [int(x) for x in S], qv, kn, vn, post)

    per_step = sum(_cdiv(P + int(S[r]), bs) - P // bs for r in range(R))
    nb, free_order = _pool(P // bs + per_step * max(1, steps), s)
    return Workload(cfg, nb, free_order, setup, [step(0)], step, _cdiv(P + hi, bs),
                    {"prefix": P, "suffix": S.tolist()})


def _decode(cfg: AttnConfig, scale: float = 1.0, steps: int = 1,
            requests: Optional[int] = None) -> Workload:
    """One decode token per sequence over prefix + evidence + generated tokens."""
    s, bs = cfg.seed, cfg.block_size
    R = requests or max(1, int(round(256 * scale)))
    P = 2048 if scale >= 1 else max(bs, int(round(2048 * scale / bs)) * bs)
    lo, hi = (256, 1024) if scale >= 1 else (max(1, int(256 * scale)), max(2, int(1024 * scale)))
    S = rng(s, TAG_LEN, 0).integers(lo, hi + 1, size=R)
    g = rng(s, TAG_LEN, 1).integers(1, 129, size=R)
    prefix = tokens(s, TAG_PREFIX_TOK, (0,), P)
    setup = _prefix_setup(cfg, [prefix])
    L0 = []
    for r in range(R):
        body = tokens(s, TAG_SUFFIX_TOK, (r,), int(S[r] + g[r] - 1))
        setup.append(Op("add", r, _concat(prefix, body)))
        k, v = _kv_values(cfg, (3, r), len(body))
        setup.append(Op("write_kv", r, k=k, v=v))
        L0.append(P + len(body))
    qv = _q_values(cfg, (0,), R)
    kn, vn = _kv_values(cfg, (2, 0), R)

    def step(st: int) -> Launch:
        pre = [Op("extend", r, tokens(s, TAG_STEP + st, (r,), 1)) for r in range(R)]
        post = [Op("truncate", r, n=L0[r]) for r in range(R)]
        return Launch(pre, list(range(R)), [1] * R, qv, kn, vn, post)

    needed = P // bs + sum(_cdiv(L0[r] + 1, bs) - P // bs for r in range(R))
    nb, free_order = _pool(needed, s)
    return Workload(cfg, nb, free_order, setup, [step(0)], step,
                    _cdiv(P + hi + 128, bs), {"prefix": P, "suffix": S.tolist(), "generated": g.tolist()})


ZIPF_S = 1.1


def zipf_probs(n: int, s: float = ZIPF_S) -> np.ndarray:
    w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    return w / w.sum()


def _mixed(cfg: AttnConfig, scale: float = 1.0, steps: int = 1,
           requests: Optional[int] = None) -> Workload:
    """Chunked-prefill chunks and decode tokens of many requests in one launch,
    over four cached prefixes chosen with Zipf(1.1) popularity."""
    s, bs = cfg.seed, cfg.block_size
    R = requests or max(2, int(round(512 * scale)))
    n_chunk_req = max(1, R // 8)
    C = 512 if scale >= 1 else max(bs, int(round(512 * scale)))
    plens = [1024, 2048, 4096, 8192] if scale >= 1 else [max(bs, int(round(x * scale / bs)) * bs)
                                                        for x in (1024, 2048, 4096, 8192)]
    lo, hi = (256, 1024) if scale >= 1 else (max(1, int(256 * scale)), max(2, int(1024 * scale)))
    prefixes = [tokens(s, TAG_PREFIX_TOK, (p,), plens[p]) for p in range(4)]
    pid = rng(s, TAG_ZIPF).choice(4, size=R, p=zipf_probs(4))
    chunk_reqs = set(rng(s, TAG_SPLIT, 0).permutation(R)[:n_chunk_req].tolist())
    cidx = rng(s, TAG_SPLIT, 1).integers(0, 2, size=R)
    S = rng(s, TAG_LEN, 0).integers(lo, hi + 1, size=R)
    g = rng(s, TAG_LEN, 1).integers(1, 129, size=R)
    setup = _prefix_setup(cfg, prefixes)
    kind, L0, q_lens = [], [], []
    for r in range(R):
        P = plens[pid[r]]
        if r in chunk_reqs:
            if cidx[r] == 1:
                body = tokens(s, TAG_SUFFIX_TOK, (r, 0), C)
                setup.append(Op("add", r, _concat(prefixes[pid[r]], body)))
                k, v = _kv_values(cfg, (3, r), C)
                setup.append(Op("write_kv", r, k=k, v=v))
                kind.append("chunk1")
                L0.append(P + C)
            else:
                kind.append("chunk0")
                L0.append(P)
            q_lens.append(C)
        else:
            body = tokens(s, TAG_SUFFIX_TOK, (r, 0), int(S[r] + g[r] - 1))
            setup.append(Op("add", r, _concat(prefixes[pid[r]], body)))
            k, v = _kv_values(cfg, (3, r), len(body))
            setup.append(Op("write_kv", r, k=k, v=v))
            kind.append("decode")
            L0.append(P + len(body))
            q_lens.append(1)
    T = int(sum(q_lens))
    qv = _q_values(cfg, (0,), T)
    kn, vn = _kv_values(cfg, (2, 0), T)

    def step(st: int) -> Launch:
        pre, post = [], []
        for r in range(R):
            if kind[r] == "chunk0":
                pre.append(Op("add", r, _concat(prefixes[pid[r]],
                                                tokens(s, TAG_SUFFIX_TOK, (r, 1, st), C))))
                post.append(Op("free", r))
            elif kind[r] == "chunk1":
                pre.append(Op("extend", r, tokens(s, TAG_SUFFIX_TOK, (r, 2, st), C)))
                post.append(Op("truncate", r, n=L0[r]))
            else:
                pre.append(Op("extend", r, tokens(s, TAG_STEP + st, (r,), 1)))
                post.append(Op("truncate", r, n=L0[r]))
        return Launch(pre, list(range(R)), list(q_lens), qv, kn, vn, post)

    base = sum(p // bs for p in plens)
    needed = base + sum(_cdiv(L0[r] + q_lens[r], bs) - plens[pid[r]] // bs for r in range(R))
    per_step = sum(_cdiv(plens[pid[r]] + C, bs) - plens[pid[r]] // bs
                   for r in range(R) if kind[r] == "chunk0")
    nb, free_order = _pool(needed + per_step * max(0, steps - 1), s)
    return Workload(cfg, nb, free_order, setup, [step(0)], step,
                    _cdiv(max(plens) + max(2 * C, hi + 128), bs),
                    {"prefixes": plens, "prefix_id": pid.tolist(), "kind": kind,
                     "chunk": C})


def _verify(cfg: AttnConfig, scale: float = 1.0, steps: int = 1,
            requests: Optional[int] = None) -> Workload:
    """Speculative verification: 4 draft tokens + 1 per request over a long
    shared prefix and a long cached private suffix, causal among the drafts."""
    s, bs = cfg.seed, cfg.block_size
    R = requests or max(1, int(round(32 * scale)))
    P = 16384 if scale >= 1 else max(bs, int(round(16384 * scale / bs)) * bs)
    Sx = 4096 if scale >= 1 else max(1, int(round(4096 * scale)))
    NQ = 5
    prefix = tokens(s, TAG_PREFIX_TOK, (0,), P)
    setup = _prefix_setup(cfg, [prefix])
    for r in range(R):
        body = tokens(s, TAG_SUFFIX_TOK, (r,), Sx)
        setup.append(Op("add", r, _concat(prefix, body)))
        k, v = _kv_values(cfg, (3, r), Sx)
        setup.append(Op("write_kv", r, k=k, v=v))
    qv = _q_values(cfg, (0,), R * NQ)
    kn, vn = _kv_values(cfg, (2, 0), R * NQ)

    def step(st: int) -> Launch:
        pre = [Op("extend", r, tokens(s, TAG_STEP + st, (r,), NQ)) for r in range(R)]
        post = [Op("truncate", r, n=P + Sx) for r in range(R)]
        return Launch(pre, list(range(R)), [NQ] * R, qv, kn, vn, post)

    needed = P // bs + R * (_cdiv(P + Sx + NQ, bs) - P // bs)
    nb, free_order = _pool(needed, s)
    return Workload(cfg, nb, free_order, setup, [step(0)], step, _cdiv(P + Sx + NQ, bs),
                    {"prefix": P, "suffix": Sx, "n_q": NQ})


def _evict(cfg: AttnConfig, scale: float = 1.0, steps: int = 1) -> Workload:
    """Prefix-cache lifecycle: two 64-token prefixes are cached in a pool of 12
    blocks (block size 16) with least-recently-used eviction.  Launch 0 admits
    two 104-token requests on the second prefix; the second request finds one
    free block and evicts the first prefix's last two blocks.  Launch 1 admits
    a request on the first prefix: it reuses the two surviving blocks (32
    tokens) and computes the other 72 tokens, the evicted 32 prefix tokens
    included, with the prefill kernel.  The hit counts follow from the
    eviction rules by hand (least recently released idle leaf first)."""
    s, bs = cfg.seed, cfg.block_size
    P, S = 64, 40
    p1, p2 = tokens(s, TAG_PREFIX_TOK, (0,), P), tokens(s, TAG_PREFIX_TOK, (1,), P)
    setup = _prefix_setup(cfg, [p1, p2])
    suf = [tokens(s, TAG_SUFFIX_TOK, (r,), S) for r in range(3)]
    k0, v0 = _kv_values(cfg, (2, 0), 2 * S)
    l0 = Launch([Op("add", 0, _concat(p2, suf[0])), Op("add", 1, _concat(p2, suf[1]))], [0, 1],
                [S, S], _q_values(cfg, (0,), 2 * S), k0, v0, [Op("free", 0), Op("free", 1)])
    q1 = P + S - 32
    k1, v1 = _kv_values(cfg, (2, 1), q1)
    l1 = Launch([Op("add", 2, _concat(p1, suf[2]))], [2], [q1], _q_values(cfg, (1,), q1), k1, v1,
                [Op("free", 2)])
    nb = 12
    free_order = rng(s, TAG_FREE).permutation(nb).astype(np.int32)
    return Workload(cfg, nb, free_order, setup, [l0, l1], None, _cdiv(P + S, bs),
                    {"prefix": P, "suffix": S, "expected_hits": [[P, P], [32]]}, evict=True)


_BUILDERS = {"tiny": _tiny, "prefill": _prefill, "decode": _decode,
             "mixed": _mixed, "verify": _verify, "evict": _evict}


def workload(name: str, scale: float = 1.0, steps: int = 1, requests: Optional[int] = None,
             **overrides) -> Workload:
    """Build the named workload.  ``scale < 1`` shrinks request counts and
    lengths for parity tests (same recipe, same seeds); ``requests`` sets the
    request count alone (prefill, decode, mixed, verify: the first requests
    of the same draws at the given scale's lengths); ``steps`` sizes the
    block pool for that many repeated launches; ``overrides`` replace config
    fields (e.g. ``dtype``, ``head_dim``)."""
    cfg = dataclasses.replace(CONFIGS[name], **overrides) if overrides else CONFIGS[name]
    if requests is not None:
        return _BUILDERS[name](cfg, scale, steps, requests=requests)
    return _BUILDERS[name](cfg, scale, steps)
