"""Shared helpers for the GPU parity tests: replay one workload through the
oracle and through libpa, compare tables bit for bit, the appended cache bit
for bit, and attention outputs within the stated tolerance."""
from __future__ import annotations

import ctypes as C
import sys

import numpy as np
import torch

from oracle.run import OracleReplay
from paper_2605_11232_amd import binding as B
from paper_2605_11232_amd.runtime import DeviceReplay, Staging, plan_words_bound

# Elementwise |o - r| <= atol + rtol * |r|: bf16 inputs with float32
# accumulation 1e-2 / 2e-2; the float32 path 1e-5 / 1e-5.
TOL = {"bf16": (1e-2, 2e-2), "f32": (1e-5, 1e-5)}
# log-sum-exp (not part of the stated tolerance; derived from float32 score
# accumulation of exactly represented products, see the design notes)
LSE_TOL = {"bf16": (2e-3, 1e-4), "f32": (1e-5, 1e-6)}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def close(out, ref, atol, rtol, what):
    out = np.asarray(out, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    m = ~np.isnan(ref)
    assert m.any(), what
    err = np.abs(out[m] - ref[m])
    bound = atol + rtol * np.abs(ref[m])
    rms = float(np.sqrt(np.mean(ref[m] ** 2))) or 1.0
    worst = int(np.argmax(err - bound))
    info = (f"{what}: max|err| {err.max():.3e}, normalized {err.max() / rms:.3e}, "
            f"worst err {err[worst]:.3e} vs bound {bound[worst]:.3e}")
    assert np.all(np.isfinite(out[m])), what + ": non-finite output"
    assert np.all(err <= bound), info
    return err.max() / rms


def key_slot_pos(off):
    """Position of token offset ``off`` inside a 32-dim group of the key
    cache (include/pa.h: the offset with bits 2 and 3 swapped)."""
    off = np.asarray(off)
    return (off & ~12) | ((off & 4) << 1) | ((off & 8) >> 1)


def compare_cache(dev: DeviceReplay, prep, k_new, v_new):
    """The appended K/V sit at their slots bit for bit (layouts as documented:
    keys [block][head][dim / 32][slot position][32], values
    [block][head][dim][offset])."""
    slots = prep.meta["slot_mapping"].astype(np.int64)
    if slots.size == 0:
        return
    bs = dev.cfg.block_size
    blk = torch.from_numpy(slots // bs).to(dev.device)
    off = torch.from_numpy(slots % bs).to(dev.device)
    pos = torch.from_numpy(key_slot_pos(slots % bs)).to(dev.device)
    kd = dev.k_cache[blk, :, :, pos, :].float().cpu().numpy().reshape(k_new.shape)
    vd = dev.v_cache[blk, :, :, off].float().cpu().numpy()
    np.testing.assert_array_equal(kd, k_new)
    np.testing.assert_array_equal(vd, v_new)


def run_parity(wl, n_launches=None, rows=None, steps=None, check_cache=True, label="",
               staged=False, stage_kernel=True, cascade=True):
    """Replay ``wl`` through both; returns per-launch normalized errors.
    ``staged``: the device side runs the benchmark's path (one library call
    for pool operations, metadata and plan into alternating pinned staging
    buffers, one upload each, a reused workspace, odd launches released by a
    caller's event; ``stage_kernel``: the upload by the library's kernel, else
    by a copy-engine copy; ``cascade``: shared-prefix groups in the plans).
    The returned device replay's ``infos`` holds each launch's plan info and
    ``outs`` its (out, lse) as float arrays."""
    cfg = wl.cfg
    atol, rtol = TOL[cfg.dtype]
    latol, lrtol = LSE_TOL[cfg.dtype]
    say(f"[parity] {label or cfg.name}: setup")
    orc = OracleReplay(wl).setup()
    dev = DeviceReplay(wl, stage_kernel=stage_kernel, cascade=cascade).setup()
    dev.infos, dev.outs = [], []
    launches = list(wl.launches[:n_launches] if n_launches else wl.launches)
    if steps:
        launches += [wl.step(s) for s in steps]
    errs = []
    stagings = None
    if staged:
        n = max(len(ln.seq_ids) for ln in launches)
        T = max(ln.total_q for ln in launches)
        words = plan_words_bound(cfg, n, T, wl.max_blocks_per_seq)
        stagings = [Staging(dev.device, n, wl.max_blocks_per_seq, T, words) for _ in range(2)]
    for li, launch in enumerate(launches):
        say(f"[parity] {label or cfg.name}: launch {li} ({launch.total_q} query tokens)"
            + (" staged" if staged else ""))
        ro = orc.launch(launch, rows=rows)
        if staged:
            T = launch.total_q
            q = torch.from_numpy(launch.q.get()).to(dev.device, dev.tdtype)
            k_new = torch.from_numpy(launch.k_new.get()).to(dev.device, dev.tdtype)
            v_new = torch.from_numpy(launch.v_new.get()).to(dev.device, dev.tdtype)
            out = torch.empty((T, cfg.num_q_heads, cfg.head_dim), dtype=dev.tdtype,
                              device=dev.device)
            lse = torch.empty((T, cfg.num_q_heads), dtype=torch.float32, device=dev.device)
            # odd launches release their staging buffer through the start
            # event of the attention call, carried by its first kernel's
            # dispatch, and time the call (the benchmark's timed steps)
            timed = (B.StreamEvent(timing=True), B.StreamEvent(timing=True)) if li % 2 else None
            p = dev.prepare_staged(launch, stagings[li % 2], q, k_new, v_new, out, lse,
                                   guard=timed[0] if timed else None)
            dev.append(p, record_guard=False)
            dev.attend(p, events=timed)
        else:
            p = dev.run(launch)
            timed = None
        torch.cuda.synchronize()
        if timed:
            assert timed[0].elapsed_time(timed[1]) > 0.0
        for k in ("block_table", "seq_lens", "cu_seqlens_q", "slot_mapping"):
            np.testing.assert_array_equal(p.meta[k], ro["meta"][k], err_msg=k)
        assert p.n_cached == ro["n_cached"]
        if check_cache:
            compare_cache(dev, p, launch.k_new.get(), launch.v_new.get())
        out = p.out.float().cpu().numpy()
        lse = p.lse.cpu().numpy()
        info = B.PlanInfo()
        C.memmove(C.byref(info), C.byref(p.info), C.sizeof(info))
        dev.infos.append(info)
        dev.outs.append((out, lse))
        errs.append(close(out, ro["out"], atol, rtol, f"out[{li}]"))
        close(lse, ro["lse"], latol, lrtol, f"lse[{li}]")
        orc.finish(launch)
        dev.finish(launch, batched=staged)
    return errs, dev, orc


def sample_rows(launch, n_random, num_q_heads, seed=0):
    """Sampled (token, head) rows: the first and last query of every request
    (random heads) plus ``n_random`` random rows."""
    r = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(launch.q_lens)])
    rows = set()
    for i in range(len(launch.q_lens)):
        if launch.q_lens[i]:
            rows.add((int(cu[i]), int(r.integers(num_q_heads))))
            rows.add((int(cu[i + 1] - 1), int(r.integers(num_q_heads))))
    for _ in range(n_random):
        rows.add((int(r.integers(cu[-1])), int(r.integers(num_q_heads))))
    return sorted(rows)
