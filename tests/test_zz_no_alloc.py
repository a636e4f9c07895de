"""pa_attn_decode_noalloc (split-K partials in the library's per-device
array) against pa_attn_decode (caller's workspace): two calls in a row, the
second on a smaller launch, each bit-identical to the workspace entry point
on the same plan and inputs, and within the bf16 tolerance of the oracle."""
import numpy as np
import pytest
import torch

from paper_2605_11232_amd import binding as B, synth
from tests.parity import TOL, LSE_TOL, close, say

pytestmark = pytest.mark.gpu


def _one(scale, seed_steps):
    from oracle.run import OracleReplay
    from paper_2605_11232_amd.runtime import DeviceReplay
    wl = synth.workload("decode", scale=scale, steps=seed_steps)
    dev = DeviceReplay(wl).setup()
    orc = OracleReplay(wl).setup()
    launch = wl.launches[0]
    ro = orc.launch(launch)
    p = dev.prepare(launch)
    assert p.info.workspace_bytes > 0          # split keys: the array is used
    assert p.info.workspace_bytes <= B.NOALLOC_WORKSPACE_BYTES
    dev.append(p)
    # the entry point with a caller workspace, then the no-allocation one
    dev.attend(p)
    out2 = torch.empty_like(p.out)
    lse2 = torch.empty_like(p.lse)
    B.attention_decode_noalloc(p.q, dev.k_cache, dev.v_cache, p.block_table, p.seq_lens, p.cu,
                               p.plan, p.info, out2, lse2)
    torch.cuda.synchronize()
    a = p.out.view(torch.int16).cpu().numpy()
    b = out2.view(torch.int16).cpu().numpy()
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(p.lse.cpu().numpy(), lse2.cpu().numpy())
    close(out2.float().cpu().numpy(), ro["out"], *TOL["bf16"], f"noalloc out @{scale}")
    close(lse2.cpu().numpy(), ro["lse"], *LSE_TOL["bf16"], f"noalloc lse @{scale}")
    return int(p.info.workspace_bytes)


def test_noalloc_decode_matches_workspace_entry_point():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    say("[noalloc] decode @0.25")
    big = _one(0.25, 2)
    say("[noalloc] decode @0.0625 (smaller, after the first)")
    small = _one(0.0625, 2)
    say(f"[noalloc] workspace bytes {big} then {small}")
    assert small < big
