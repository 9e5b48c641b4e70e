"""Long-trace drift on the GPU against the oracle's (App. B.1, Sec. 3.2).

The quantized GDN trajectory (decode steps and window commits, W = 128, r = 8)
and the unquantized fp32 trajectory (the baseline kernel) run side by side on
the GPU from the same fp32 initial state; every 1024 tokens, right after a
commit, the relative Frobenius distance of the dequantized state from the fp32
state and the relative L2 distance of that token's outputs are taken per tile.
The oracle's ``run_drift`` computes the same two curves on the same tiles and
tokens.  The two must agree point by point to 1e-3 relative: the quantized
trajectories are the same (the GPU reproduces the oracle's records and commits
bit for bit), and the two fp32 baselines differ only by fp32 summation order,
about 1e-7 of a state whose distance from the quantized one is about 3e-3.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2609_38166_amd import binding as B, synth

from . import gpu_harness as H

pytestmark = pytest.mark.gpu

EVERY = 1024


def gpu_drift(wl, S0, tok, every=EVERY):
    """Per-tile state and output drift [tiles][steps // every] on the GPU."""
    dims = H.gdims(wl)
    st = B.State.empty(dims)
    S0t = H.dev(S0.transpose(0, 2, 1).astype(np.float32))
    B.leapquant_quantize_state(dims, S0t, st)
    F = S0t.clone()
    Sq = torch.empty_like(F)
    dt = H.DeviceTokens(wl, tok)
    o1 = torch.empty((wl.tiles, wl.dv), dtype=torch.float32, device="cuda")
    o2 = torch.empty_like(o1)
    sd, od = [], []
    for t in range(wl.steps):
        x = dt.step(t)
        B.leapquant_decode_step(dims, st, *x, o1)
        B.leapquant_baseline_step(dims, F, B.LQ_STATE_F32, *x, o2)
        if (t + 1) % wl.window == 0:
            B.leapquant_window_commit(dims, st)
        if (t + 1) % every == 0:
            B.leapquant_dequantize_state(dims, st, Sq)
            d = (Sq - F).flatten(1).double().norm(dim=1) / F.flatten(1).double().norm(dim=1)
            e = (o1 - o2).double().norm(dim=1) / o2.double().norm(dim=1)
            sd.append(d.cpu().numpy())
            od.append(e.cpu().numpy())
    assert B.leapquant_check_error(st) == 0
    return np.stack(sd, axis=1), np.stack(od, axis=1)


@pytest.mark.parametrize("gate_scale", [0.1, 0.001])
def test_long_trace_drift_matches_oracle(gate_scale):
    """One request (16 tiles) of the long GDN trace, 4096 tokens; gate scale
    0.1 is the workload's (state half-life about 9 tokens), 0.001 a long-memory
    variant whose state keeps thousands of tokens of history."""
    wl = synth.WORKLOADS["gdn_long"].with_(batch=1, steps=4096, gate_scale=gate_scale)
    H.log(f"long trace: {wl.tiles} tiles, {wl.steps} tokens, gate scale {gate_scale}")
    cfg = H.ocfg(wl)
    S0 = H.oracle_prefill_state(wl)
    streams, tok = H.decode_tokens(wl)
    otok = synth.tile_major(wl, streams, tok)
    d_orc, o_orc = O.run_drift(cfg, S0, otok, EVERY)
    d_gpu, o_gpu = gpu_drift(wl, S0, tok)
    H.log(f"state drift gpu {d_gpu.mean(axis=0)} oracle {d_orc.mean(axis=0)}; "
          f"output drift gpu {o_gpu.mean(axis=0)} oracle {o_orc.mean(axis=0)}")
    assert np.all(np.isfinite(d_gpu)) and np.all(d_orc > 0)
    # The quantization error itself: about 1e-3 .. 1e-1 of the state's norm for 8 bits.
    assert 1e-4 < d_orc.mean() < 0.2
    np.testing.assert_allclose(d_gpu, d_orc, rtol=1e-3)
    np.testing.assert_allclose(o_gpu, o_orc, rtol=1e-3)


def test_long_trace_full_length_matches_oracle():
    """The whole 32768-token long trace (W = 128, r = 8, the workload's gates)
    on two tiles of its first request, GPU against the oracle at every 1024th
    token: 32 points per tile."""
    wl = synth.WORKLOADS["gdn_long"].with_(batch=1, heads_v=2, heads_k=2)
    H.log(f"long trace, full length: {wl.tiles} tiles, {wl.steps} tokens")
    cfg = H.ocfg(wl)
    S0 = H.oracle_prefill_state(wl)
    streams, tok = H.decode_tokens(wl)
    otok = synth.tile_major(wl, streams, tok)
    d_orc, o_orc = O.run_drift(cfg, S0, otok, EVERY)
    d_gpu, o_gpu = gpu_drift(wl, S0, tok)
    assert d_gpu.shape == (2, 32)
    H.log(f"state drift gpu {d_gpu.mean():.5f} oracle {d_orc.mean():.5f}; worst point ratio "
          f"{np.max(np.abs(d_gpu / d_orc - 1)):.4f}")
    np.testing.assert_allclose(d_gpu, d_orc, rtol=1e-3)
    np.testing.assert_allclose(o_gpu, o_orc, rtol=1e-3)
