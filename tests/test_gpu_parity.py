"""GPU parity of every kernel behind the C ABI against the CPU oracle.

Bars: outputs and dequantized states within relative L2 1e-3 per tile, INT8 /
E4M3 codes equal in >= 99.9 % of entries and at most one grid step apart
elsewhere, FP16 records bit-equal in >= 99.9 % of entries.  Code-level
parity is checked window by window (the GPU starts each window from the
oracle's representation): a free-running fp32 trajectory and an fp64 one drift
apart at the level of the quantization noise itself, because any rounding
decision that flips propagates, so free-running runs are checked by properties.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2609_38166_amd import binding as B
from paper_2609_38166_amd import synth
from tests import gpu_harness as H

pytestmark = pytest.mark.gpu

W_ = synth.WORKLOADS
SMALL = {
    "gdn_tiny": W_["gdn_tiny"],
    "kda_small": W_["kda_kimi"].with_(name="kda_small", batch=2, heads_v=4, heads_k=4, steps=128,
                                      prefill=256),
    "gqa_int8_small": W_["gdn_qwen3next"].with_(name="gqa_int8_small", batch=2, heads_v=4,
                                                heads_k=2, steps=128, prefill=256),
    "gqa_e4m3_small": W_["gdn_qwen3next"].with_(name="gqa_e4m3_small", batch=2, heads_v=4,
                                                heads_k=2, steps=128, prefill=256,
                                                code=synth.CODE_E4M3),
    "stress_small": W_["gdn_stress"].with_(name="stress_small", batch=4, heads_v=32, heads_k=32,
                                           steps=64, prefill=128),
    "kda_w16_r4": W_["kda_kimi"].with_(name="kda_w16_r4", batch=2, heads_v=4, heads_k=4, steps=64,
                                       window=16, n_comp=4, prefill=128),
    # per-channel gate with grouped key heads (two value heads per key head) and E4M3 codes
    "kda_gqa_e4m3": W_["kda_kimi"].with_(name="kda_gqa_e4m3", batch=2, heads_v=4, heads_k=2, steps=64,
                                         window=32, n_comp=8, prefill=128, code=synth.CODE_E4M3),
    "kda_int4_small": W_["kda_kimi"].with_(name="kda_int4_small", batch=2, heads_v=4, heads_k=4,
                                           steps=128, prefill=256, code=synth.CODE_INT4),
    "gdn_int6_small": W_["gdn_tiny"].with_(name="gdn_int6_small", code=synth.CODE_INT6),
    # corners of the window / token / smoothing sweeps (the paper's ablations)
    "per_step_w1": W_["gdn_tiny"].with_(name="per_step_w1", steps=24, window=1, n_comp=0, smooth=0),
    "w4_r2": W_["gdn_tiny"].with_(name="w4_r2", steps=64, window=4, n_comp=2),
    "w8_r16": W_["gdn_tiny"].with_(name="w8_r16", steps=64, window=8, n_comp=16),
    "w32_r4_nosmooth": W_["kda_kimi"].with_(name="w32_r4_nosmooth", batch=2, heads_v=4, heads_k=4,
                                            steps=64, window=32, n_comp=4, smooth=0, prefill=128),
    # power-sweep counts other than the workloads' four: one sweep per token, and sixteen
    "kda_pi1": W_["kda_kimi"].with_(name="kda_pi1", batch=2, heads_v=4, heads_k=4, steps=64, window=16,
                                    n_comp=4, prefill=128, power_iters=1),
    "gdn_pi16": W_["gdn_tiny"].with_(name="gdn_pi16", steps=64, window=16, n_comp=8, power_iters=16),
    # the largest window of the scalar gate (four record passes in the decode), and a
    # ragged tile count (3 requests x 5 heads)
    "gdn_w256": W_["gdn_tiny"].with_(name="gdn_w256", batch=2, heads_v=2, heads_k=2, steps=256, window=256,
                                     prefill=128),
    # the largest windows of the per-channel gate: three and six record passes of 48 in
    # the decode, eight and sixteen passes of 16 in the commit
    "kda_w128": W_["kda_kimi"].with_(name="kda_w128", batch=1, heads_v=4, heads_k=4, steps=256, window=128,
                                     prefill=128),
    "kda_w256": W_["kda_kimi"].with_(name="kda_w256", batch=1, heads_v=2, heads_k=2, steps=256, window=256,
                                     prefill=128),
    "ragged_3x5": W_["gdn_tiny"].with_(name="ragged_3x5", batch=3, heads_v=5, heads_k=5, steps=48, prefill=128),
    # a launch of one workgroup
    "kda_one_tile": W_["kda_kimi"].with_(name="kda_one_tile", batch=1, heads_v=1, heads_k=1, steps=80, window=32,
                                         prefill=128),
    # b_t = 0 rows of the instance table: Mamba2 (scalar decay), GLA / RWKV6 (per-channel)
    "mamba2_small": W_["gdn_tiny"].with_(name="mamba2_small", rule=1),
    "gla_small": W_["kda_kimi"].with_(name="gla_small", batch=2, heads_v=4, heads_k=4, steps=128,
                                      prefill=256, rule=1),
    # the same rows with the other code formats
    "mamba2_e4m3": W_["gdn_tiny"].with_(name="mamba2_e4m3", rule=1, code=synth.CODE_E4M3),
    "mamba2_int4": W_["gdn_tiny"].with_(name="mamba2_int4", rule=1, code=synth.CODE_INT4, n_comp=8),
    "gla_int6": W_["kda_kimi"].with_(name="gla_int6", batch=2, heads_v=4, heads_k=4, steps=64, window=32,
                                     n_comp=4, prefill=128, rule=1, code=synth.CODE_INT6),
    # the per-window BF16 state (row f3): BF16 rounding at window ends, no tokens
    "bf16w_gdn": W_["gdn_tiny"].with_(name="bf16w_gdn", code=synth.CODE_BF16, n_comp=0, smooth=0),
    "bf16w_kda": W_["kda_kimi"].with_(name="bf16w_kda", batch=2, heads_v=4, heads_k=4, steps=128, window=32,
                                      prefill=256, code=synth.CODE_BF16, n_comp=0, smooth=0),
    "bf16w_gqa_w1": W_["gdn_qwen3next"].with_(name="bf16w_gqa_w1", batch=2, heads_v=4, heads_k=2, steps=12,
                                              window=1, prefill=64, code=synth.CODE_BF16, n_comp=0, smooth=0),
}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    yield
    torch.cuda.synchronize()


def _tokens_random(wl, T, seed):
    st = synth.Streams(wl.with_(seed=seed), synth.PHASE_DECODE)
    tok = st.draw(T)
    st.close()
    return st, tok


@pytest.mark.parametrize("rule", [0, 1])
@pytest.mark.parametrize("gate", [synth.GATE_SCALAR, synth.GATE_DIAG])
@pytest.mark.parametrize("dtype", [B.LQ_STATE_F32, B.LQ_STATE_BF16])
def test_baseline_step_parity(gate, dtype, rule):
    wl = W_["gdn_tiny"].with_(batch=2, heads_v=4, heads_k=2, gate=gate, rule=rule)
    H.log(f"baseline gate={gate} dtype={dtype} rule={rule}")
    rng = np.random.default_rng(5)
    S0 = rng.standard_normal((wl.tiles, wl.dk, wl.dv)).astype(np.float32).astype(np.float64)
    if dtype == B.LQ_STATE_BF16:
        S0 = O.f32_to_bf16_bits(S0.astype(np.float32)).astype(np.uint32) << 16
        S0 = S0.view(np.float32).astype(np.float64)
    streams, tok = _tokens_random(wl, 24, 77)
    o_ref, S_ref = O.run_baseline(H.ocfg(wl), S0, synth.tile_major(wl, streams, tok),
                                  mode=O.STATE_F32 if dtype == B.LQ_STATE_F32 else O.STATE_BF16)
    dims = H.gdims(wl)
    S_t = np.ascontiguousarray(S0.transpose(0, 2, 1)).astype(np.float32)
    if dtype == B.LQ_STATE_BF16:
        S_g = H.dev(S_t).to(torch.bfloat16)
    else:
        S_g = H.dev(S_t)
    dt = H.DeviceTokens(wl, tok)
    o = torch.empty((wl.tiles, wl.dv), dtype=torch.float32, device="cuda")
    outs = []
    for t in range(24):
        B.leapquant_baseline_step(dims, S_g, dtype, *dt.step(t), o)
        outs.append(o.cpu().numpy())
    og = np.stack(outs, axis=1)
    Sg = S_g.float().cpu().numpy().transpose(0, 2, 1)
    tol = 1e-5 if dtype == B.LQ_STATE_F32 else 2e-3
    assert H.rel_rows(og, o_ref) < tol
    assert H.rel_rows(Sg.reshape(wl.tiles, -1), S_ref.reshape(wl.tiles, -1)) < tol
    if dtype == B.LQ_STATE_BF16:
        # the stored state is bf16 with its values mostly equal to the oracle's
        ref_bits = O.f32_to_bf16_bits(S_ref.astype(np.float32))
        got_bits = S_g.view(torch.int16).cpu().numpy().view(np.uint16).transpose(0, 2, 1)
        assert np.mean(ref_bits == got_bits) > 0.99


def test_prefill_parity_fp32():
    """512-token fp32 prefill of the tiny GDN workload (the initial-state recipe)."""
    wl = W_["gdn_tiny"]
    st = synth.Streams(wl, synth.PHASE_PREFILL)
    tok = st.draw(wl.prefill)
    _, S_ref = O.run_baseline(H.ocfg(wl), np.zeros((wl.tiles, 128, 128)),
                              synth.tile_major(wl, st, tok), mode=O.STATE_F32, want_o=False)
    dims = H.gdims(wl)
    S_g = torch.zeros((wl.tiles, 128, 128), dtype=torch.float32, device="cuda")
    dt = H.DeviceTokens(wl, tok)
    o = torch.empty((wl.tiles, 128), dtype=torch.float32, device="cuda")
    for t in range(wl.prefill):
        B.leapquant_baseline_step(dims, S_g, B.LQ_STATE_F32, *dt.step(t), o)
    Sg = S_g.cpu().numpy().transpose(0, 2, 1)
    assert H.rel_rows(Sg.reshape(wl.tiles, -1), S_ref.reshape(wl.tiles, -1)) < 1e-5


def _states_with_edges(n, seed):
    rng = np.random.default_rng(seed)
    S = []
    for i in range(n):
        s = sum(np.outer(rng.standard_normal(128), rng.standard_normal(128)) * 0.7 ** j for j in range(6))
        s = s + 0.3 * rng.standard_normal((128, 128))
        s[rng.choice(128, 2, replace=False), :] *= 20
        s[:, rng.choice(128, 2, replace=False)] *= 20
        S.append(s)
    S = np.stack(S)
    S[1] = 0.0                                   # all-zero tile
    S[2][:, [5, 99]] = 0.0                       # zero value columns
    S[3] = np.outer(rng.standard_normal(128), rng.standard_normal(128))   # rank one
    return S.astype(np.float32).astype(np.float64)   # both sides get the same fp32 values


@pytest.mark.parametrize("code", [synth.CODE_INT8, synth.CODE_E4M3, synth.CODE_INT4, synth.CODE_INT6])
@pytest.mark.parametrize("r", [0, 4, 8])
@pytest.mark.parametrize("smooth", [0, 1])
def test_quantize_state_parity(code, r, smooth):
    H.log(f"quantize code={code} r={r} smooth={smooth}")
    wl = W_["gdn_tiny"].with_(batch=4, heads_v=8, heads_k=8, n_comp=r, code=code)
    S = _states_with_edges(wl.tiles, 100 + r)
    cfg = H.ocfg(wl, smooth=smooth)
    exp = {"Z": [], "delta": [], "c": [], "Kt": [], "Ut": []}
    for i in range(wl.tiles):
        rep = O.quantize(cfg, S[i])
        for k_ in exp:
            exp[k_].append(getattr(rep, k_))
    exp = {k_: np.stack(v_) for k_, v_ in exp.items()}
    dims = H.gdims(wl, smooth=smooth)
    st = B.State.empty(dims)
    st.rec_len.fill_(5)
    B.leapquant_quantize_state(dims, H.dev(S.transpose(0, 2, 1).astype(np.float32)), st)
    got = H.download_rep(st)
    assert np.all(got["rec_len"] == 0)
    cr = H.compare_rep(cfg, got, exp, code)
    H.log(cr)
    assert cr["code_eq"] >= 0.999 and cr["code_maxdiff"] <= 1, cr
    assert cr["deq_rel"] <= 1e-3 and cr["delta_rel"] <= 1e-5 and cr["c_rel"] <= 1e-5, cr
    if r:
        assert cr["comp_rel"] <= 1e-3, cr
    assert not got["Z"][1].any() and not got["delta"][1].any()
    assert got["delta"][2][5] == 0 and got["delta"][2][99] == 0


@pytest.mark.parametrize("power_iters", [1, 64])
def test_quantize_state_parity_power_iters(power_iters):
    """The sweep count at its ends (one sweep per token, and the 64 the ABI
    allows): codes, scales and Compensator Tokens as the oracle's."""
    H.log(f"quantize power_iters={power_iters}")
    wl = W_["gdn_tiny"].with_(batch=4, heads_v=8, heads_k=8, n_comp=8, power_iters=power_iters)
    S = _states_with_edges(wl.tiles, 300 + power_iters)
    cfg = H.ocfg(wl)
    exp = {"Z": [], "delta": [], "c": [], "Kt": [], "Ut": []}
    for i in range(wl.tiles):
        rep = O.quantize(cfg, S[i])
        for k_ in exp:
            exp[k_].append(getattr(rep, k_))
    exp = {k_: np.stack(v_) for k_, v_ in exp.items()}
    dims = H.gdims(wl)
    st = B.State.empty(dims)
    B.leapquant_quantize_state(dims, H.dev(S.transpose(0, 2, 1).astype(np.float32)), st)
    got = H.download_rep(st)
    cr = H.compare_rep(cfg, got, exp, wl.code)
    H.log(cr)
    assert cr["code_eq"] >= 0.999 and cr["code_maxdiff"] <= 1, cr
    assert cr["deq_rel"] <= 1e-3 and cr["delta_rel"] <= 1e-5 and cr["c_rel"] <= 1e-5, cr
    assert cr["comp_rel"] <= 1e-3, cr


def test_quantize_state_parity_bf16():
    """The BF16 state: quantization is the BF16 rounding of every entry (edge
    tiles included), bit for bit."""
    wl = W_["gdn_tiny"].with_(batch=4, heads_v=8, heads_k=8, n_comp=0, code=synth.CODE_BF16, smooth=0)
    S = _states_with_edges(wl.tiles, 150)
    S[0, 0, :8] = np.float32([1e-39, -3e-40, 0.0, -0.0, 1e-45, 3.0e38, -1.17e-38, 7e-39])
    cfg = H.ocfg(wl)
    exp = {"Z": [], "delta": [], "c": [], "Kt": [], "Ut": []}
    for i in range(wl.tiles):
        rep = O.quantize(cfg, S[i])
        for k_ in exp:
            exp[k_].append(getattr(rep, k_))
    exp = {k_: np.stack(v_) for k_, v_ in exp.items()}
    dims = H.gdims(wl)
    st = B.State.empty(dims)
    st.rec_len.fill_(3)
    B.leapquant_quantize_state(dims, H.dev(S.transpose(0, 2, 1).astype(np.float32)), st)
    got = H.download_rep(st)
    assert np.all(got["rec_len"] == 0)
    assert np.array_equal(got["Z"], exp["Z"])
    assert np.all(got["delta"] == 1.0) and np.all(got["c"] == 1.0)


@pytest.mark.parametrize("name", ["gdn_tiny", "kda_small", "gqa_e4m3_small", "kda_int4_small", "gdn_int6_small",
                                  "bf16w_kda"])
def test_dequantize_state_parity(name):
    """Base + open-window records, materialised on the GPU from the oracle's
    representation and records, equals the oracle's dense window state."""
    wl = SMALL[name]
    H.log(f"dequantize {name}")
    cfg = H.ocfg(wl)
    S0 = H.oracle_prefill_state(wl)
    streams, tok = H.decode_tokens(wl, n=wl.window + wl.window // 2 + 1)
    ref = O.run_dense(cfg, S0, synth.tile_major(wl, streams, tok), snapshots=True)
    n = int(ref["rec_len"][0])
    assert n > 0
    dims = H.gdims(wl)
    st = B.State.empty(dims)
    H.upload_rep(st, np.arange(wl.tiles), ref["Z"][:, 1], ref["delta"][:, 1], ref["c"][:, 1],
                 ref["Kt"][:, 1], ref["Ut"][:, 1])
    W, g = wl.window, wl.g
    st.rec_a.view(wl.tiles, W, g)[:] = H.dev(ref["rec_a"].astype(np.float16))
    st.rec_k.view(wl.tiles, W, wl.dk)[:] = H.dev(ref["rec_k"].astype(np.float16))
    st.rec_u.view(wl.tiles, W, wl.dv)[:] = H.dev(ref["rec_u"].astype(np.float16))
    st.rec_len.fill_(n)
    S_out = torch.empty((wl.tiles, 128, 128), dtype=torch.float32, device="cuda")
    B.leapquant_dequantize_state(dims, st, S_out)
    Sg = S_out.cpu().numpy().transpose(0, 2, 1)
    assert H.rel_rows(Sg.reshape(wl.tiles, -1), ref["S_final"].reshape(wl.tiles, -1)) < 1e-5


@pytest.mark.parametrize("name", list(SMALL))
def test_window_synchronised_parity(name):
    wl = SMALL[name]
    H.log(f"window-sync {name}")
    H.window_sync_parity(wl)


@pytest.mark.parametrize("name", ["gdn_tiny", "kda_free"])
def test_free_running_tiny(name):
    """A whole trajectory on the GPU alone: from the oracle's fp32 initial
    state, its own quantization, the decode steps and the commits of its own
    records, with nothing handed back from the oracle (GDN tiny: 256 steps, 16
    commits; KDA: 8 tiles, 256 steps, 4 commits of 64 records, r = 8).  Every
    output and every window-end representation is held to the bars (outputs
    and dequantized states within 1e-3, codes equal in >= 99.9 % and at most
    one step apart).  The quantized trajectory's distance from the unquantized
    fp32 one is reported beside the oracle's."""
    wl = W_["gdn_tiny"] if name == "gdn_tiny" else SMALL["kda_small"].with_(name="kda_free", steps=256)
    H.log(f"free-running {wl.name}")
    cfg = H.ocfg(wl)
    S0 = H.oracle_prefill_state(wl)
    streams, tok = H.decode_tokens(wl)
    otok = synth.tile_major(wl, streams, tok)
    ref = O.run_dense(cfg, S0, otok, snapshots=True)
    o_fp, _ = O.run_baseline(cfg, S0, otok, mode=O.STATE_F32)
    dims = H.gdims(wl)
    st = B.State.empty(dims)
    B.leapquant_quantize_state(dims, H.dev(S0.transpose(0, 2, 1).astype(np.float32)), st)
    dt = H.DeviceTokens(wl, tok)
    o = torch.empty((wl.tiles, 128), dtype=torch.float32, device="cuda")
    outs, worst = [], {"code_eq": 1.0, "code_maxdiff": 0, "deq_rel": 0.0, "comp_rel": 0.0}
    for t in range(wl.steps):
        B.leapquant_decode_step(dims, st, *dt.step(t), o)
        outs.append(o.cpu().numpy())
        if (t + 1) % wl.window == 0:
            B.leapquant_window_commit(dims, st)
            w = (t + 1) // wl.window
            exp = {k_: ref[k_][:, w] for k_ in ("Z", "delta", "c", "Kt", "Ut")}
            cr = H.compare_rep(cfg, H.download_rep(st), exp, wl.code)
            worst["code_eq"] = min(worst["code_eq"], cr["code_eq"])
            for k_ in ("code_maxdiff", "deq_rel", "comp_rel"):
                worst[k_] = max(worst[k_], cr.get(k_, 0))
    og = np.stack(outs, axis=1)
    assert np.all(np.isfinite(og))
    assert B.leapquant_check_error(st) == 0
    o_rel = H.rel_rows(og, ref["o"])
    e_gpu, e_orc = H.rel(og, o_fp), H.rel(ref["o"], o_fp)
    H.log(f"free-running: o_rel {o_rel:.3e} worst commit {worst}; "
          f"gpu-vs-fp32 {e_gpu:.3e} oracle-vs-fp32 {e_orc:.3e}")
    assert o_rel <= 1e-3
    assert worst["code_eq"] >= 0.999 and worst["code_maxdiff"] <= 1, worst
    assert worst["deq_rel"] <= 1e-3 and worst["comp_rel"] <= 1e-3, worst


def test_partial_windows_mask_and_reset():
    """Ragged schedule: 21 tokens, then a commit of request 0 only (a partial
    window), a commit on its now-empty window (a no-op), and a commit of
    everything (request 1's 21 records)."""
    wl = SMALL["kda_small"].with_(steps=40)
    cfg = H.ocfg(wl)
    S0 = H.oracle_prefill_state(wl)
    streams, tok = H.decode_tokens(wl)
    otok = synth.tile_major(wl, streams, tok)
    dims = H.gdims(wl)
    st = B.State.empty(dims)
    rep0 = O.run_dense(cfg, S0, {k_: v_[:, :0] for k_, v_ in otok.items()}, snapshots=True)
    H.upload_rep(st, np.arange(wl.tiles), rep0["Z"][:, 0], rep0["delta"][:, 0], rep0["c"][:, 0],
                 rep0["Kt"][:, 0], rep0["Ut"][:, 0])
    dt = H.DeviceTokens(wl, tok)
    o = torch.empty((wl.tiles, 128), dtype=torch.float32, device="cuda")
    for t in range(21):
        B.leapquant_decode_step(dims, st, *dt.step(t), o)
    mask = torch.tensor([1, 0], dtype=torch.int32, device="cuda")
    before = H.download_rep(st)
    B.leapquant_window_commit(dims, st, mask)
    after = H.download_rep(st)
    h = wl.heads_v
    assert np.all(after["rec_len"][:h] == 0) and np.all(after["rec_len"][h:] == 21)
    for k_ in ("Z", "delta", "c", "Kt", "Ut"):
        assert np.array_equal(after[k_][h:], before[k_][h:])       # unselected: untouched
    # request 0 committed a partial window of 21 tokens from its own records:
    # against the oracle's quantization of its dense state after 21 tokens
    sub = {k_: v_[:h, :21] for k_, v_ in otok.items()}
    ref = O.run_dense(cfg, S0[:h], sub, snapshots=False, history=True)
    exp = {"Z": [], "delta": [], "c": [], "Kt": [], "Ut": []}
    for i in range(h):
        rp = O.quantize(cfg, ref["S_final"][i])
        for k_ in exp:
            exp[k_].append(getattr(rp, k_))
    exp = {k_: np.stack(v_) for k_, v_ in exp.items()}
    got = {k_: after[k_][:h] for k_ in ("Z", "delta", "c", "Kt", "Ut")}
    cr = H.compare_rep(cfg, got, exp, wl.code)
    H.log("partial chained", cr)
    assert cr["code_eq"] >= 0.999 and cr["code_maxdiff"] <= 1 and cr["deq_rel"] <= 1e-3, cr
    assert cr.get("comp_rel", 0.0) <= 1e-3, cr
    # the same partial commit from the oracle's records is exact
    st2 = B.State.empty(dims)
    H.upload_rep(st2, np.arange(wl.tiles), rep0["Z"][:, 0], rep0["delta"][:, 0], rep0["c"][:, 0],
                 rep0["Kt"][:, 0], rep0["Ut"][:, 0])
    full = O.run_dense(cfg, S0, {k_: v_[:, :21] for k_, v_ in otok.items()}, snapshots=False,
                       history=True)
    H.upload_records(st2, full["hist_a"], full["hist_k"], full["hist_u"])
    B.leapquant_window_commit(dims, st2, mask)
    got2 = H.download_rep(st2)
    got2 = {k_: got2[k_][:h] for k_ in ("Z", "delta", "c", "Kt", "Ut")}
    cr2 = H.compare_rep(cfg, got2, exp, wl.code)
    assert cr2["code_eq"] >= 0.999 and cr2["code_maxdiff"] <= 1 and cr2["deq_rel"] <= 1e-3, cr2
    assert cr2["delta_rel"] <= 1e-5 and cr2["c_rel"] <= 1e-5, cr2
    # empty windows: commit is a no-op
    snap = H.download_rep(st)
    B.leapquant_window_commit(dims, st, torch.tensor([1, 0], dtype=torch.int32, device="cuda"))
    again = H.download_rep(st)
    for k_ in ("Z", "delta", "c", "Kt", "Ut", "rec_len"):
        assert np.array_equal(again[k_], snap[k_])
    B.leapquant_window_commit(dims, st)     # all: request 1 commits its 21 records
    assert np.all(H.download_rep(st)["rec_len"] == 0)
    assert B.leapquant_check_error(st) == 0


MIXED = {
    "kda_mixed": (SMALL["kda_small"].with_(name="kda_mixed", batch=6, steps=64), [0, 1, 31, 32, 62, 63]),
    "gqa_mixed": (SMALL["gqa_int8_small"].with_(name="gqa_mixed", batch=6, steps=64), [63, 0, 17, 48, 1, 62]),
    # scalar gate at the largest window: positions in each of the decode's four record passes
    "gdn_w256_mixed": (SMALL["gdn_w256"].with_(name="gdn_w256_mixed", batch=5), [0, 63, 64, 130, 255]),
}


@pytest.mark.parametrize("name", list(MIXED))
def test_requests_at_different_window_positions_in_one_launch(name):
    """A serving batch whose requests sit at different positions of their
    windows: request b has n_b buffered records (the heads of a request share
    its position, as grouped heads share q and k).  One decode launch must give
    every tile the oracle's output for its own token n_b and append its record
    at slot n_b, reading no slot at or past n_b (those hold NaN); a commit of
    the resulting partial windows (p = n_b + 1 records, teacher-forced from the
    oracle's records) must give the oracle's quantization of the reconstructed
    state (Sec. 3.4 Eq. (smooth), Sec. 3.3)."""
    wl, pos = MIXED[name]
    W, Bn, Hv = wl.window, wl.batch, wl.heads_v
    assert len(pos) == Bn and max(pos) < W
    cfg = H.ocfg(wl)
    dims = H.gdims(wl)
    S0 = H.oracle_prefill_state(wl)
    streams, tok = H.decode_tokens(wl, n=W)
    otok = synth.tile_major(wl, streams, tok)
    ref = O.run_dense(cfg, S0, otok, snapshots=True, history=True)
    n_t = np.repeat(np.asarray(pos), Hv)                                 # position per tile
    tiles = np.arange(wl.tiles)
    start = [ref[k_][:, 0] for k_ in ("Z", "delta", "c", "Kt", "Ut")]
    nan16 = torch.tensor(0x7E00, dtype=torch.int16, device="cuda")

    def open_windows(st, n):
        """Oracle records 0..n_t-1 per tile, NaN in every later slot, rec_len = n_t."""
        H.upload_records(st, ref["hist_a"], ref["hist_k"], ref["hist_u"])
        g = wl.dk if wl.gate == synth.GATE_DIAG else 1
        ra = st.rec_a.view(wl.tiles, W, g).view(torch.int16)
        rk = st.rec_k.view(wl.tiles, W, wl.dk).view(torch.int16)
        ru = st.rec_u.view(wl.tiles, W, wl.dv).view(torch.int16)
        past = torch.as_tensor(np.arange(W)[None, :] >= n[:, None], device="cuda")
        for x in (ra, rk, ru):
            x[past] = nan16
        st.rec_len.view(-1)[:] = torch.as_tensor(n, dtype=torch.int32, device="cuda")

    st = B.State.empty(dims)
    H.upload_rep(st, tiles, *start)
    open_windows(st, n_t)
    # the launch: request b takes token pos[b] of its own stream
    sm = synth.step_major_full(wl, tok)
    rq = np.arange(Bn)
    args = [H.dev(np.ascontiguousarray(sm[f][np.asarray(pos), rq])) for f in ("q", "k", "v", "alpha", "beta")]
    o = torch.empty((Bn, Hv, wl.dv), dtype=torch.float32, device="cuda")
    B.leapquant_decode_step(dims, st, *args, o)
    og = o.view(wl.tiles, wl.dv).cpu().numpy()
    exp_o = ref["o"][tiles, n_t]
    o_rel = H.rel_rows(og[:, None], exp_o[:, None])
    g = wl.dk if wl.gate == synth.GATE_DIAG else 1
    got_len = st.rec_len.view(-1).cpu().numpy()
    rk = st.rec_k.view(wl.tiles, W, wl.dk)[tiles, n_t].cpu().numpy().view(np.uint16)
    ru = st.rec_u.view(wl.tiles, W, wl.dv)[tiles, n_t].cpu().numpy().view(np.uint16)
    ra = st.rec_a.view(wl.tiles, W, g)[tiles, n_t].cpu().numpy().view(np.uint16)
    ek = H.f16_bits(ref["hist_k"][tiles, n_t])
    eu = H.f16_bits(ref["hist_u"][tiles, n_t])
    ea = H.f16_bits(ref["hist_a"][tiles, n_t])
    u_rel = H.rel_rows(H.f16_vals(ru)[:, None], ref["hist_u"][tiles, n_t][:, None])
    H.log(f"[{name}] o_rel {o_rel:.3e} u_rel {u_rel:.3e} k_eq {np.mean(rk == ek):.5f} "
          f"u_eq {np.mean(ru == eu):.5f}")
    assert B.leapquant_check_error(st) == 0
    assert np.array_equal(got_len, n_t + 1)
    assert np.all(np.isfinite(og)) and o_rel <= 1e-3
    assert np.array_equal(ra, ea)
    assert np.mean(rk == ek) >= 0.999 and int(H._f16_ulp_dist(rk, ek).max()) <= 1
    assert np.mean(ru == eu) >= 0.999 and int(H._f16_ulp_dist(ru, eu).max()) <= 1 and u_rel <= 1e-3
    # commit of the partial windows, from the oracle's records
    p_t = n_t + 1
    st2 = B.State.empty(dims)
    H.upload_rep(st2, tiles, *start)
    open_windows(st2, p_t)
    B.leapquant_window_commit(dims, st2)
    got = H.download_rep(st2)
    assert np.all(got["rec_len"] == 0) and B.leapquant_check_error(st2) == 0
    exp = {k_: [] for k_ in ("Z", "delta", "c", "Kt", "Ut")}
    for i in tiles:
        rep0 = O.Rep(*(x[i] for x in start))
        p = int(p_t[i])
        Sp = O.reconstruct(cfg, rep0, None, ref["hist_a"][i, :p], ref["hist_k"][i, :p], ref["hist_u"][i, :p])
        rp = O.quantize(cfg, Sp)
        for k_ in exp:
            exp[k_].append(getattr(rp, k_))
    exp = {k_: np.stack(v_) for k_, v_ in exp.items()}
    cr = H.compare_rep(cfg, {k_: got[k_] for k_ in exp}, exp, wl.code)
    H.log(f"[{name}] partial-window commit {cr}")
    assert cr["code_eq"] >= 0.999 and cr["code_maxdiff"] <= 1 and cr["deq_rel"] <= 1e-3, cr
    assert cr.get("comp_rel", 0.0) <= 1e-3 and cr["delta_rel"] <= 1e-5 and cr["c_rel"] <= 1e-5, cr


VIEWS = {
    # 3 requests x 5 heads at W = 21: the group starting at request 1 puts rec_len
    # 20 bytes and the scalar gate's rec_a 210 bytes into their arrays
    "gdn_groups": SMALL["ragged_3x5"].with_(name="gdn_groups", window=21, steps=30),
    "kda_groups": SMALL["kda_small"].with_(name="kda_groups", batch=3, heads_v=5, heads_k=5, window=16,
                                           steps=24, n_comp=4, prefill=128),
}


@pytest.mark.parametrize("name", list(VIEWS))
def test_request_groups_as_state_views(name):
    """Requests split into groups [0, 1) and [1, 3), each run through views into
    the whole state (State.requests) on a stream of its own: decode outputs and
    the state after a full window's commit and a partial window are
    bit-identical to whole-batch calls."""
    wl = VIEWS[name]
    dims = H.gdims(wl)
    S = H.oracle_prefill_state(wl)
    _, tok = H.decode_tokens(wl)
    dt = H.DeviceTokens(wl, tok)
    whole = B.State.empty(dims)
    B.leapquant_quantize_state(dims, H.dev(S.transpose(0, 2, 1).astype(np.float32)), whole)
    grouped = B.State(dims, *[getattr(whole, f).clone() for f in B.FIELDS])
    groups = [(0, 1), (1, 3)]
    views = [grouped.requests(b0, b1) for b0, b1 in groups]
    streams = [torch.cuda.Stream() for _ in groups]
    o_whole = torch.empty((wl.batch, wl.heads_v, wl.dv), dtype=torch.float32, device="cuda")
    o_grp = torch.empty_like(o_whole)
    main = torch.cuda.current_stream()
    for t in range(wl.steps):
        B.leapquant_decode_step(dims, whole, *dt.step(t), o_whole)
        for s_ in streams:
            s_.wait_stream(main)
        for (b0, b1), v, s_ in zip(groups, views, streams):
            x = [a[b0:b1] for a in dt.step(t)]
            B.leapquant_decode_step(v.dims, v, *x, o_grp[b0:b1], stream=s_)
            if (t + 1) % wl.window == 0:
                B.leapquant_window_commit(v.dims, v, stream=s_)
        for s_ in streams:
            main.wait_stream(s_)
        if (t + 1) % wl.window == 0:
            B.leapquant_window_commit(dims, whole)
        assert torch.equal(o_grp, o_whole), t
    torch.cuda.synchronize()
    for f in B.FIELDS:
        assert torch.equal(getattr(grouped, f), getattr(whole, f)), f
    assert int(whole.rec_len[0, 0]) == wl.steps % wl.window
    assert B.leapquant_check_error(grouped) == 0


def test_full_window_raises_device_error_and_leaves_state():
    wl = SMALL["gdn_tiny"].with_(window=2, steps=3)
    dims = H.gdims(wl)
    cfg = H.ocfg(wl)
    S0 = H.oracle_prefill_state(wl.with_(prefill=32))
    st = B.State.empty(dims)
    rep = O.run_dense(cfg, S0, {k_: v_[:, :0] for k_, v_ in synth.tile_major(
        wl, *H.decode_tokens(wl)).items()}, snapshots=True)
    H.upload_rep(st, np.arange(wl.tiles), rep["Z"][:, 0], rep["delta"][:, 0], rep["c"][:, 0],
                 rep["Kt"][:, 0], rep["Ut"][:, 0])
    _, tok = H.decode_tokens(wl)
    dt = H.DeviceTokens(wl, tok)
    o = torch.empty((wl.tiles, 128), dtype=torch.float32, device="cuda")
    B.leapquant_decode_step(dims, st, *dt.step(0), o)
    B.leapquant_decode_step(dims, st, *dt.step(1), o)
    assert B.leapquant_check_error(st) == 0
    before = {f: getattr(st, f).clone() for f in B.FIELDS if f != "err"}
    B.leapquant_decode_step(dims, st, *dt.step(2), o)
    assert torch.isnan(o).all()
    assert B.leapquant_check_error(st) == B.LQ_DEVERR_WINDOW_FULL
    assert B.leapquant_check_error(st) == 0          # cleared
    for f, t in before.items():
        assert torch.equal(getattr(st, f), t), f


def test_corrupt_window_length_is_rejected_on_device():
    wl = SMALL["gdn_tiny"].with_(window=4)
    dims = H.gdims(wl)
    st = B.State.empty(dims)
    st.rec_len.fill_(7)
    S_out = torch.zeros((wl.tiles, 128, 128), dtype=torch.float32, device="cuda")
    B.leapquant_dequantize_state(dims, st, S_out)
    B.leapquant_window_commit(dims, st)
    assert B.leapquant_check_error(st) == B.LQ_DEVERR_BAD_REC_LEN
    assert not S_out.any() and torch.all(st.rec_len == 7)


def test_decode_is_deterministic():
    wl = SMALL["kda_small"].with_(steps=20)
    dims = H.gdims(wl)
    S0 = H.oracle_prefill_state(wl)
    _, tok = H.decode_tokens(wl)
    dt = H.DeviceTokens(wl, tok)
    res = []
    for _ in range(2):
        st = B.State.empty(dims)
        B.leapquant_quantize_state(dims, H.dev(S0.transpose(0, 2, 1).astype(np.float32)), st)
        o = torch.empty((wl.tiles, 128), dtype=torch.float32, device="cuda")
        outs = []
        for t in range(20):
            B.leapquant_decode_step(dims, st, *dt.step(t), o)
            outs.append(o.clone())
            if t == 9:
                B.leapquant_window_commit(dims, st)
        res.append((torch.stack(outs), st.codes.clone(), st.comp_u.clone(), st.rec_u.clone()))
    for a, b in zip(res[0], res[1]):
        assert torch.equal(a, b)


# --------------------------------------------------------------------------- full sizes

FULL = {
    "kda_kimi": (W_["kda_kimi"], 32, 1),
    "gdn_qwen3next_int8": (W_["gdn_qwen3next"], 32, 1),
    "gdn_qwen3next_e4m3": (W_["gdn_qwen3next"].with_(name="gdn_qwen3next_e4m3", code=synth.CODE_E4M3), 32, 1),
    "gdn_stress": (W_["gdn_stress"], 48, 2),
    "gdn_long": (W_["gdn_long"], 24, 1),
    "kda_kimi_int4": (W_["kda_kimi_int4"], 32, 1),
    "kda_kimi_int6": (W_["kda_kimi_int6"], 32, 1),
    "kda_kimi_bf16w": (W_["kda_kimi_bf16w"], 32, 1),
}


@pytest.mark.parametrize("name", list(FULL))
def test_full_size_window_parity(name):
    """Every launch at the workload's full size (all tiles, as benchmarked); the
    oracle checks a seeded tile sample (outlier tiles included where only a
    fraction has them).  gdn_long has W = 128, so its decode takes two record
    passes."""
    wl, n, windows = FULL[name]
    H.sampled_window_parity(wl, n_sample=n, n_windows=windows)


def test_full_size_bulk_quantize_parity():
    """leapquant_quantize_state over all 262144 cached states (17.2 GB fp32 in
    HBM); the oracle quantizes a seeded sample of them."""
    wl = W_["bulk_quantize"]
    dims = H.gdims(wl)
    cfg = H.ocfg(wl)
    vt = H.sample_tiles(wl, 32)
    g = torch.Generator(device="cuda")
    g.manual_seed(wl.seed)
    S = torch.randn((wl.batch, wl.heads_v, wl.dv, wl.dk), device="cuda", generator=g)
    Ss = np.stack([synth.bulk_states(wl, 1, first=int(t))[0] for t in vt])     # [n][dv][dk]
    S.view(wl.tiles, wl.dv, wl.dk)[torch.as_tensor(vt, device="cuda")] = H.dev(Ss)
    st = B.State.empty(dims)
    B.leapquant_quantize_state(dims, S, st)
    got = H.download_rep(st, vt)
    del S
    exp = {"Z": [], "delta": [], "c": [], "Kt": [], "Ut": []}
    for i in range(len(vt)):
        rep = O.quantize(cfg, Ss[i].T.astype(np.float64))
        for k_ in exp:
            exp[k_].append(getattr(rep, k_))
    exp = {k_: np.stack(v_) for k_, v_ in exp.items()}
    cr = H.compare_rep(cfg, got, exp, wl.code)
    H.log(f"[bulk_quantize] full size: {cr}")
    assert cr["code_eq"] >= 0.999 and cr["code_maxdiff"] <= 1, cr
    assert cr["deq_rel"] <= 1e-3 and cr.get("comp_rel", 0.0) <= 1e-3, cr
    assert cr["delta_rel"] <= 1e-5 and cr["c_rel"] <= 1e-5, cr
    assert np.all(got["rec_len"] == 0)
