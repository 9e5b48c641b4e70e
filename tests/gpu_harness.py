"""Shared machinery of the GPU parity tests.

The HIP path (through the C ABI) and the CPU oracle are fed the same seeded
synthetic inputs.  Nothing computed on the GPU is ever handed to the oracle:
where a test starts the GPU from a given representation, that representation
is the oracle's (or the generator's).  Layout conversions only: the oracle
stores a tile as S[k][v], the library as S^T[v][k].
"""
from __future__ import annotations

import sys
import time

import numpy as np
import torch

from oracle import oracle as O
from paper_2609_38166_amd import binding as B
from paper_2609_38166_amd import synth


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to("cuda")


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def rel_rows(a, b):
    """Max over leading indices of the relative L2 error of the last axis."""
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    num = np.linalg.norm(a - b, axis=-1)
    den = np.maximum(np.linalg.norm(b, axis=-1), 1e-300)
    return float(np.max(num / den))


def f16_bits(x):
    return np.asarray(x, np.float64).astype(np.float16).view(np.uint16)


def f16_vals(bits):
    return np.asarray(bits, np.uint16).view(np.float16).astype(np.float64)


def ocfg(wl: synth.Workload, **kw) -> O.Cfg:
    args = dict(dk=wl.dk, dv=wl.dv, window=wl.window, n_comp=wl.n_comp,
                power_iters=wl.power_iters, gate=wl.gate, code=wl.code, smooth=wl.smooth,
                rule=wl.rule)
    args.update(kw)
    return O.make_cfg(**args)


def gdims(wl: synth.Workload, **kw) -> B.lq_dims:
    args = dict(window=wl.window, n_comp=wl.n_comp, power_iters=wl.power_iters, gate=wl.gate,
                code=wl.code, smooth=wl.smooth, d_k=wl.dk, d_v=wl.dv, rule=wl.rule)
    args.update(kw)
    return B.make_dims(wl.batch, wl.heads_v, wl.heads_k, **args)


# --------------------------------------------------------------------------- codes

def code_ordinal(Z, code):
    """Position of each code on the ordered grid of representable values."""
    if code == synth.CODE_BF16:
        b = np.asarray(Z, np.uint16).astype(np.int64)
        mag = b & 0x7FFF
        return np.where(b & 0x8000, -mag, mag)
    Z = np.asarray(Z, np.uint8)
    if code != synth.CODE_E4M3:
        return Z.view(np.int8).astype(np.int64)
    mag = (Z & 0x7F).astype(np.int64)
    return np.where(Z & 0x80, -mag, mag)


def code_agreement(Zg, Zo, code):
    """(fraction equal, max distance on the code grid)."""
    a, b = code_ordinal(Zg, code), code_ordinal(Zo, code)
    d = np.abs(a - b)
    return float(np.mean(d == 0)), int(d.max()) if d.size else 0


# --------------------------------------------------------------------------- representation I/O

CODE_BITS = {synth.CODE_INT8: 8, synth.CODE_E4M3: 8, synth.CODE_INT4: 4, synth.CODE_INT6: 6, synth.CODE_BF16: 16}


def pack_codes(Zt, code):
    """[n][rows][128] code bytes (one code per byte, two's complement for the
    integer formats) to the library's row layout: INT4 two per byte (even
    channel low), INT6 four per three bytes (channel 4i+q at bits 6q of the
    little-endian 24-bit group i).  The BF16 state: its 16-bit values as bytes."""
    if code == synth.CODE_BF16:
        return np.ascontiguousarray(np.asarray(Zt, np.uint16)).view(np.uint8)
    Zt = np.asarray(Zt, np.uint8)
    if CODE_BITS[code] == 8:
        return Zt
    c = Zt.astype(np.uint32)
    if code == synth.CODE_INT4:
        c = c & 0xF
        return (c[..., 0::2] | (c[..., 1::2] << 4)).astype(np.uint8)
    c = c & 0x3F
    g = c[..., 0::4] | (c[..., 1::4] << 6) | (c[..., 2::4] << 12) | (c[..., 3::4] << 18)
    out = np.empty(Zt.shape[:-1] + (Zt.shape[-1] * 3 // 4,), np.uint8)
    out[..., 0::3], out[..., 1::3], out[..., 2::3] = g & 0xFF, (g >> 8) & 0xFF, (g >> 16) & 0xFF
    return out


def unpack_codes(P, code, n_ch=128):
    """Inverse of pack_codes: one two's-complement code per byte (BF16 bits for
    the BF16 state)."""
    if code == synth.CODE_BF16:
        return np.ascontiguousarray(np.asarray(P, np.uint8)).view(np.uint16)
    P = np.asarray(P, np.uint8)
    if CODE_BITS[code] == 8:
        return P
    out = np.empty(P.shape[:-1] + (n_ch,), np.int64)
    p = P.astype(np.int64)
    if code == synth.CODE_INT4:
        lo, hi = p & 0xF, p >> 4
        out[..., 0::2], out[..., 1::2] = lo, hi
        out = np.where(out >= 8, out - 16, out)
    else:
        g = p[..., 0::3] | (p[..., 1::3] << 8) | (p[..., 2::3] << 16)
        for q in range(4):
            out[..., q::4] = (g >> (6 * q)) & 0x3F
        out = np.where(out >= 32, out - 64, out)
    return out.astype(np.int8).view(np.uint8)


def upload_rep(st: B.State, idx, Z, delta, c, Kt, Ut):
    """Write oracle-layout representations of tiles `idx` into the GPU state and
    open an empty window."""
    dims = st.dims
    n, dk, dv, r = len(idx), dims.d_k, dims.d_v, dims.n_comp
    idx_t = torch.as_tensor(np.asarray(idx, np.int64), device="cuda")
    rowb = dk * CODE_BITS[dims.code] // 8
    st.codes.view(-1, dv, rowb)[idx_t] = dev(pack_codes(np.asarray(Z).transpose(0, 2, 1), dims.code))
    st.scale.view(-1, dv)[idx_t] = dev(np.asarray(delta, np.float32))
    st.smooth.view(-1, dk)[idx_t] = dev(np.asarray(c, np.float32))
    if r:
        st.comp_k.view(-1, r, dk)[idx_t] = dev(np.asarray(Kt, np.float64).astype(np.float16))
        st.comp_u.view(-1, r, dv)[idx_t] = dev(np.asarray(Ut, np.float64).astype(np.float16))
    st.rec_len.view(-1)[idx_t] = 0


def download_rep(st: B.State, idx=None) -> dict:
    dims = st.dims
    dk, dv, r = dims.d_k, dims.d_v, dims.n_comp
    sl = slice(None) if idx is None else torch.as_tensor(np.asarray(idx, np.int64), device="cuda")
    out = {
        "Z": unpack_codes(st.codes.view(-1, dv, dk * CODE_BITS[dims.code] // 8)[sl].cpu().numpy(),
                          dims.code, dk).transpose(0, 2, 1).copy(),
        "delta": st.scale.view(-1, dv)[sl].cpu().numpy(),
        "c": st.smooth.view(-1, dk)[sl].cpu().numpy(),
        "rec_len": st.rec_len.view(-1)[sl].cpu().numpy(),
    }
    if r:
        out["Kt"] = st.comp_k.view(-1, r, dk)[sl].cpu().numpy().astype(np.float64)
        out["Ut"] = st.comp_u.view(-1, r, dv)[sl].cpu().numpy().astype(np.float64)
    else:
        out["Kt"] = np.zeros((out["Z"].shape[0], 0, dk))
        out["Ut"] = np.zeros((out["Z"].shape[0], 0, dv))
    return out


def dequant_oracle(cfg, rep: dict) -> np.ndarray:
    """Oracle dequantization of a batch of representations (oracle layout)."""
    n = rep["Z"].shape[0]
    return np.stack([O.dequantize(cfg, O.Rep(rep["Z"][i], rep["delta"][i], rep["c"][i],
                                             rep["Kt"][i], rep["Ut"][i])) for i in range(n)])


def compare_rep(cfg, got: dict, exp: dict, code) -> dict:
    """Agreement of two batches of representations (both oracle layout)."""
    eq, md = code_agreement(got["Z"], exp["Z"], code)
    out = {"code_eq": eq, "code_maxdiff": md,
           "delta_rel": float(np.max(np.abs(got["delta"] - exp["delta"]) /
                                     np.maximum(np.abs(exp["delta"]), 1e-30))),
           "c_rel": float(np.max(np.abs(got["c"] - exp["c"]) / np.maximum(np.abs(exp["c"]), 1e-30))),
           "deq_rel": rel_rows(dequant_oracle(cfg, got).reshape(len(got["Z"]), -1),
                               dequant_oracle(cfg, exp).reshape(len(exp["Z"]), -1))}
    if got["Kt"].shape[1]:
        pg = np.einsum("nrk,nrv->nkv", got["Kt"], got["Ut"]).reshape(len(got["Z"]), -1)
        pe = np.einsum("nrk,nrv->nkv", exp["Kt"], exp["Ut"]).reshape(len(exp["Z"]), -1)
        out["comp_rel"] = rel_rows(pg, pe)
    return out


# --------------------------------------------------------------------------- workload inputs

def oracle_prefill_state(wl: synth.Workload, vtiles=None, threads=None) -> np.ndarray:
    """Initial fp32 states (oracle layout [tiles][dk][dv]): the unquantized fp32
    recurrence over `prefill` tokens from zero, then the outlier lines."""
    st = synth.Streams(wl, synth.PHASE_PREFILL, vtiles)
    tok = synth.tile_major(wl, st, st.draw(wl.prefill))
    st.close()
    n = len(st.vtiles)
    cfg = ocfg(wl)
    _, Sp = O.run_baseline(cfg, np.zeros((n, wl.dk, wl.dv)), tok, mode=O.STATE_F32, threads=threads,
                           want_o=False)
    F = synth.outlier_factor(synth.outliers(wl, st.vtiles))
    return (Sp.astype(np.float32) * F).astype(np.float64)


def decode_tokens(wl: synth.Workload, vtiles=None, n=None):
    st = synth.Streams(wl, synth.PHASE_DECODE, vtiles)
    tok = st.draw(wl.steps if n is None else n)
    st.close()
    return st, tok


class DeviceTokens:
    """Step-major device copies of a full-batch token stream."""

    def __init__(self, wl: synth.Workload, tok: dict):
        sm = synth.step_major_full(wl, tok)
        self.q, self.k, self.v = dev(sm["q"]), dev(sm["k"]), dev(sm["v"])
        self.alpha, self.beta = dev(sm["alpha"]), dev(sm["beta"])
        self.T = sm["v"].shape[0]

    def step(self, t):
        return self.q[t], self.k[t], self.v[t], self.alpha[t], self.beta[t]


# --------------------------------------------------------------------------- the parity protocol

def _f16_ulp_dist(a_bits, b_bits):
    """Distance in units of the last place between fp16 bit patterns."""
    def ordinal(b):
        b = np.asarray(b, np.int64)
        mag = b & 0x7FFF
        return np.where(b & 0x8000, -mag, mag)
    return np.abs(ordinal(a_bits) - ordinal(b_bits))


def upload_records(st: B.State, hist_a, hist_k, hist_u, idx=None):
    """Write [tiles][n][...] record values (FP16-representable) into the open
    window of tiles `idx` (default: every tile) and set their rec_len = n."""
    n = hist_a.shape[1]
    dims = st.dims
    t = dims.batch * dims.heads_v
    W, g = dims.window, (dims.d_k if dims.gate == B.LQ_GATE_DIAG else 1)
    sel = slice(None) if idx is None else torch.as_tensor(np.asarray(idx, np.int64), device="cuda")
    ra, rk, ru = st.rec_a.view(t, W, g), st.rec_k.view(t, W, dims.d_k), st.rec_u.view(t, W, dims.d_v)
    ra[sel, :n] = dev(np.asarray(hist_a).astype(np.float16))
    rk[sel, :n] = dev(np.asarray(hist_k).astype(np.float16))
    ru[sel, :n] = dev(np.asarray(hist_u).astype(np.float16))
    st.rec_len.view(-1)[sel] = n


def quant_noise(cfg, start, exp, hist_a, hist_k, hist_u) -> np.ndarray:
    """Per tile: the oracle's own quantization error at a window end,
    |dequant(Q(S_p)) - S_p| / |S_p|, with S_p reconstructed from the
    window-start representation and the records (Sec. 3.4 Eq. (smooth))."""
    out = []
    for i in range(len(exp["Z"])):
        rep0 = O.Rep(*(start[k_][i] for k_ in ("Z", "delta", "c", "Kt", "Ut")))
        rep1 = O.Rep(*(exp[k_][i] for k_ in ("Z", "delta", "c", "Kt", "Ut")))
        Sp = O.reconstruct(cfg, rep0, None, hist_a[i], hist_k[i], hist_u[i])
        out.append(rel(O.dequantize(cfg, rep1), Sp))
    return np.asarray(out)


def chained_ratio(cfg, got, exp, noise) -> float:
    """Largest per-tile distance between the GPU's commit of its own records and
    the oracle's commit, in units of the oracle's own quantization error."""
    dg = dequant_oracle(cfg, got).reshape(len(got["Z"]), -1)
    de = dequant_oracle(cfg, exp).reshape(len(exp["Z"]), -1)
    d = np.linalg.norm(dg - de, axis=1) / np.maximum(np.linalg.norm(de, axis=1), 1e-300)
    return float(np.max(d / np.maximum(noise, 1e-300)))


def window_sync_parity(wl: synth.Workload, n_windows=None, check=True):
    """Window-by-window parity on every tile of a (small) workload.

    The oracle runs the whole trajectory in dense form.  For each window:
      decode  -- the GPU starts from the oracle's window-start representation
                 and runs the W decode steps itself; its outputs and FP16
                 records are compared with the oracle's;
      commit  -- teacher-forced: the GPU commits the oracle's window-start
                 representation plus the oracle's records (the gate on codes);
      chained -- the GPU commits its own records from the decode pass (the
                 path the library runs), gated at the same bars.
    Nothing from the GPU is handed to the oracle.
    """
    cfg = ocfg(wl)
    dims = gdims(wl)
    t0 = time.time()
    S0 = oracle_prefill_state(wl)
    streams, tok = decode_tokens(wl)
    T = wl.steps if n_windows is None else min(wl.steps, n_windows * wl.window)
    otok = synth.tile_major(wl, streams, tok)
    otok = {k_: v_[:, :T] for k_, v_ in otok.items()}
    ref = O.run_dense(cfg, S0, otok, snapshots=True, history=True)
    log(f"[{wl.name}] oracle {time.time() - t0:.1f}s tiles={wl.tiles} T={T}")
    dt = DeviceTokens(wl, {k_: v_[:T] for k_, v_ in tok.items()})

    def decode(st, t, o):
        B.leapquant_decode_step(dims, st, *dt.step(t), o)

    return window_protocol(wl.name, cfg, dims, ref, T, decode, check)


def window_protocol(name, cfg, dims, ref, T, decode, check=True, sample=None, fill=None):
    """The per-window checks of window_sync_parity, for an oracle trajectory
    `ref` (run_dense with snapshots and history) over T steps; decode(st, t, o)
    issues the GPU's step t into o [batch][heads_v][d_v].  With `sample` (tile
    indices) the oracle covers those tiles only: every launch still covers all
    tiles, fill(st) first gives the others a valid representation, and only the
    sample is compared."""
    n_tiles = dims.batch * dims.heads_v
    dk, dv, W, code = dims.d_k, dims.d_v, dims.window, dims.code
    g = dk if dims.gate == B.LQ_GATE_DIAG else 1
    st = B.State.empty(dims)
    if fill is not None:
        fill(st)
    o = torch.empty((dims.batch, dims.heads_v, dv), dtype=torch.float32, device="cuda")
    vt = np.arange(n_tiles) if sample is None else np.asarray(sample, np.int64)
    idx = None if sample is None else vt
    vt_t = torch.as_tensor(vt, device="cuda")
    agg = {"o_rel": 0.0, "u_eq": [], "k_eq": [], "a_eq": [], "rec_ulp": 0, "u_rel": 0.0}
    tf = {"code_eq": [], "code_maxdiff": 0, "deq_rel": 0.0, "comp_rel": 0.0, "delta_rel": 0.0,
          "c_rel": 0.0}
    ch = {"code_eq": [], "code_maxdiff": 0, "deq_rel": 0.0, "comp_rel": 0.0, "ratio": 0.0, "noise": 0.0}
    for w in range(T // W):
        sl = slice(w * W, (w + 1) * W)
        exp = {k_: ref[k_][:, w + 1] for k_ in ("Z", "delta", "c", "Kt", "Ut")}
        start = [ref[k_][:, w] for k_ in ("Z", "delta", "c", "Kt", "Ut")]
        upload_rep(st, vt, *start)
        outs = []
        for j in range(W):
            decode(st, w * W + j, o)
            outs.append(o.view(n_tiles, dv)[vt_t].cpu().numpy())
        og = np.stack(outs, axis=1)
        agg["o_rel"] = max(agg["o_rel"], rel_rows(og, ref["o"][:, sl]))
        ru = st.rec_u.view(n_tiles, W, dv)[vt_t].cpu().numpy().view(np.uint16)
        rk = st.rec_k.view(n_tiles, W, dk)[vt_t].cpu().numpy().view(np.uint16)
        ra = st.rec_a.view(n_tiles, W, g)[vt_t].cpu().numpy().view(np.uint16)
        eu, ek, ea = f16_bits(ref["hist_u"][:, sl]), f16_bits(ref["hist_k"][:, sl]), f16_bits(ref["hist_a"][:, sl])
        agg["u_eq"].append(np.mean(ru == eu))
        agg["k_eq"].append(np.mean(rk == ek))
        agg["a_eq"].append(np.mean(ra == ea))
        # a record that rounds differently may differ by one unit in its last place
        agg["rec_ulp"] = max(agg["rec_ulp"], int(_f16_ulp_dist(rk, ek).max()),
                             int(_f16_ulp_dist(ru, eu).max()))
        agg["u_rel"] = max(agg["u_rel"], rel_rows(f16_vals(ru), ref["hist_u"][:, sl]))
        # chained commit of the GPU's own records (every tile)
        B.leapquant_window_commit(dims, st, None)
        got = download_rep(st, idx)
        assert np.all(st.rec_len.cpu().numpy() == 0)
        cr = compare_rep(cfg, got, exp, code)
        ch["code_eq"].append(cr["code_eq"])
        ch["code_maxdiff"] = max(ch["code_maxdiff"], cr["code_maxdiff"])
        ch["deq_rel"] = max(ch["deq_rel"], cr["deq_rel"])
        ch["comp_rel"] = max(ch["comp_rel"], cr.get("comp_rel", 0.0))
        noise = quant_noise(cfg, {k_: ref[k_][:, w] for k_ in ("Z", "delta", "c", "Kt", "Ut")}, exp,
                            ref["hist_a"][:, sl], ref["hist_k"][:, sl], ref["hist_u"][:, sl])
        ch["ratio"] = max(ch["ratio"], chained_ratio(cfg, got, exp, noise))
        ch["noise"] = max(ch["noise"], float(noise.max()))
        # teacher-forced commit of the oracle's records
        upload_rep(st, vt, *start)
        upload_records(st, ref["hist_a"][:, sl], ref["hist_k"][:, sl], ref["hist_u"][:, sl], idx=idx)
        B.leapquant_window_commit(dims, st, None)
        got = download_rep(st, idx)
        cr = compare_rep(cfg, got, exp, code)
        tf["code_eq"].append(cr["code_eq"])
        tf["code_maxdiff"] = max(tf["code_maxdiff"], cr["code_maxdiff"])
        for k_ in ("deq_rel", "comp_rel", "delta_rel", "c_rel"):
            tf[k_] = max(tf[k_], cr.get(k_, 0.0))
    bits = B.leapquant_check_error(st)
    summary = {
        "o_rel": agg["o_rel"], "u_eq": float(np.min(agg["u_eq"])), "k_eq": float(np.min(agg["k_eq"])),
        "a_eq": float(np.min(agg["a_eq"])), "rec_ulp": agg["rec_ulp"], "u_rel": agg["u_rel"],
        "tf_code_eq": float(np.mean(tf["code_eq"])), "tf_code_eq_min": float(np.min(tf["code_eq"])),
        "tf_code_maxdiff": tf["code_maxdiff"], "tf_deq_rel": tf["deq_rel"],
        "tf_comp_rel": tf["comp_rel"], "tf_delta_rel": tf["delta_rel"], "tf_c_rel": tf["c_rel"],
        "ch_code_eq": float(np.mean(ch["code_eq"])), "ch_code_maxdiff": ch["code_maxdiff"],
        "ch_deq_rel": ch["deq_rel"], "ch_comp_rel": ch["comp_rel"],
        "ch_ratio": ch["ratio"], "q_noise": ch["noise"], "err_bits": bits,
    }
    log(f"[{name}] {summary}")
    if check:
        assert bits == 0, summary
        assert summary["o_rel"] <= 1e-3, summary
        assert summary["a_eq"] == 1.0 and summary["k_eq"] >= 0.999, summary
        assert summary["u_eq"] >= 0.999 and summary["u_rel"] <= 1e-3, summary
        assert summary["rec_ulp"] <= 1, summary
        assert summary["tf_code_eq"] >= 0.999 and summary["tf_code_maxdiff"] <= 1, summary
        assert summary["tf_deq_rel"] <= 1e-3 and summary["tf_comp_rel"] <= 1e-3, summary
        assert summary["tf_delta_rel"] <= 1e-5 and summary["tf_c_rel"] <= 1e-5, summary
        # chained commit (the product path: the GPU commits its own records) at
        # the same bars as the teacher-forced one
        assert summary["ch_code_eq"] >= 0.999 and summary["ch_code_maxdiff"] <= 1, summary
        assert summary["ch_deq_rel"] <= 1e-3 and summary["ch_comp_rel"] <= 1e-3, summary
    return summary


# --------------------------------------------------------------------------- full-size launches

def sample_tiles(wl: synth.Workload, n: int, salt: int = 0) -> np.ndarray:
    """A seeded sample of n tile indices; for workloads whose outliers sit in a
    fraction of the tiles, half of the sample is drawn from those tiles."""
    if n >= wl.tiles:
        return np.arange(wl.tiles)
    rng = np.random.default_rng([wl.seed, 77, salt])
    pick = set()
    if wl.outliers == "frac":
        hot = np.nonzero((synth.outliers(wl)["row_f"] > 1.0).any(axis=1))[0]
        pick.update(rng.choice(hot, min(n // 2, len(hot)), replace=False).tolist())
    rest = np.setdiff1d(np.arange(wl.tiles), np.fromiter(pick, np.int64, len(pick)))
    pick.update(rng.choice(rest, n - len(pick), replace=False).tolist())
    return np.sort(np.fromiter(pick, np.int64, len(pick)))


def filler_state(st: B.State, wl: synth.Workload):
    """Valid representations for the tiles no oracle looks at: a random fp32
    state quantized on the GPU (their values never reach a comparison)."""
    g = torch.Generator(device="cuda")
    g.manual_seed(wl.seed)
    S = torch.randn((wl.batch, wl.heads_v, wl.dv, wl.dk), device="cuda", generator=g)
    S *= 0.1
    B.leapquant_quantize_state(st.dims, S, st)
    torch.cuda.synchronize()
    del S


def sampled_window_parity(wl: synth.Workload, n_sample=32, n_windows=1, check=True):
    """Window-synchronised parity at the workload's full size: every launch
    covers all tiles (the launch configuration of the benchmark), and a seeded
    sample of tiles is compared with the oracle, which runs those tiles only
    (tiles are independent).  Same protocol and bars as window_sync_parity."""
    cfg = ocfg(wl)
    dims = gdims(wl)
    t0 = time.time()
    vt = sample_tiles(wl, n_sample)
    T = min(wl.steps, n_windows * wl.window)
    S0 = oracle_prefill_state(wl, vtiles=vt)
    ost = synth.Streams(wl, synth.PHASE_DECODE, vt)
    otok = synth.tile_major(wl, ost, ost.draw(T))
    ost.close()
    ref = O.run_dense(cfg, S0, otok, snapshots=True, history=True)
    log(f"[{wl.name}] oracle {time.time() - t0:.1f}s on {len(vt)} of {wl.tiles} tiles, T={T}")
    fst = synth.Streams(wl, synth.PHASE_DECODE)
    dt = DeviceTokens(wl, fst.draw(T))
    fst.close()
    log(f"[{wl.name}] full-batch tokens on device {time.time() - t0:.1f}s")

    def decode(st, t, o):
        B.leapquant_decode_step(dims, st, *dt.step(t), o)

    return window_protocol(f"{wl.name} full size", cfg, dims, ref, T, decode, check, sample=vt,
                           fill=lambda st: filler_state(st, wl))
