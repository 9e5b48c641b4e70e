"""Throughput of the LeapQuant 8-bit decode path on one MI355X.

One benchmark step is one pass of the whole hot path over one batch: the
window-start quantization of the prefill state (leapquant_quantize_state),
then T decode tokens (one leapquant_decode_step launch per token over every
(request, head) tile) with a leapquant_window_commit after every W tokens.
The metric is token-head decode steps per second (tiles x T / time), reported
with the effective HBM bandwidth of the algorithmic bytes, its fraction of the
8 TB/s peak, and the speedup over the per-step bf16 and fp32 dense-state
baselines run on the same tokens.

Inputs are synthetic and seeded (paper_2609_38166_amd.synth): they are
generated on the host, copied to HBM before the timed region, and the initial
state is built on the GPU by an fp32 prefill recurrence plus outlier lines.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="kda_kimi")
    ap.add_argument("--no-graph", action="store_true", help="launch eagerly instead of replaying a HIP graph")
    ap.add_argument("--no-baselines", action="store_true")
    ap.add_argument("--sweep", action="store_true",
                    help="kernel-speed sweep mirroring the paper's ablations (GDN, batch 256): "
                         "per-step vs per-window codes, Compensator Tokens, smoothing, window and "
                         "token counts; one JSON line per configuration")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the 6- and 4-bit code variants of the headline layer")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-tiles", type=int, default=8192)
    ap.add_argument("--profile", action="store_true",
                    help="short run for profilers: setup, warmup and the timed steps only")
    ap.add_argument("--long-trace", action="store_true",
                    help="long-trace drift of the quantized GDN trajectory from the fp32 one (32 x 16 tiles, "
                         "32768 tokens, W = 128, r = 8), every 1024 tokens; one JSON line")
    ap.add_argument("--gate-scale", type=float, default=0.1,
                    help="decay = exp(-s softplus(N(0,1))) for --long-trace (0.1: the workload's gates; "
                         "0.001: a long-memory variant)")
    ap.add_argument("--commit-split", action="store_true",
                    help="commit and quantize launch times on the KDA workload for r = 0, 4, 8 and 1, 2, 4 power "
                         "sweeps, and the split of the commit into base, per-token and per-sweep costs; one JSON line")
    ap.add_argument("--profile-decode", action="store_true",
                    help="short run for profilers: setup, then the decode with rotating batches (the "
                         "roofline timing), eight steps of each dense baseline and one device copy for "
                         "calibrating byte counters")
    return ap.parse_args()


# ----------------------------------------------------------------------------- bytes

def rec_bytes(wl):
    return 2 * (wl.dk + wl.dv) + 2 * wl.g          # FP16 key, correction, decay


CODE_BITS = {0: 8, 1: 8, 2: 4, 3: 6, 4: 16}


def scale_bytes(wl):
    """Row scales and smoothing; the BF16 state (code 4) has none."""
    return 0 if wl.code == 4 else 4 * (wl.dk + wl.dv)


def code_bytes(wl):
    return wl.dk * wl.dv * CODE_BITS[wl.code] // 8


def decode_bytes(wl, i):
    """Algorithmic bytes of one tile's decode at window position i (1-based)."""
    inputs = 4 * (2 * wl.dk) * wl.heads_k / wl.heads_v + 4 * wl.dv + 4 * wl.g + 4
    return (code_bytes(wl) + scale_bytes(wl) + 2 * wl.n_comp * (wl.dk + wl.dv)
            + (i - 1) * rec_bytes(wl) + rec_bytes(wl) + inputs + 4 * wl.dv + 8)


def rep_bytes(wl):
    return code_bytes(wl) + scale_bytes(wl) + 2 * wl.n_comp * (wl.dk + wl.dv)


def commit_bytes(wl, p):
    return rep_bytes(wl) + p * rec_bytes(wl) + rep_bytes(wl) + 8


def quantize_bytes(wl):
    return 4 * wl.dk * wl.dv + rep_bytes(wl) + 4


def baseline_bytes(wl, width):
    inputs = 4 * (2 * wl.dk) * wl.heads_k / wl.heads_v + 4 * wl.dv + 4 * wl.g + 4
    return 2 * width * wl.dk * wl.dv + inputs + 4 * wl.dv


# ----------------------------------------------------------------------------- setup

def device_tokens(wl, phase, T, chunk=64):
    """Step-major device tensors of T tokens, generated in chunks on the host."""
    import torch
    from paper_2609_38166_amd import synth
    B, Hv, Hk = wl.batch, wl.heads_v, wl.heads_k
    q = torch.empty((T, B, Hk, wl.dk), dtype=torch.float32, device="cuda")
    k = torch.empty_like(q)
    v = torch.empty((T, B, Hv, wl.dv), dtype=torch.float32, device="cuda")
    a = torch.empty((T, B, Hv, wl.dk) if wl.gate == synth.GATE_DIAG else (T, B, Hv),
                    dtype=torch.float32, device="cuda")
    b = torch.empty((T, B, Hv), dtype=torch.float32, device="cuda")
    st = synth.Streams(wl, phase)
    for t0 in range(0, T, chunk):
        n = min(chunk, T - t0)
        sm = synth.step_major_full(wl, st.draw(n))
        for dst, key in ((q, "q"), (k, "k"), (v, "v"), (a, "alpha"), (b, "beta")):
            dst[t0:t0 + n].copy_(torch.from_numpy(sm[key]))
    st.close()
    return q, k, v, a, b


def prefill_state(wl, dims):
    """Initial states S^T [B][Hv][dv][dk]: fp32 prefill on the GPU, then outliers."""
    import torch
    from paper_2609_38166_amd import binding as B_, synth
    S = torch.zeros((wl.batch, wl.heads_v, wl.dv, wl.dk), dtype=torch.float32, device="cuda")
    o = torch.empty((wl.batch, wl.heads_v, wl.dv), dtype=torch.float32, device="cuda")
    st = synth.Streams(wl, synth.PHASE_PREFILL)
    chunk = 64
    for t0 in range(0, wl.prefill, chunk):
        n = min(chunk, wl.prefill - t0)
        sm = synth.step_major_full(wl, st.draw(n))
        dev = {kk: torch.from_numpy(vv).cuda() for kk, vv in sm.items()}
        for t in range(n):
            B_.leapquant_baseline_step(dims, S, B_.LQ_STATE_F32, dev["q"][t], dev["k"][t],
                                       dev["v"][t], dev["alpha"][t], dev["beta"][t], o)
    st.close()
    out = synth.outliers(wl)
    rf = torch.from_numpy(out["row_f"]).cuda().view(wl.batch, wl.heads_v, 1, wl.dk)
    cf = torch.from_numpy(out["col_f"]).cuda().view(wl.batch, wl.heads_v, wl.dv, 1)
    S *= torch.maximum(rf, cf)
    torch.cuda.synchronize()
    return S


# ----------------------------------------------------------------------------- timing

class Runner:
    def __init__(self, wl, dims, S0, toks, use_graph):
        import torch
        from paper_2609_38166_amd import binding as B_
        self.wl, self.dims, self.S0, self.toks = wl, dims, S0, toks
        self.B_ = B_
        self.st = B_.State.empty(dims)
        self.o = torch.empty((wl.batch, wl.heads_v, wl.dv), dtype=torch.float32, device="cuda")
        self.graph = None
        if use_graph:
            self._capture()

    def _calls(self):
        """Prepared launches of one step on the current stream."""
        B_, wl, d, st = self.B_, self.wl, self.dims, self.st
        q, k, v, a, b = self.toks
        calls = []
        s = st.struct()
        self._keep = [s]
        L = B_.lib()
        import ctypes as C
        stream = B_._stream(None)
        calls.append(B_.Prepared(L.leapquant_quantize_state, C.byref(d), self.S0.data_ptr(),
                                 C.byref(s), stream))
        for t in range(wl.steps):
            calls.append(B_.Prepared(L.leapquant_decode_step, C.byref(d), C.byref(s), q[t].data_ptr(),
                                     k[t].data_ptr(), v[t].data_ptr(), a[t].data_ptr(),
                                     b[t].data_ptr(), self.o.data_ptr(), stream))
            if (t + 1) % wl.window == 0:
                calls.append(B_.Prepared(L.leapquant_window_commit, C.byref(d), C.byref(s), None,
                                         stream))
        return calls

    def _capture(self):
        import torch
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for c in self._calls():     # one eager pass on the capture stream first
                c()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            for c in self._calls():
                c()
        torch.cuda.synchronize()

    def step(self):
        if self.graph is not None:
            self.graph.replay()
        else:
            for c in self._calls_cache():
                c()

    def _calls_cache(self):
        if not hasattr(self, "_cc"):
            self._cc = self._calls()
        return self._cc


def time_steps(fn, steps, warmup):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return e0.elapsed_time(e1) / 1e3, wall


def per_launch_times(wl, dims, S0, toks, reps=3):
    """Average kernel durations, measured with HIP events on the stream the
    kernels run on: the decode launches of one whole window (positions 1..W)
    replayed as one graph, divided by W; the commit that ends the window; the
    window-start quantization.  toks = (q, k, v, alpha, beta), or (q, k, b, v,
    alpha, beta) for the general rule (read vectors b given)."""
    import torch
    from paper_2609_38166_amd import binding as B_
    st = B_.State.empty(dims)
    o = torch.empty((wl.batch, wl.heads_v, wl.dv), dtype=torch.float32, device="cuda")
    W = wl.window

    def window():
        for i in range(W):
            if len(toks) == 6:
                B_.leapquant_decode_step_general(dims, st, *(t_[i] for t_ in toks), o)
            else:
                B_.leapquant_decode_step(dims, st, *(t_[i] for t_ in toks), o)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        B_.leapquant_quantize_state(dims, S0, st)
        window()
        B_.leapquant_window_commit(dims, st)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        window()
    torch.cuda.synchronize()

    def ev():
        return torch.cuda.Event(enable_timing=True)
    res = {"decode": [], "commit": [], "quantize": []}
    for rep in range(reps + 1):
        e = [ev() for _ in range(6)]
        e[0].record()
        B_.leapquant_quantize_state(dims, S0, st)
        e[1].record()
        e[2].record()
        g.replay()
        e[3].record()
        e[4].record()
        B_.leapquant_window_commit(dims, st)
        e[5].record()
        torch.cuda.synchronize()
        if rep == 0:
            continue                      # first pass warms caches and clocks
        res["quantize"].append(e[0].elapsed_time(e[1]))
        res["decode"].append(e[2].elapsed_time(e[3]) / W)
        res["commit"].append(e[4].elapsed_time(e[5]))
    bits = B_.leapquant_check_error(st)
    if bits:
        raise RuntimeError(f"device error bits {bits} during the per-launch timing")
    return {k_: float(np.mean(v_)) for k_, v_ in (("decode_ms", res["decode"]),
                                                   ("commit_ms", res["commit"]),
                                                   ("quantize_ms", res["quantize"]))}


def rwkv7_tokens(wl, n_sub, seed):
    """Step-major device inputs of n_sub / 2 RWKV7 tokens as general-rule
    sub-steps (q, k, b, v, alpha, beta): an erase with alpha = w, k = kappa,
    b = a . kappa, v = 0, then a write with alpha = 1, k = k, b = 0, v = v; both
    take the receptance r as query and beta = 1.  Drawn on the device:
    w = exp(-e^-0.5 sigmoid(z)), a = sigmoid(z), kappa, k, r unit-norm
    Gaussian, v ~ N(0, I)."""
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    n = n_sub // 2
    shp = (n, wl.batch, wl.heads_v, wl.dk)

    def rnd(shape=shp):
        return torch.randn(shape, generator=g, device="cuda")

    def unit():
        x = rnd()
        return x / x.norm(dim=-1, keepdim=True)

    def inter(x0, x1):
        out = torch.empty((2 * n,) + tuple(x0.shape[1:]), device="cuda")
        out[0::2], out[1::2] = x0, x1
        return out

    w = torch.exp(-np.exp(-0.5) * torch.sigmoid(rnd()))
    a = torch.sigmoid(rnd())
    kap, k, r = unit(), unit(), unit()
    v = rnd((n, wl.batch, wl.heads_v, wl.dv))
    zero = torch.zeros(shp, device="cuda")
    toks = (inter(r, r), inter(kap, k), inter(a * kap, zero), inter(torch.zeros_like(v), v),
            inter(w, torch.ones(shp, device="cuda")), torch.ones((2 * n, wl.batch, wl.heads_v), device="cuda"))
    return tuple(t_.contiguous() for t_ in toks)


def bulk_quantize(reps=3):
    """leapquant_quantize_state over the bulk prefix-cache workload: 8192
    cached requests x 32 heads (262144 fp32 states, 17.2 GB resident in HBM),
    r = 8.  Returns ms per pass and GB/s of fp32 state read.  The states are
    drawn on the device (N(0, 1)); the kernel's work does not depend on the
    values."""
    import torch
    from paper_2609_38166_amd import binding as B_, synth
    wl = synth.WORKLOADS["bulk_quantize"]
    dims = B_.make_dims(wl.batch, wl.heads_v, wl.heads_k, window=wl.window, n_comp=wl.n_comp,
                        power_iters=wl.power_iters, gate=wl.gate, code=wl.code)
    g = torch.Generator(device="cuda")
    g.manual_seed(wl.seed)
    S = torch.randn((wl.batch, wl.heads_v, wl.dv, wl.dk), dtype=torch.float32, device="cuda", generator=g)
    st = B_.State.empty(dims)
    B_.leapquant_quantize_state(dims, S, st)
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        B_.leapquant_quantize_state(dims, S, st)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    if B_.leapquant_check_error(st):
        raise RuntimeError("device error during the bulk quantization")
    ms = float(np.median(ts))
    nbytes = S.numel() * 4
    del S, st
    torch.cuda.empty_cache()
    return {"states": wl.tiles, "ms": round(ms, 3), "gbps": round(nbytes / (ms * 1e-3) / 1e9, 1),
            "fp32_bytes": nbytes, "n_comp": wl.n_comp,
            "note": "fp64 fit, smoothing and codes per state: bound by vector-ALU issue, not by HBM"}


def decode_rotating(wl, dims, S0, toks, copies=2, reps=3):
    """Average decode launch duration when `copies` independent batches of the
    same size take turns launch by launch (positions 1..W each, one graph), so
    that between two steps of one batch the others stream through the 256 MB
    Infinity Cache and evict its state: every step reads its codes from HBM.
    (In a loop over one batch its codes can stay resident from one step to the
    next when they fit.)"""
    import torch
    from paper_2609_38166_amd import binding as B_
    sts = [B_.State.empty(dims) for _ in range(copies)]
    o = torch.empty((wl.batch, wl.heads_v, wl.dv), dtype=torch.float32, device="cuda")
    q, k, v, a, b = toks
    W = wl.window

    def window():
        for i in range(W):
            for st in sts:
                B_.leapquant_decode_step(dims, st, q[i], k[i], v[i], a[i], b[i], o)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for st in sts:
            B_.leapquant_quantize_state(dims, S0, st)
        window()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        window()
    torch.cuda.synchronize()
    ts = []
    for rep in range(reps + 1):
        for st in sts:
            B_.leapquant_quantize_state(dims, S0, st)      # rec_len := 0
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        if rep:
            ts.append(e0.elapsed_time(e1) / (copies * W))
    for st in sts:
        if B_.leapquant_check_error(st):
            raise RuntimeError("device error during the rotating-batch decode timing")
    del sts
    return float(np.mean(ts))


def cold_copies(wl):
    """Batches to rotate so that the others' state (codes, scales, compensators
    and the window's records) exceeds 512 MB, twice the Infinity Cache."""
    per = wl.tiles * (code_bytes(wl) + scale_bytes(wl) + 2 * wl.n_comp * (wl.dk + wl.dv)
                      + wl.window * rec_bytes(wl))
    return max(2, 1 + int(np.ceil(512e6 / per)))


def staggered_windows(wl, dims, S0, toks, groups=(1, 4), reps=3, one_batch=False):
    """Average time per decode step over one window cycle (W steps, one commit
    per request) when the requests are split into G groups whose windows are
    offset by W/G steps, replayed as one graph.  Each group runs on its own
    stream (its commit follows its own decode; the other groups' decodes can
    run beside it), or with one_batch every step is one decode launch over all
    requests at their mixed window positions, followed by a commit masked to
    the group whose window just ended.  G = 1 is the aligned schedule of the
    headline step."""
    import torch
    from paper_2609_38166_amd import binding as B_
    W, Bt = wl.window, wl.batch
    q, k, v, a, b = toks
    st = B_.State.empty(dims)
    o = torch.empty((wl.batch, wl.heads_v, wl.dv), dtype=torch.float32, device="cuda")

    def sub(b0, b1):
        v = st.requests(b0, b1)
        return v.dims, v

    res = {}
    for G in groups:
        R = Bt // G
        parts = [(gi * R, (gi + 1) * R, (gi * W // G) % W) + sub(gi * R, (gi + 1) * R) for gi in range(G)]
        streams = [torch.cuda.Stream() for _ in range(G)]
        masks = []
        for b0, b1, _, _, _ in parts:
            mk = torch.zeros(Bt, dtype=torch.int32, device="cuda")
            mk[b0:b1] = 1
            masks.append(mk)

        def cycle_one_batch():
            for t in range(W):
                B_.leapquant_decode_step(dims, st, q[t], k[t], v[t], a[t], b[t], o)
                for (b0, b1, off, _, _), mk in zip(parts, masks):
                    if (t + 1 + off) % W == 0:
                        B_.leapquant_window_commit(dims, st, mk)

        def cycle_streams():
            main = torch.cuda.current_stream()
            for s_ in streams:
                s_.wait_stream(main)
            for t in range(W):
                for (b0, b1, off, d, sv), s_ in zip(parts, streams):
                    with torch.cuda.stream(s_):
                        B_.leapquant_decode_step(d, sv, q[t][b0:b1], k[t][b0:b1], v[t][b0:b1], a[t][b0:b1],
                                                 b[t][b0:b1], o[b0:b1])
                        if (t + 1 + off) % W == 0:
                            B_.leapquant_window_commit(d, sv)
            for s_ in streams:
                main.wait_stream(s_)

        cycle = cycle_one_batch if one_batch else cycle_streams

        def reset():
            B_.leapquant_quantize_state(dims, S0, st)
            for b0, b1, off, _, _ in parts:
                st.rec_len[b0:b1] = off

        reset()
        cycle()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        reset()
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            cycle()
        ts = []
        for rep in range(reps + 1):
            reset()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            g.replay()
            e1.record()
            torch.cuda.synchronize()
            if rep:
                ts.append(e0.elapsed_time(e1) / W)
        if B_.leapquant_check_error(st):
            raise RuntimeError("device error during the staggered-window timing")
        res[f"G{G}{'_one_batch' if one_batch else ''}_us_per_step"] = round(float(np.mean(ts)) * 1e3, 2)
        del g
    del st
    return res


def fused_schedules(wl, dims, S0, toks, G=4, reps=3):
    """The decode step fused with the window-end commit (row f2), per decode step
    over one window cycle, replayed as one graph each:
      aligned_unfused -- W decode launches, then a commit of every tile (the
                         headline schedule);
      aligned_fused   -- W - 1 decode launches, then one fused launch that
                         decodes and commits every tile;
      staggered_fused -- requests in G groups whose windows are offset by W/G
                         steps; every step is one fused launch, in which the
                         group whose window fills commits;
      staggered_unfused -- the same schedule as a decode launch plus a commit
                         masked to that group.
    commit_share_aligned is the commit's part of the aligned unfused cycle."""
    import torch
    from paper_2609_38166_amd import binding as B_
    W, Bt = wl.window, wl.batch
    q, k, v, a, b = toks
    st = B_.State.empty(dims)
    o = torch.empty((wl.batch, wl.heads_v, wl.dv), dtype=torch.float32, device="cuda")
    R = Bt // G
    offs = torch.as_tensor([(bi // R) * W // G for bi in range(Bt)], dtype=torch.int32, device="cuda")
    masks = []
    for gi in range(G):
        mk = torch.zeros(Bt, dtype=torch.int32, device="cuda")
        mk[gi * R:(gi + 1) * R] = 1
        masks.append(mk)

    def aligned(fused):
        def cycle():
            for t in range(W):
                if fused and t == W - 1:
                    B_.leapquant_decode_step_commit(dims, st, q[t], k[t], v[t], a[t], b[t], o)
                else:
                    B_.leapquant_decode_step(dims, st, q[t], k[t], v[t], a[t], b[t], o)
            if not fused:
                B_.leapquant_window_commit(dims, st)
        return cycle, False

    def staggered(fused):
        def cycle():
            for t in range(W):
                if fused:
                    B_.leapquant_decode_step_commit(dims, st, q[t], k[t], v[t], a[t], b[t], o)
                else:
                    B_.leapquant_decode_step(dims, st, q[t], k[t], v[t], a[t], b[t], o)
                    for gi in range(G):
                        if (t + 1 + gi * W // G) % W == 0:
                            B_.leapquant_window_commit(dims, st, masks[gi])
        return cycle, True

    res = {}
    for name, (cycle, stag) in (("aligned_unfused", aligned(False)), ("aligned_fused", aligned(True)),
                                ("staggered_unfused", staggered(False)), ("staggered_fused", staggered(True))):
        def reset():
            B_.leapquant_quantize_state(dims, S0, st)
            if stag:
                st.rec_len.copy_(offs[:, None].expand(Bt, wl.heads_v))
        reset()
        cycle()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        reset()
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            cycle()
        ts = []
        for rep in range(reps + 1):
            reset()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            g.replay()
            e1.record()
            torch.cuda.synchronize()
            if rep:
                ts.append(e0.elapsed_time(e1) / W)
        if B_.leapquant_check_error(st):
            raise RuntimeError(f"device error during the {name} schedule")
        res[f"{name}_us_per_step"] = round(float(np.mean(ts)) * 1e3, 2)
        del g
    del st
    res["groups"] = G
    return res


def device_inputs(wl, T, seed):
    """Step-major tokens of T steps and an fp32 state drawn on the device with
    the workload's distributions (unit q and k, v ~ N(0, I), beta = sigmoid(N),
    decay = exp(-0.1 softplus(N))).  For throughput only: no kernel's work
    depends on the values."""
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    B_, Hv, Hk = wl.batch, wl.heads_v, wl.heads_k

    def rn(*shape):
        return torch.randn(shape, generator=g, device="cuda")
    q, k = rn(T, B_, Hk, wl.dk), rn(T, B_, Hk, wl.dk)
    q /= q.norm(dim=-1, keepdim=True)
    k /= k.norm(dim=-1, keepdim=True)
    v = rn(T, B_, Hv, wl.dv)
    a = torch.exp(-0.1 * torch.nn.functional.softplus(rn(T, B_, Hv, wl.dk) if wl.g > 1 else rn(T, B_, Hv)))
    b = torch.sigmoid(rn(T, B_, Hv))
    S0 = rn(B_, Hv, wl.dv, wl.dk) * 0.1
    return S0, (q, k, v, a, b)


def config_line(wl, args):
    """Throughput of one more workload shape: kernel times over one window
    (cache-resident and with rotating batches), token-head steps/s from the
    kernel times of the whole T-token trace, the decode's roofline, and the
    per-step bf16 / fp32 baselines at the same shape."""
    import torch
    from paper_2609_38166_amd import binding as B_
    dims = B_.make_dims(wl.batch, wl.heads_v, wl.heads_k, window=wl.window, n_comp=wl.n_comp,
                        power_iters=wl.power_iters, gate=wl.gate, code=wl.code)
    W = wl.window
    S0, toks = device_inputs(wl, W, wl.seed + 17)
    kt = per_launch_times(wl, dims, S0, toks)
    ncold = cold_copies(wl)
    cold = decode_rotating(wl, dims, S0, toks, copies=ncold)
    dbytes = float(np.mean([decode_bytes(wl, i) for i in range(1, W + 1)])) * wl.tiles
    step_ms = cold + kt["commit_ms"] / W                      # per token, commits amortised
    trace_ms = cold * wl.steps + kt["commit_ms"] * (wl.steps // W) + kt["quantize_ms"]
    q, k, v, a, b = toks
    base = {}
    for name, dtype, tdt in (("bf16", B_.LQ_STATE_BF16, torch.bfloat16), ("fp32", B_.LQ_STATE_F32, torch.float32)):
        S = S0.to(tdt).contiguous()
        o = torch.empty((wl.batch, wl.heads_v, wl.dv), dtype=torch.float32, device="cuda")

        def run(S=S, o=o, dtype=dtype):
            for t in range(W):
                B_.leapquant_baseline_step(dims, S, dtype, q[t], k[t], v[t], a[t], b[t], o)
        run()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            run()
        bs, _ = time_steps(g.replay, 2, 1)
        base[name] = bs / (2 * W) * 1e3
        del S, g
    out = {"workload": wl.name, "tiles": wl.tiles, "heads_k": wl.heads_k, "tokens": wl.steps, "window": W,
           "n_comp": wl.n_comp, "code": {0: "int8", 1: "e4m3", 2: "int4", 3: "int6"}[wl.code],
           "value": round(wl.tiles * wl.steps / (trace_ms * 1e-3), 1), "unit": "token-head steps/s",
           "ms_per_trace_from_kernels": round(trace_ms, 3),
           "decode_us": round(cold * 1e3, 2), "decode_us_cache_resident": round(kt["decode_ms"] * 1e3, 2),
           "commit_us": round(kt["commit_ms"] * 1e3, 2), "quantize_us": round(kt["quantize_ms"] * 1e3, 2),
           "roofline": {"kernel": "decode_step", "bound": "hbm",
                        "achieved": round(dbytes / (cold * 1e-3) / 1e9, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(dbytes / (cold * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                        "bytes_per_launch": round(dbytes), "rotating_batches": ncold},
           "bf16_us_per_step": round(base["bf16"] * 1e3, 2), "fp32_us_per_step": round(base["fp32"] * 1e3, 2),
           "speedup_vs_bf16": round(base["bf16"] / step_ms, 3), "speedup_vs_fp32": round(base["fp32"] / step_ms, 3),
           "data": "device-drawn state and tokens with the workload's distributions"}
    return out


def copy_calibration(nbytes=1 << 30):
    """One plain device-to-device copy of known size, for scaling the HBM byte
    counters of a profiler run (FETCH_SIZE / WRITE_SIZE of this dispatch are
    compared with nbytes read and nbytes written)."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def stream_rw_ceiling(nbytes, reps=5):
    """Measured HBM rate (bytes read + bytes written per second) of a kernel
    that reads a buffer and writes it back in place with coalesced 16-byte
    plain loads and stores, nothing else: the ceiling of the dense baselines'
    access pattern at the same state size."""
    import ctypes as C
    import torch
    from paper_2609_38166_amd import build as lib_build
    L = C.CDLL(lib_build.BENCH_LIB)
    L.lqb_stream_rw.argtypes = [C.c_void_p, C.c_size_t, C.c_int, C.c_void_p]
    L.lqb_stream_rw.restype = C.c_int
    buf = torch.zeros(nbytes // 4, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    best = None
    for grid in (256 * 16, 256 * 64, 256 * 256):
        def launch():
            rc = L.lqb_stream_rw(buf.data_ptr(), nbytes, grid, stream.cuda_stream)
            if rc != 0:
                raise RuntimeError(f"lqb_stream_rw failed: {rc}")
        launch()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            launch()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3)
        gbs = 2 * nbytes / float(np.median(ts)) / 1e9
        if best is None or gbs > best["gbps"]:
            best = {"gbps": round(gbs, 1), "frac_of_hbm_peak": round(gbs / PEAK_HBM_GBS, 4), "bytes": nbytes,
                    "grid": grid}
    del buf
    return best


def stream_read_ceiling(nbytes=4 << 30, reps=5):
    """Measured HBM read rate of a kernel that only streams a 4 GiB buffer
    (non-temporal 16-byte coalesced loads, far beyond the 256 MB Infinity
    Cache): the practical read ceiling next to which the decode's rate is read."""
    import ctypes as C
    import torch
    from paper_2609_38166_amd import build as lib_build
    L = C.CDLL(lib_build.BENCH_LIB)
    L.lqb_stream_read.argtypes = [C.c_void_p, C.c_size_t, C.c_void_p, C.c_int, C.c_void_p]
    L.lqb_stream_read.restype = C.c_int
    buf = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    grid = 256 * 128
    sink = torch.empty(grid, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    def launch():
        rc = L.lqb_stream_read(buf.data_ptr(), nbytes, sink.data_ptr(), grid, stream.cuda_stream)
        if rc != 0:
            raise RuntimeError(f"lqb_stream_read failed: {rc}")
    launch()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        launch()
        e1.record(stream)
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) * 1e-3)
    del buf, sink
    gbs = nbytes / float(np.median(ts)) / 1e9
    return {"gbps": round(gbs, 1), "frac_of_hbm_peak": round(gbs / PEAK_HBM_GBS, 4), "bytes": nbytes}


DECODE_SOURCES = ("csrc/lq_decode.hip", "csrc/lq_decode.hpp", "csrc/lq_device.hpp", "build.py")


def decode_source_sha():
    """sha256 over the decode kernel's sources (launch, body, device helpers)
    and the build script that sets its compiler options, in that order."""
    import hashlib
    h = hashlib.sha256()
    for f in DECODE_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2609_38166_amd", f), "rb").read())
    return h.hexdigest()


def traffic_from_profile(wl):
    """HBM bytes per decode launch from the committed counter summary, if it
    was taken on the current decode kernel source; None otherwise."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"decode_step_traffic_{wl.name}.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and line.startswith("- "):
            key, val = line[2:].split(":", 1)
            fields[key.strip()] = val.strip().strip("`")
    if fields.get("decode source sha256") != decode_source_sha() or "traffic bytes per launch" not in fields:
        return None
    return float(fields["traffic bytes per launch"])


def cpu_baseline(wl, n_tiles):
    """The CPU oracle (fp64, OpenMP over tiles) on a bounded sample of the same
    workload: window-start quantization, all T tokens and the commits."""
    from oracle import oracle as O
    from paper_2609_38166_amd import synth
    tiles = np.linspace(0, wl.tiles - 1, n_tiles).astype(int)
    cfg = O.make_cfg(dk=wl.dk, dv=wl.dv, window=wl.window, n_comp=wl.n_comp,
                     power_iters=wl.power_iters, gate=wl.gate, code=wl.code)
    pst = synth.Streams(wl, synth.PHASE_PREFILL, tiles)
    ptok = synth.tile_major(wl, pst, pst.draw(wl.prefill))
    _, Sp = O.run_baseline(cfg, np.zeros((n_tiles, wl.dk, wl.dv)), ptok, mode=O.STATE_F32,
                           want_o=False)
    F = synth.outlier_factor(synth.outliers(wl, tiles))
    S0 = (Sp.astype(np.float32) * F).astype(np.float64)
    dst = synth.Streams(wl, synth.PHASE_DECODE, tiles)
    tok = synth.tile_major(wl, dst, dst.draw(wl.steps))
    threads = O.default_threads()
    t0 = time.perf_counter()
    O.run_dense(cfg, S0, tok, snapshots=False, threads=threads)
    dt = time.perf_counter() - t0
    return {"value": round(n_tiles * wl.steps / dt, 1), "unit": "token-head steps/s",
            "cores": threads, "kind": "oracle",
            "sample": f"{n_tiles} of {wl.tiles} tiles (evenly spaced), all {wl.steps} tokens, "
                      f"quantize + decode + commits in fp64, {dt:.2f} s"}


# ----------------------------------------------------------------------------- sweep

SWEEP = (  # label, W, r, smooth, code (0: INT8, 4: BF16 state)
    ("bf16 per-window", 16, 0, 0, 4),
    ("int8 per-step", 1, 0, 0),
    ("int8 per-window", 16, 0, 0),
    ("+ compensator tokens", 16, 4, 0),
    ("+ smoothing (LeapQuant)", 16, 4, 1),
    ("window 4", 4, 4, 1), ("window 8", 8, 4, 1), ("window 32", 32, 4, 1), ("window 64", 64, 4, 1),
    ("tokens 2", 16, 2, 1), ("tokens 8", 16, 8, 1), ("tokens 16", 16, 16, 1),
)


def sweep(args):
    """Per-step cost of each configuration on a GDN layer at batch 256 (32 value
    heads, 16 key heads, d = 128): average decode launch over one window plus the
    window's commit divided by W, against the per-step fp32 and bf16 baselines."""
    import torch
    from paper_2609_38166_amd import binding as B_, synth
    base = synth.WORKLOADS["gdn_qwen3next"].with_(name="gdn_b256", batch=256, steps=64)
    dims0 = B_.make_dims(base.batch, base.heads_v, base.heads_k, window=64, n_comp=4,
                         power_iters=base.power_iters, gate=base.gate, code=base.code)
    toks = device_tokens(base, synth.PHASE_DECODE, 64)
    S0 = prefill_state(base, dims0)
    q, k, v, a, b = toks
    res = {}
    for name, dtype, width, tdt in (("fp32", B_.LQ_STATE_F32, 4, torch.float32),
                                    ("bf16", B_.LQ_STATE_BF16, 2, torch.bfloat16)):
        S = S0.to(tdt).contiguous()
        o = torch.empty((base.batch, base.heads_v, base.dv), dtype=torch.float32, device="cuda")

        def run(S=S, o=o, dtype=dtype):
            for t in range(64):
                B_.leapquant_baseline_step(dims0, S, dtype, q[t], k[t], v[t], a[t], b[t], o)
        run()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            run()
        bs, _ = time_steps(g.replay, 3, 1)
        res[name] = bs / (3 * 64) * 1e6
        print(json.dumps({"sweep": f"{name} per-step", "us_per_step": round(res[name], 2),
                          "speedup_vs_fp32": round(res["fp32"] / res[name], 3)}), flush=True)
        del S
    for row in SWEEP:
        label, W, r, smooth = row[:4]
        code = row[4] if len(row) > 4 else base.code
        wl = base.with_(window=W, n_comp=r, smooth=smooth, code=code)
        dims = B_.make_dims(wl.batch, wl.heads_v, wl.heads_k, window=W, n_comp=r,
                            power_iters=wl.power_iters, gate=wl.gate, code=wl.code, smooth=smooth)
        kt = per_launch_times(wl, dims, S0, toks)
        step = kt["decode_ms"] * 1e3 + kt["commit_ms"] * 1e3 / W
        print(json.dumps({"sweep": label, "window": W, "n_comp": r, "smooth": smooth, "code": code,
                          "decode_us": round(kt["decode_ms"] * 1e3, 2),
                          "commit_us": round(kt["commit_ms"] * 1e3, 2),
                          "us_per_step": round(step, 2),
                          "speedup_vs_fp32": round(res["fp32"] / step, 3),
                          "speedup_vs_bf16": round(res["bf16"] / step, 3)}), flush=True)


# ----------------------------------------------------------------------------- commit split

def commit_split(args):
    """Where the window commit's time goes (KDA workload, 8192 tiles, W = 64):
    the commit and the quantization timed (per_launch_times) with r = 0, 4, 8
    Compensator Tokens at 4 power sweeps and with 1 and 2 sweeps at r = 8, on
    the same device-drawn state and tokens.  The commit at r = 0 is the base
    (reconstruction of the window, smoothing, codes); the r = 8 times at 1, 2
    and 4 sweeps give the cost of one token-sweep (least squares over the
    three) and, with the base, the cost of a token outside its sweeps."""
    from paper_2609_38166_amd import binding as B_, synth
    wl0 = synth.WORKLOADS["kda_kimi"]
    S0, toks = device_inputs(wl0, wl0.window, wl0.seed + 17)
    rows = []
    for r, pi in ((0, 4), (4, 4), (8, 1), (8, 2), (8, 4)):
        wl = wl0.with_(n_comp=r, power_iters=pi)
        dims = B_.make_dims(wl.batch, wl.heads_v, wl.heads_k, window=wl.window, n_comp=r, power_iters=pi,
                            gate=wl.gate, code=wl.code)
        kt = per_launch_times(wl, dims, S0, toks)
        rows.append({"n_comp": r, "power_iters": pi, "commit_us": round(kt["commit_ms"] * 1e3, 1),
                     "quantize_us": round(kt["quantize_ms"] * 1e3, 1)})
        log(f"[commit split] {rows[-1]}")
    base = rows[0]["commit_us"]
    pis = np.array([1.0, 2.0, 4.0])
    c8 = np.array([rows[2]["commit_us"], rows[3]["commit_us"], rows[4]["commit_us"]])
    slope, icpt = np.polyfit(pis, c8, 1)
    out = {"commit_split": {
        "workload": "kda_kimi: 8192 tiles, W = 64, per-channel gate, int8",
        "runs": rows,
        "base_us": base,
        "per_token_sweep_us": round(slope / 8, 2),
        "per_token_outside_sweeps_us": round((icpt - base) / 8, 2),
        "fp64_fma_bound_us_r8_4sweeps": round(8192 * 2.74e6 * 2 / 78.6e12 * 1e6, 1),
        "note": ("base = the commit at r = 0 (window reconstruction, smoothing, codes); the r = 8 commit is "
                 "base + 8 x (per-token cost + power_iters x per-token-sweep cost)")}}
    print(json.dumps(out), flush=True)


# ----------------------------------------------------------------------------- long trace

def long_trace(args, every=1024, chunk=256):
    """Drift of the quantized trajectory from the unquantized fp32 one over the
    long GDN trace (App. B.1 Eq. (deviation), Sec. 3.2): both on the GPU from the
    same fp32 initial state (fp32 prefill plus outlier lines) and the same tokens;
    every `every` tokens (right after a window commit) the relative Frobenius
    distance of the dequantized state from the fp32 baseline state, per tile,
    and the relative L2 distance of that token's outputs."""
    import torch
    from paper_2609_38166_amd import binding as B_, synth
    wl = synth.WORKLOADS["gdn_long"].with_(gate_scale=args.gate_scale)
    dims = B_.make_dims(wl.batch, wl.heads_v, wl.heads_k, window=wl.window, n_comp=wl.n_comp,
                        power_iters=wl.power_iters, gate=wl.gate, code=wl.code)
    t0 = time.time()
    S0 = prefill_state(wl, dims)
    st = B_.State.empty(dims)
    B_.leapquant_quantize_state(dims, S0, st)
    F = S0.clone()
    o1 = torch.empty((wl.batch, wl.heads_v, wl.dv), dtype=torch.float32, device="cuda")
    o2 = torch.empty_like(o1)
    Sq = torch.empty_like(S0)
    streams = synth.Streams(wl, synth.PHASE_DECODE)
    curve = []
    t = 0
    while t < wl.steps:
        sm = synth.step_major_full(wl, streams.draw(chunk))
        dv_ = {k_: torch.from_numpy(v_).cuda() for k_, v_ in sm.items()}
        for i in range(chunk):
            x = (dv_["q"][i], dv_["k"][i], dv_["v"][i], dv_["alpha"][i], dv_["beta"][i])
            B_.leapquant_decode_step(dims, st, *x, o1)
            B_.leapquant_baseline_step(dims, F, B_.LQ_STATE_F32, *x, o2)
            t += 1
            if t % wl.window == 0:
                B_.leapquant_window_commit(dims, st)
            if t % every == 0:
                B_.leapquant_dequantize_state(dims, st, Sq)
                d = ((Sq - F).flatten(2).norm(dim=-1) / F.flatten(2).norm(dim=-1)).flatten()
                od = ((o1 - o2).norm(dim=-1) / o2.norm(dim=-1)).flatten()
                curve.append({"step": t, "state_drift_mean": float(d.mean()), "state_drift_max": float(d.max()),
                              "output_drift_mean": float(od.mean()), "output_drift_max": float(od.max())})
                log(f"[long trace] {curve[-1]}")
    streams.close()
    if B_.leapquant_check_error(st):
        raise RuntimeError("device error during the long trace")
    means = [c["state_drift_mean"] for c in curve]
    out = {"long_trace": {
        "workload": f"{wl.name}: GDN batch {wl.batch} x {wl.heads_v} heads, {wl.steps} tokens, W={wl.window}, "
                    f"r={wl.n_comp}, int8 state, gate scale {wl.gate_scale}",
        "every": every, "curve": curve,
        "first_to_last_ratio": round(means[-1] / means[0], 4) if means and means[0] > 0 else None,
        "reference": "unquantized fp32 recurrence (the baseline kernel) from the same initial state",
        "note": ("synthetic gates: state half-life about 9 tokens, so the quantization error cannot "
                 "accumulate and the curve is flat by construction" if wl.gate_scale >= 0.05 else
                 "long-memory variant: decays close to 1, so the state's memory is set by the delta "
                 "rule's erase along each key (about d_k / beta tokens)"),
        "seconds": round(time.time() - t0, 1)}}
    print(json.dumps(out), flush=True)


# ----------------------------------------------------------------------------- main

def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the decode path has no "
              "cross-GPU step -- tiles shard by request and head", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2609_38166_amd import binding as B_, synth
    B_.lib()
    torch.cuda.set_device(0)
    if args.sweep:
        sweep(args)
        return
    if args.long_trace:
        long_trace(args)
        return
    if args.commit_split:
        commit_split(args)
        return
    wl = synth.WORKLOADS[args.workload]
    dims = B_.make_dims(wl.batch, wl.heads_v, wl.heads_k, window=wl.window, n_comp=wl.n_comp,
                        power_iters=wl.power_iters, gate=wl.gate, code=wl.code)
    t0 = time.time()
    log(f"[bench] {wl.name}: tiles={wl.tiles} T={wl.steps} W={wl.window} r={wl.n_comp}")
    toks = device_tokens(wl, synth.PHASE_DECODE, wl.steps)
    log(f"[bench] decode inputs on device ({time.time() - t0:.1f}s)")
    S0 = prefill_state(wl, dims)
    log(f"[bench] prefill done ({time.time() - t0:.1f}s)")

    if args.profile_decode:
        ncold = cold_copies(wl)
        cold = decode_rotating(wl, dims, S0, toks, copies=ncold, reps=2)
        # eight steps of each dense baseline, for their counters
        q, k, v, a, b = toks
        for dtype, tdt in ((B_.LQ_STATE_F32, torch.float32), (B_.LQ_STATE_BF16, torch.bfloat16)):
            S = S0.to(tdt).contiguous()
            o = torch.empty((wl.batch, wl.heads_v, wl.dv), dtype=torch.float32, device="cuda")
            for t in range(8):
                B_.leapquant_baseline_step(dims, S, dtype, q[t], k[t], v[t], a[t], b[t], o)
            torch.cuda.synchronize()
            del S
        copy_calibration()
        print(json.dumps({"profile_decode_us": round(cold * 1e3, 2), "rotating_batches": ncold}), flush=True)
        return

    runner = Runner(wl, dims, S0, toks, use_graph=not args.no_graph)
    log("[bench] runner ready")
    secs, wall = time_steps(runner.step, args.steps, args.warmup)
    bits = B_.leapquant_check_error(runner.st)
    if bits:
        raise RuntimeError(f"device error bits {bits} after the timed steps")
    ms_step = secs / args.steps * 1e3
    tile_steps = wl.tiles * wl.steps
    value = tile_steps * args.steps / secs
    log(f"[bench] leapquant {ms_step:.3f} ms/step, {value:.4g} token-head steps/s")
    if args.profile:
        copy_calibration()
        print(json.dumps({"profile_ms_per_step": ms_step}), flush=True)
        return

    kt = per_launch_times(wl, dims, S0, toks)
    W = wl.window
    dec_bytes = [decode_bytes(wl, i) * wl.tiles for i in range(1, W + 1)]
    dec_avg_bytes = float(np.mean(dec_bytes))
    achieved = dec_avg_bytes / (kt["decode_ms"] * 1e-3) / 1e9
    step_bytes = (sum(dec_bytes) * (wl.steps // W) + commit_bytes(wl, W) * wl.tiles * (wl.steps // W)
                  + quantize_bytes(wl) * wl.tiles)
    eff = step_bytes / (ms_step * 1e-3) / 1e9
    log(f"[bench] decode {kt['decode_ms'] * 1e3:.1f} us/launch ({achieved:.0f} GB/s, codes cache-resident), "
        f"commit {kt['commit_ms'] * 1e3:.1f} us, quantize {kt['quantize_ms'] * 1e3:.1f} us")
    traffic = traffic_from_profile(wl)
    # The roofline is taken where no batch's state can stay in the Infinity Cache
    # between its steps: batches rotate launch by launch (cold_copies).
    ncold = cold_copies(wl)
    cold = decode_rotating(wl, dims, S0, toks, copies=ncold)
    achieved_cold = dec_avg_bytes / (cold * 1e-3) / 1e9
    log(f"[bench] decode with {ncold} rotating batches {cold * 1e3:.1f} us/launch ({achieved_cold:.0f} GB/s)")

    out = {
        "metric": "token-head decode steps/s + effective HBM GB/s (% of peak), speedup vs bf16 state",
        "value": round(value, 1),
        "unit": "token-head steps/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32+f64", "data": "synthetic",
        "config": {"workload": f"{wl.name}: KDA (per-channel gate) batch {wl.batch}, {wl.heads_v} heads, "
                               f"d_k=d_v={wl.dk}, {wl.steps} decode tokens, W={wl.window}, "
                               f"r={wl.n_comp}, int8 state" if wl.gate == synth.GATE_DIAG else wl.name,
                   "tiles": wl.tiles, "tokens": wl.steps, "window": wl.window, "n_comp": wl.n_comp,
                   "graph": not args.no_graph},
        "effective_gbps": round(eff, 1),
        "frac_of_hbm_peak": round(eff / PEAK_HBM_GBS, 4),
        "roofline": {"kernel": "decode_step", "bound": "hbm", "achieved": round(achieved_cold, 1),
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(achieved_cold / PEAK_HBM_GBS, 4),
                     "traffic": None if traffic is None else round(traffic),
                     "bytes_per_launch": round(dec_avg_bytes), "avg_launch_us": round(cold * 1e3, 2),
                     "timing": f"{ncold} batches rotate launch by launch (positions 1..W), so every step reads "
                               "its state from HBM",
                     "cache_resident": {
                         "avg_launch_us": round(kt["decode_ms"] * 1e3, 2), "achieved": round(achieved, 1),
                         "frac": round(achieved / PEAK_HBM_GBS, 4),
                         "note": "one batch, as in the headline step: its int8 codes (134 MB) can stay in the "
                                 "256 MB Infinity Cache from one step to the next"}},
        "kernels_us": {"decode_avg": round(kt["decode_ms"] * 1e3, 2),
                       "decode_avg_cold": round(cold * 1e3, 2),
                       "commit": round(kt["commit_ms"] * 1e3, 2),
                       "quantize": round(kt["quantize_ms"] * 1e3, 2)},
    }

    if not args.no_variants:
        out["bulk_quantize"] = bulk_quantize()
        log(f"[bench] bulk quantize {out['bulk_quantize']}")
        out["staggered_windows"] = staggered_windows(wl, dims, S0, toks)
        out["staggered_windows"].update(staggered_windows(wl, dims, S0, toks, groups=(4,), one_batch=True))
        out["staggered_windows"]["note"] = ("requests in G groups whose windows are offset by W/G, one stream "
                                            "per group (one_batch: one decode launch over the mixed window "
                                            "positions, then a commit masked to the group whose window ended); "
                                            "per decode step over one window cycle incl. commits")
        log(f"[bench] staggered windows {out['staggered_windows']}")
        fs = fused_schedules(wl, dims, S0, toks)
        dec_us = kt["decode_ms"] * 1e3
        fs["commit_share_aligned"] = round(kt["commit_ms"] * 1e3 / (W * dec_us + kt["commit_ms"] * 1e3), 4)
        fs["note"] = ("decode fused with the window-end commit (leapquant_decode_step_commit) against a "
                      "decode launch plus a commit, aligned and staggered (G groups, one batch); per decode "
                      "step over one window cycle incl. commits")
        out["fused_commit"] = fs
        log(f"[bench] fused commit {fs}")
    ceil = stream_read_ceiling()
    out["stream_read_ceiling"] = ceil
    out["roofline"]["frac_of_stream_ceiling"] = round(achieved_cold / ceil["gbps"], 4)
    log(f"[bench] streaming-read ceiling {ceil}")

    if not args.no_variants and wl.name == "kda_kimi":
        # One GPU's share under 8-way tensor parallelism (heads split across GPUs):
        # the first heads_v / 8 heads of every request, 1024 tiles -- a single
        # round of resident decode workgroups, so occupancy and the tail differ.
        sw = wl.with_(name="kda_kimi_tp8_shard", heads_v=wl.heads_v // 8, heads_k=wl.heads_k // 8)
        sd = B_.make_dims(sw.batch, sw.heads_v, sw.heads_k, window=sw.window, n_comp=sw.n_comp,
                          power_iters=sw.power_iters, gate=sw.gate, code=sw.code)
        s_S0 = S0[:, :sw.heads_v].contiguous()
        s_toks = tuple(t_[:W, :, :(sw.heads_k if j < 2 else sw.heads_v)].contiguous()
                       for j, t_ in enumerate(toks))
        sk = per_launch_times(sw, sd, s_S0, s_toks)
        sstep = sk["decode_ms"] * sw.steps + sk["commit_ms"] * (sw.steps // W) + sk["quantize_ms"]
        sbytes = float(np.mean([decode_bytes(sw, i) for i in range(1, W + 1)])) * sw.tiles
        out["tp8_shard"] = {"tiles": sw.tiles, "heads_v": sw.heads_v,
                            "value_from_kernels": round(sw.tiles * sw.steps / (sstep * 1e-3), 1),
                            "decode_us": round(sk["decode_ms"] * 1e3, 2),
                            "decode_gbps": round(sbytes / (sk["decode_ms"] * 1e-3) / 1e9, 1),
                            "commit_us": round(sk["commit_ms"] * 1e3, 2),
                            "quantize_us": round(sk["quantize_ms"] * 1e3, 2)}
        log(f"[bench] tp8 shard: {out['tp8_shard']}")
        del s_S0, s_toks

        # the same layer with the paper's lower-bit residual codes (same inputs)
        var = {}
        for vname in ("kda_kimi_int6", "kda_kimi_int4", "kda_kimi_bf16w"):
            vw = synth.WORKLOADS[vname]
            vd = B_.make_dims(vw.batch, vw.heads_v, vw.heads_k, window=vw.window, n_comp=vw.n_comp,
                              power_iters=vw.power_iters, gate=vw.gate, code=vw.code, smooth=vw.smooth)
            vk = per_launch_times(vw, vd, S0, toks)
            vstep = (vk["decode_ms"] * vw.steps + vk["commit_ms"] * (vw.steps // vw.window)
                     + vk["quantize_ms"])
            vb = float(np.mean([decode_bytes(vw, i) for i in range(1, vw.window + 1)])) * vw.tiles
            var[vname] = {"value": round(vw.tiles * vw.steps / (vstep * 1e-3), 1),
                          "ms_per_step_from_kernels": round(vstep, 3),
                          "decode_us": round(vk["decode_ms"] * 1e3, 2),
                          "commit_us": round(vk["commit_ms"] * 1e3, 2),
                          "decode_bytes_per_launch": round(vb),
                          "decode_gbps": round(vb / (vk["decode_ms"] * 1e-3) / 1e9, 1)}
            log(f"[bench] {vname}: {var[vname]}")
        out["code_variants"] = var

        # RWKV7 at the same shape (App. A): two general-rule sub-steps per token,
        # W = 64 sub-steps (32 tokens) per window, per-channel gate, r = 8, int8
        rw = wl.with_(name="rwkv7_kimi_shape", rule=2)
        rd = B_.make_dims(rw.batch, rw.heads_v, rw.heads_v, window=rw.window, n_comp=rw.n_comp,
                          power_iters=rw.power_iters, gate=rw.gate, code=rw.code, rule=2)
        r_toks = rwkv7_tokens(rw, rw.window, 20260010)
        rk_ = per_launch_times(rw, rd, S0, r_toks)
        n_sub = 2 * rw.steps
        rstep = (rk_["decode_ms"] * n_sub + rk_["commit_ms"] * (n_sub // rw.window) + rk_["quantize_ms"])
        rb = float(np.mean([decode_bytes(rw, i) for i in range(1, rw.window + 1)])) * rw.tiles
        # per sub-step: q, k, b, v, alpha, beta inputs (the general rule reads b as well)
        rb += 4 * rw.dk * rw.tiles
        out["rwkv7"] = {"tiles": rw.tiles, "tokens": rw.steps, "sub_steps_per_window": rw.window,
                        "value": round(rw.tiles * rw.steps / (rstep * 1e-3), 1),
                        "unit": "token-head steps/s (two decode launches per token)",
                        "ms_per_step_from_kernels": round(rstep, 3),
                        "decode_us": round(rk_["decode_ms"] * 1e3, 2),
                        "decode_gbps": round(rb / (rk_["decode_ms"] * 1e-3) / 1e9, 1),
                        "commit_us": round(rk_["commit_ms"] * 1e3, 2)}
        log(f"[bench] rwkv7: {out['rwkv7']}")
        del r_toks

    if not args.no_variants and wl.name == "kda_kimi":
        # the other workload shapes: the GQA GDN layer with INT8 and E4M3 states,
        # and the large-batch GDN stress case with its frequent commits (W = 32)
        cl = {}
        for cw in (synth.WORKLOADS["gdn_qwen3next"],
                   synth.WORKLOADS["gdn_qwen3next"].with_(name="gdn_qwen3next_e4m3", code=synth.CODE_E4M3),
                   synth.WORKLOADS["gdn_stress"]):
            cl[cw.name] = config_line(cw, args)
            log(f"[bench] {cw.name}: {cl[cw.name]}")
            torch.cuda.empty_cache()
        out["configs"] = cl

    if not args.no_baselines:
        q, k, v, a, b = toks
        res = {}
        for name, dtype, width, tdt in (("bf16", B_.LQ_STATE_BF16, 2, torch.bfloat16),
                                        ("fp32", B_.LQ_STATE_F32, 4, torch.float32)):
            S = S0.to(tdt).contiguous()
            o = torch.empty((wl.batch, wl.heads_v, wl.dv), dtype=torch.float32, device="cuda")

            def run(S=S, o=o, dtype=dtype):
                for t in range(wl.steps):
                    B_.leapquant_baseline_step(dims, S, dtype, q[t], k[t], v[t], a[t], b[t], o)
            g = None
            if not args.no_graph:
                run()
                torch.cuda.synchronize()
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g):
                    run()
            fn = g.replay if g is not None else run
            bs, _ = time_steps(fn, args.steps, args.warmup)
            rate = tile_steps * args.steps / bs
            gbs = baseline_bytes(wl, width) * tile_steps * args.steps / bs / 1e9
            res[name] = {"value": round(rate, 1), "ms_per_step": round(bs / args.steps * 1e3, 4),
                         "effective_gbps": round(gbs, 1), "frac_of_hbm_peak": round(gbs / PEAK_HBM_GBS, 4)}
            del S
            torch.cuda.empty_cache()
            rw = stream_rw_ceiling(wl.tiles * wl.dk * wl.dv * width)
            res[name]["rw_ceiling_gbps"] = rw["gbps"]
            res[name]["frac_of_rw_ceiling"] = round(gbs / rw["gbps"], 4)
            log(f"[bench] {name} baseline {res[name]}")
        out["baselines"] = res
        out["speedup_vs_bf16"] = round(value / res["bf16"]["value"], 3)
        out["speedup_vs_fp32"] = round(value / res["fp32"]["value"], 3)
        out["byte_ratio_bound_vs_bf16"] = round(
            baseline_bytes(wl, 2) * wl.steps / (step_bytes / wl.tiles), 3)

    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle) ...")
        out["cpu_baseline"] = cpu_baseline(wl, min(args.cpu_sample_tiles, wl.tiles))
        log(f"[bench] cpu baseline {out['cpu_baseline']}")

    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
