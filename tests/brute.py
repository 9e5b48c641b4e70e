"""A second, deliberately naive float64 statement of the per-window method for
tiny tiles (d <= 8), written independently of the C oracle: every quantization
code is chosen by exhaustive search over all codes, every cumulative decay is an
explicit product, every state is a dense matrix.  Used only to pin the oracle.
"""
from __future__ import annotations

import numpy as np

F16 = np.float16


def f16(x):
    return np.float64(np.float16(np.float32(x)))


def int8_codes_bruteforce(x32: float, delta32: float, qmax: int = 127) -> int:
    """Nearest code in [-qmax, qmax] to x/delta (exhaustive), ties to even."""
    cand = np.arange(-qmax, qmax + 1, dtype=np.float64)
    target = np.float64(x32) / np.float64(delta32)
    d = np.abs(target - cand)
    best = np.flatnonzero(d == d.min())
    if len(best) == 1:
        return int(cand[best[0]])
    even = [int(cand[b]) for b in best if int(cand[b]) % 2 == 0]
    return even[0]


def quantize(S, r, iters, smooth=True, qmax=127):
    """S: [dk][dv] float64.  Returns (Z int [dk][dv], delta f32 [dv], c f32 [dk], Kt, Ut).
    qmax: largest integer code (127, 31 or 7 for 8-, 6- or 4-bit codes)."""
    dk, dv = S.shape
    M = S.astype(np.float64).copy()
    Kt = np.zeros((r, dk))
    Ut = np.zeros((r, dv))
    for h in range(r):
        x = np.array([np.sqrt(sum(M[k, v] ** 2 for v in range(dv))) for k in range(dk)])
        n = np.sqrt(sum(xi * xi for xi in x))
        if not n > 0:
            continue
        x = x * (1.0 / n)
        ok = True
        for _ in range(iters):
            y = np.array([sum(M[k, v] * x[k] for k in range(dk)) for v in range(dv)])
            x = np.array([sum(M[k, v] * y[v] for v in range(dv)) for k in range(dk)])
            n = np.sqrt(sum(xi * xi for xi in x))
            if not n > 0:
                ok = False
                break
            x = x * (1.0 / n)
        if not ok:
            continue
        kh = np.array([f16(xi) for xi in x])
        uh = np.array([f16(sum(M[k, v] * kh[k] for k in range(dk))) for v in range(dv)])
        Kt[h], Ut[h] = kh, uh
        M = M - np.outer(kh, uh)
    c = np.ones(dk, np.float32)
    if smooth:
        for k in range(dk):
            m = sum(abs(M[k, v]) for v in range(dv)) / dv
            c[k] = np.float32(np.sqrt(max(m, np.float64(np.float32(1e-12)))))
    Rc = np.zeros((dk, dv), np.float32)
    for k in range(dk):
        ic = np.float32(1.0) / c[k]
        for v in range(dv):
            Rc[k, v] = np.float32(np.float32(M[k, v]) * ic)
    Z = np.zeros((dk, dv), np.int64)
    delta = np.zeros(dv, np.float32)
    for v in range(dv):
        a = np.float32(np.max(np.abs(Rc[:, v])))
        if a == 0:
            continue
        delta[v] = np.float32(a / np.float32(qmax))
        for k in range(dk):
            Z[k, v] = int8_codes_bruteforce(Rc[k, v], np.float64(a) / qmax, qmax)
    return Z, delta, c, Kt, Ut


def dequantize(Z, delta, c, Kt, Ut):
    return (c.astype(np.float64)[:, None] * (Z * delta.astype(np.float64)[None, :])) + Kt.T @ Ut


def window_trajectory(S0, toks, W, r, iters, gate_diag, smooth=True):
    """Dense per-window trajectory with FP16 records.  toks: list of dicts with
    q, k, v (float32 arrays), alpha (scalar or [dk]) and beta."""
    dk, dv = S0.shape
    rep = quantize(S0, r, iters, smooth)
    S = dequantize(*rep)
    outs, reps = [], [rep]
    n = 0
    for t in toks:
        a = np.array([f16(x) for x in np.atleast_1d(t["alpha"])])
        D = np.diag(a if gate_diag else np.full(dk, a[0]))
        A = D @ S
        u = np.array([f16(np.float64(t["v"][j]) - (A[:, j] @ t["k"].astype(np.float64))) for j in range(dv)])
        tk = np.array([f16(np.float32(t["beta"]) * np.float32(t["k"][i])) for i in range(dk)])
        S = A + np.outer(tk, u)
        outs.append(S.T @ t["q"].astype(np.float64))
        n += 1
        if n == W:
            rep = quantize(S, r, iters, smooth)
            reps.append(rep)
            S = dequantize(*rep)
            n = 0
    return np.array(outs), reps
