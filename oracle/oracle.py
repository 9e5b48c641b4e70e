"""ctypes wrapper of the LeapQuant CPU oracle (test infrastructure only).

Only the test-suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  The product package never does.

Layouts are the paper's: one tile's state is S[d_k][d_v] (row = key channel),
codes Z[d_k][d_v], scales delta[d_v], smoothing c[d_k], compensators
Kt[r][d_k] / Ut[r][d_v], records (alpha_j, k~_j, u_j) as values.  Batched
drivers take token inputs as [tiles][T][...] arrays.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblqoracle.so")

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _b  # type: ignore
            _b.build()
        _lib = C.CDLL(LIB_PATH)
        _declare(_lib)
    return _lib


class Cfg(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "dk", "dv", "window", "n_comp", "power_iters", "gate", "code", "smooth",
        "quantize", "round_records", "rule")]


class _Inputs(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("q", "k", "v", "alpha", "beta", "b")]


class _Outputs(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in (
        "Z", "delta", "c", "Kt", "Ut", "S_final", "rec_a", "rec_k", "rec_u", "rec_len", "hist_a",
        "hist_k", "hist_u")]


GATE_SCALAR, GATE_DIAG = 0, 1
RULE_DELTA, RULE_ADD, RULE_GENERAL = 0, 1, 2   # b_t = D_t k_t (delta rule), b_t = 0, b_t given
CODE_INT8, CODE_E4M3, CODE_INT4, CODE_INT6, CODE_BF16 = 0, 1, 2, 3, 4
STATE_EXACT, STATE_F32, STATE_BF16 = 0, 1, 2


def make_cfg(dk=128, dv=128, window=16, n_comp=4, power_iters=4, gate=GATE_SCALAR,
             code=CODE_INT8, smooth=1, quantize=1, round_records=1, rule=RULE_DELTA) -> Cfg:
    return Cfg(dk, dv, window, n_comp, power_iters, gate, code, smooth, quantize, round_records, rule)


def code_dtype(cfg: Cfg):
    """Storage of one code: a byte, or the two bytes of a BF16 state entry."""
    return np.uint16 if cfg.code == CODE_BF16 else np.uint8


def _p(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _declare(L):
    vp, i32, f32 = C.c_void_p, C.c_int32, C.c_float
    for pre in ("lqo64_", "lqo32_"):
        getattr(L, pre + "quantize").argtypes = [vp] * 7
        getattr(L, pre + "dequantize").argtypes = [vp] * 7
        getattr(L, pre + "recurrent_step").argtypes = [vp, vp, vp, vp, vp, vp, vp, f32, vp, i32]
        getattr(L, pre + "window_step").argtypes = [vp, vp, vp, vp, vp, vp, vp, f32, vp, vp, vp, vp]
        getattr(L, pre + "readout_step").argtypes = [vp] * 10 + [i32] + [vp] * 5 + [f32] + [vp] * 4
        getattr(L, pre + "reconstruct").argtypes = [vp] * 10 + [i32, vp]
        for fn in ("run_dense", "run_readout"):
            getattr(L, pre + fn).argtypes = [vp, i32, i32, vp, vp, vp, vp, i32]
        getattr(L, pre + "run_baseline").argtypes = [vp, i32, i32, vp, vp, vp, vp, i32, i32]
        getattr(L, pre + "run_drift").argtypes = [vp, i32, i32, i32, vp, vp, vp, vp, i32]
    L.lqo_f32_to_f16_n.argtypes = [vp, vp, C.c_long]
    L.lqo_f32_to_bf16_n.argtypes = [vp, vp, C.c_long]
    L.lqo_f32_to_e4m3_n.argtypes = [vp, vp, C.c_long]
    L.lqo_e4m3_to_f32_n.argtypes = [vp, vp, C.c_long]


def _fn(name, prec):
    return getattr(lib(), ("lqo64_" if prec == 64 else "lqo32_") + name)


def default_threads() -> int:
    n = os.cpu_count() or 1
    return max(1, min(n, 16))


# --------------------------------------------------------------------------
# storage formats
# --------------------------------------------------------------------------

def f32_to_f16_bits(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.empty(x.shape, np.uint16)
    lib().lqo_f32_to_f16_n(_p(x), _p(y), x.size)
    return y


def f32_to_bf16_bits(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.empty(x.shape, np.uint16)
    lib().lqo_f32_to_bf16_n(_p(x), _p(y), x.size)
    return y


def f32_to_e4m3(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.empty(x.shape, np.uint8)
    lib().lqo_f32_to_e4m3_n(_p(x), _p(y), x.size)
    return y


def e4m3_to_f32(b) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint8)
    y = np.empty(b.shape, np.float32)
    lib().lqo_e4m3_to_f32_n(_p(b), _p(y), b.size)
    return y


# --------------------------------------------------------------------------
# single tile
# --------------------------------------------------------------------------

@dataclass
class Rep:
    """Quantized window-start representation of one tile."""
    Z: np.ndarray       # uint8 [dk][dv] code bytes (uint16 BF16 bits for the BF16 state)
    delta: np.ndarray   # float32 [dv]
    c: np.ndarray       # float32 [dk]
    Kt: np.ndarray      # float64 [r][dk] (FP16 values)
    Ut: np.ndarray      # float64 [r][dv]


def quantize(cfg: Cfg, S, prec=64) -> Rep:
    S = np.ascontiguousarray(S, dtype=np.float64)
    r = max(cfg.n_comp, 1)
    rep = Rep(np.zeros((cfg.dk, cfg.dv), code_dtype(cfg)), np.zeros(cfg.dv, np.float32),
              np.zeros(cfg.dk, np.float32), np.zeros((r, cfg.dk)), np.zeros((r, cfg.dv)))
    _fn("quantize", prec)(C.byref(cfg), _p(S), _p(rep.Z), _p(rep.delta), _p(rep.c),
                          _p(rep.Kt), _p(rep.Ut))
    rep.Kt, rep.Ut = rep.Kt[:cfg.n_comp], rep.Ut[:cfg.n_comp]
    return rep


def dequantize(cfg: Cfg, rep: Rep, prec=64) -> np.ndarray:
    S = np.zeros((cfg.dk, cfg.dv))
    Kt = np.ascontiguousarray(rep.Kt) if cfg.n_comp else np.zeros((1, cfg.dk))
    Ut = np.ascontiguousarray(rep.Ut) if cfg.n_comp else np.zeros((1, cfg.dv))
    _fn("dequantize", prec)(C.byref(cfg), _p(np.ascontiguousarray(rep.Z)),
                            _p(np.ascontiguousarray(rep.delta)), _p(np.ascontiguousarray(rep.c)),
                            _p(Kt), _p(Ut), _p(S))
    return S


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _read_vec(cfg: Cfg, b):
    """The read vector argument: required by the general rule, unused otherwise."""
    if cfg.rule == RULE_GENERAL:
        if b is None:
            raise ValueError("the general rule needs the read vector b")
        b = _f32(b)
        if b.shape != (cfg.dk,):
            raise ValueError(f"b must have shape ({cfg.dk},)")
        return b
    return None


def recurrent_step(cfg: Cfg, S, q, k, v, alpha, beta, mode=STATE_EXACT, prec=64, b=None):
    """One token of the unquantized recurrence; returns (S_new, o)."""
    S = np.array(S, dtype=np.float64, order="C")
    o = np.zeros(cfg.dv)
    alpha = _f32(np.atleast_1d(alpha))
    bv = _read_vec(cfg, b)
    _fn("recurrent_step", prec)(C.byref(cfg), _p(S), _p(_f32(q)), _p(_f32(k)), _p(bv), _p(_f32(v)),
                                _p(alpha), float(beta), _p(o), mode)
    return S, o


def window_step(cfg: Cfg, S, q, k, v, alpha, beta, prec=64, b=None):
    """One token of the per-window method, dense form; returns (S_new, o, (a, k~, u))."""
    S = np.array(S, dtype=np.float64, order="C")
    g = cfg.dk if cfg.gate else 1
    o, ra, rk, ru = np.zeros(cfg.dv), np.zeros(g), np.zeros(cfg.dk), np.zeros(cfg.dv)
    bv = _read_vec(cfg, b)
    _fn("window_step", prec)(C.byref(cfg), _p(S), _p(_f32(q)), _p(_f32(k)), _p(bv), _p(_f32(v)),
                             _p(_f32(np.atleast_1d(alpha))), float(beta), _p(o), _p(ra), _p(rk), _p(ru))
    return S, o, (ra, rk, ru)


def readout_step(cfg: Cfg, rep: Rep | None, S0, rec_a, rec_k, rec_u, q, k, v, alpha, beta, prec=64,
                 b=None):
    """One token in readout form from a fixed base; returns (o, (a, k~, u))."""
    g = cfg.dk if cfg.gate else 1
    n = 0 if rec_a is None else len(rec_a)
    ra = np.ascontiguousarray(np.zeros((1, g)) if n == 0 else rec_a, dtype=np.float64)
    rk = np.ascontiguousarray(np.zeros((1, cfg.dk)) if n == 0 else rec_k, dtype=np.float64)
    ru = np.ascontiguousarray(np.zeros((1, cfg.dv)) if n == 0 else rec_u, dtype=np.float64)
    o, na, nk, nu = np.zeros(cfg.dv), np.zeros(g), np.zeros(cfg.dk), np.zeros(cfg.dv)
    if rep is None:
        args = [None, None, None, None, None, _p(np.ascontiguousarray(S0, dtype=np.float64))]
    else:
        Kt = np.ascontiguousarray(rep.Kt) if cfg.n_comp else np.zeros((1, cfg.dk))
        Ut = np.ascontiguousarray(rep.Ut) if cfg.n_comp else np.zeros((1, cfg.dv))
        args = [_p(np.ascontiguousarray(rep.Z)), _p(rep.delta), _p(rep.c), _p(Kt), _p(Ut), None]
    bv = _read_vec(cfg, b)
    _fn("readout_step", prec)(C.byref(cfg), *args, _p(ra), _p(rk), _p(ru), n, _p(_f32(q)),
                              _p(_f32(k)), _p(bv), _p(_f32(v)), _p(_f32(np.atleast_1d(alpha))),
                              float(beta), _p(o), _p(na), _p(nk), _p(nu))
    return o, (na, nk, nu)


def reconstruct(cfg: Cfg, rep: Rep | None, S0, rec_a, rec_k, rec_u, prec=64) -> np.ndarray:
    """Window-end state from the base and n buffered records (Eq. (smooth))."""
    g = cfg.dk if cfg.gate else 1
    n = 0 if rec_a is None else len(rec_a)
    ra = np.ascontiguousarray(np.zeros((1, g)) if n == 0 else rec_a, dtype=np.float64)
    rk = np.ascontiguousarray(np.zeros((1, cfg.dk)) if n == 0 else rec_k, dtype=np.float64)
    ru = np.ascontiguousarray(np.zeros((1, cfg.dv)) if n == 0 else rec_u, dtype=np.float64)
    out = np.zeros((cfg.dk, cfg.dv))
    if rep is None:
        args = [None, None, None, None, None, _p(np.ascontiguousarray(S0, dtype=np.float64))]
    else:
        Kt = np.ascontiguousarray(rep.Kt) if cfg.n_comp else np.zeros((1, cfg.dk))
        Ut = np.ascontiguousarray(rep.Ut) if cfg.n_comp else np.zeros((1, cfg.dv))
        args = [_p(np.ascontiguousarray(rep.Z)), _p(rep.delta), _p(rep.c), _p(Kt), _p(Ut), None]
    _fn("reconstruct", prec)(C.byref(cfg), *args, _p(ra), _p(rk), _p(ru), n, _p(out))
    return out


# --------------------------------------------------------------------------
# batched trajectories
# --------------------------------------------------------------------------

def _inputs(tok: dict, tiles: int, T: int, cfg: Cfg):
    g = cfg.dk if cfg.gate else 1
    arrs = {
        "q": _f32(tok["q"]).reshape(tiles, T, cfg.dk),
        "k": _f32(tok["k"]).reshape(tiles, T, cfg.dk),
        "v": _f32(tok["v"]).reshape(tiles, T, cfg.dv),
        "alpha": _f32(tok["alpha"]).reshape(tiles, T, g),
        "beta": _f32(tok["beta"]).reshape(tiles, T),
    }
    if cfg.rule == RULE_GENERAL:
        if "b" not in tok:
            raise ValueError("the general rule needs read vectors tok['b'] [tiles][T][dk]")
        arrs["b"] = _f32(tok["b"]).reshape(tiles, T, cfg.dk)
    st = _Inputs(*[_p(arrs.get(n)) for n in ("q", "k", "v", "alpha", "beta", "b")])
    return st, arrs


def _run_window(name, cfg: Cfg, S_init, tok: dict, snapshots=True, threads=None, prec=64,
                history=False):
    S_init = np.ascontiguousarray(S_init, dtype=np.float64)
    tiles = S_init.shape[0]
    T = np.asarray(tok["q"]).shape[1]
    st, keep = _inputs(tok, tiles, T, cfg)
    g = cfg.dk if cfg.gate else 1
    r = max(cfg.n_comp, 1)
    W = cfg.window
    ns = 1 + T // W
    res = {"o": np.zeros((tiles, T, cfg.dv)), "S_final": np.zeros((tiles, cfg.dk, cfg.dv)),
           "rec_a": np.zeros((tiles, W, g)), "rec_k": np.zeros((tiles, W, cfg.dk)),
           "rec_u": np.zeros((tiles, W, cfg.dv)), "rec_len": np.zeros(tiles, np.int32)}
    if snapshots:
        res.update({"Z": np.zeros((tiles, ns, cfg.dk, cfg.dv), code_dtype(cfg)),
                    "delta": np.zeros((tiles, ns, cfg.dv), np.float32),
                    "c": np.zeros((tiles, ns, cfg.dk), np.float32),
                    "Kt": np.zeros((tiles, ns, r, cfg.dk)), "Ut": np.zeros((tiles, ns, r, cfg.dv))})
    if history:
        res.update({"hist_a": np.zeros((tiles, T, g)), "hist_k": np.zeros((tiles, T, cfg.dk)),
                    "hist_u": np.zeros((tiles, T, cfg.dv))})
    out = _Outputs(*[_p(res.get(n)) for n in ("Z", "delta", "c", "Kt", "Ut", "S_final", "rec_a",
                                             "rec_k", "rec_u", "rec_len", "hist_a", "hist_k",
                                             "hist_u")])
    _fn(name, prec)(C.byref(cfg), tiles, T, _p(S_init), C.byref(st), _p(res["o"]), C.byref(out),
                    threads or default_threads())
    if snapshots:
        res["Kt"] = res["Kt"][:, :, :cfg.n_comp]
        res["Ut"] = res["Ut"][:, :, :cfg.n_comp]
    del keep
    return res


def run_dense(cfg: Cfg, S_init, tok: dict, snapshots=True, threads=None, prec=64,
              history=False) -> dict:
    """Per-window method in dense form over [tiles] independent tiles."""
    return _run_window("run_dense", cfg, S_init, tok, snapshots, threads, prec, history)


def run_readout(cfg: Cfg, S_init, tok: dict, snapshots=True, threads=None, prec=64,
                history=False) -> dict:
    """Per-window method in readout form (the structure a decode kernel follows)."""
    return _run_window("run_readout", cfg, S_init, tok, snapshots, threads, prec, history)


def run_baseline(cfg: Cfg, S_init, tok: dict, mode=STATE_F32, threads=None, prec=64,
                 want_o=True):
    """Unquantized recurrence; the state is rounded per `mode` after each token."""
    S_init = np.ascontiguousarray(S_init, dtype=np.float64)
    tiles = S_init.shape[0]
    T = np.asarray(tok["q"]).shape[1]
    st, keep = _inputs(tok, tiles, T, cfg)
    o = np.zeros((tiles, T, cfg.dv)) if want_o else None
    S_final = np.zeros((tiles, cfg.dk, cfg.dv))
    _fn("run_baseline", prec)(C.byref(cfg), tiles, T, _p(S_init), C.byref(st), _p(o), _p(S_final),
                              mode, threads or default_threads())
    del keep
    return o, S_final


def run_drift(cfg: Cfg, S_init, tok: dict, every: int, threads=None, prec=64):
    """Relative state and output drift of the quantized trajectory from fp32."""
    S_init = np.ascontiguousarray(S_init, dtype=np.float64)
    tiles = S_init.shape[0]
    T = np.asarray(tok["q"]).shape[1]
    st, keep = _inputs(tok, tiles, T, cfg)
    nd = T // every
    drift = np.zeros((tiles, nd))
    odrift = np.zeros((tiles, nd))
    _fn("run_drift", prec)(C.byref(cfg), tiles, T, every, _p(S_init), C.byref(st), _p(drift),
                           _p(odrift), threads or default_threads())
    del keep
    return drift, odrift
