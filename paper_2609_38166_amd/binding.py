"""Thin ctypes binding of libleapquant.so (the C ABI in include/leapquant.h).

Argument marshalling only: torch tensors are passed as raw device pointers and
the current HIP stream; every step runs in the library's HIP kernels.  Loading
fails loudly if the library has not been built -- there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
# The library; LEAPQUANT_LIB may name another build of it (a measurement
# variant made by build.py), which must export the same symbols.
LIB_PATH = os.environ.get("LEAPQUANT_LIB") or os.path.join(_PKG, "libleapquant.so")

LQ_OK, LQ_EINVAL, LQ_EALIGN, LQ_EUNSUPPORTED, LQ_EHIP, LQ_EDEVICE = 0, -1, -2, -3, -4, -5
LQ_GATE_SCALAR, LQ_GATE_DIAG = 0, 1
LQ_CODE_INT8, LQ_CODE_E4M3, LQ_CODE_INT4, LQ_CODE_INT6, LQ_CODE_BF16 = 0, 1, 2, 3, 4
CODE_BITS = {LQ_CODE_INT8: 8, LQ_CODE_E4M3: 8, LQ_CODE_INT4: 4, LQ_CODE_INT6: 6, LQ_CODE_BF16: 16}
LQ_STATE_F32, LQ_STATE_BF16 = 0, 1
LQ_RULE_DELTA, LQ_RULE_ADD, LQ_RULE_GENERAL = 0, 1, 2
LQ_DEVERR_WINDOW_FULL = 1
LQ_DEVERR_BAD_REC_LEN = 2

EXPORTS = ("leapquant_state_bytes", "leapquant_quantize_state", "leapquant_decode_step",
           "leapquant_decode_step_general", "leapquant_decode_step_commit", "leapquant_window_commit",
           "leapquant_baseline_step",
           "leapquant_baseline_step_general", "leapquant_dequantize_state",
           "leapquant_check_error", "leapquant_strerror", "leapquant_last_hip_error")


class LeapQuantError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = f"{where}: {strerror(status)} (status {status})"
        if status == LQ_EHIP:
            msg += f": {_lib().leapquant_last_hip_error().decode()}"
        super().__init__(msg)
        self.status = status


class lq_dims(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "batch", "heads_v", "heads_k", "d_k", "d_v", "window", "n_comp", "power_iters", "gate",
        "code", "smooth", "rule")]


class lq_state(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in (
        "codes", "scale", "smooth", "comp_k", "comp_u", "rec_k", "rec_u", "rec_a", "rec_len", "err")]


_L = None


def _lib():
    global _L
    if _L is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2609_38166_amd/build.py "
                              "(or __graft_entry__.build()); there is no fallback path")
        L = C.CDLL(LIB_PATH)
        vp, i32 = C.c_void_p, C.c_int32
        L.leapquant_state_bytes.argtypes = [vp, vp]
        L.leapquant_quantize_state.argtypes = [vp, vp, vp, vp]
        L.leapquant_decode_step.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.leapquant_decode_step_general.argtypes = [vp] * 10
        L.leapquant_decode_step_commit.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.leapquant_window_commit.argtypes = [vp, vp, vp, vp]
        L.leapquant_baseline_step.argtypes = [vp, vp, i32, vp, vp, vp, vp, vp, vp, vp]
        L.leapquant_baseline_step_general.argtypes = [vp, vp, i32] + [vp] * 8
        L.leapquant_dequantize_state.argtypes = [vp, vp, vp, vp]
        L.leapquant_check_error.argtypes = [vp, vp, vp]
        L.leapquant_strerror.argtypes = [i32]
        L.leapquant_strerror.restype = C.c_char_p
        L.leapquant_last_hip_error.argtypes = []
        L.leapquant_last_hip_error.restype = C.c_char_p
        for n in EXPORTS:
            if n not in ("leapquant_strerror", "leapquant_last_hip_error"):
                getattr(L, n).restype = C.c_int32
        _L = L
    return _L


def lib():
    return _lib()


def strerror(status: int) -> str:
    return _lib().leapquant_strerror(status).decode()


def _check(status: int, where: str):
    if status != LQ_OK:
        raise LeapQuantError(status, where)


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _need(t, nbytes: int, name: str, dtype=None):
    """Marshalling check: a contiguous device tensor (of `dtype`, if given)
    holding at least nbytes.  Raw integer addresses are passed through."""
    if t is None:
        raise ValueError(f"{name} is required")
    if isinstance(t, int):
        return
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{name} holds {have} bytes, the call needs {nbytes}")


def _check_state(dims, st):
    for f, nb in zip(FIELDS, leapquant_state_bytes(dims)):
        if f in ("comp_k", "comp_u") and dims.n_comp == 0:
            continue
        _need(getattr(st, f), nb, f"state.{f}")


def _check_tokens(dims, q, k, v, alpha, beta, o):
    t, tk = dims.batch * dims.heads_v, dims.batch * dims.heads_k
    g = dims.d_k if dims.gate == LQ_GATE_DIAG else 1
    f32 = torch.float32
    _need(q, tk * dims.d_k * 4, "q", f32)
    _need(k, tk * dims.d_k * 4, "k", f32)
    _need(v, t * dims.d_v * 4, "v", f32)
    _need(alpha, t * g * 4, "alpha", f32)
    _need(beta, t * 4, "beta", f32)
    _need(o, t * dims.d_v * 4, "o", f32)


def _check_read(dims, b):
    _need(b, dims.batch * dims.heads_v * dims.d_k * 4, "b", torch.float32)


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def make_dims(batch, heads_v, heads_k=None, window=16, n_comp=4, power_iters=4,
              gate=LQ_GATE_SCALAR, code=LQ_CODE_INT8, smooth=1, d_k=128, d_v=128,
              rule=LQ_RULE_DELTA) -> lq_dims:
    return lq_dims(batch, heads_v, heads_k or heads_v, d_k, d_v, window, n_comp, power_iters, gate,
                   code, smooth, rule)


FIELDS = ("codes", "scale", "smooth", "comp_k", "comp_u", "rec_k", "rec_u", "rec_a", "rec_len", "err")


def leapquant_state_bytes(dims: lq_dims) -> list[int]:
    out = (C.c_size_t * 10)()
    _check(_lib().leapquant_state_bytes(C.byref(dims), out), "leapquant_state_bytes")
    return list(out)


@dataclass
class State:
    """Device buffers of the quantized state, allocated by torch (caller-owned).
    The FP16 buffers are float16 tensors (the C ABI sees their bits as uint16)."""
    dims: lq_dims
    codes: torch.Tensor
    scale: torch.Tensor
    smooth: torch.Tensor
    comp_k: torch.Tensor
    comp_u: torch.Tensor
    rec_k: torch.Tensor
    rec_u: torch.Tensor
    rec_a: torch.Tensor
    rec_len: torch.Tensor
    err: torch.Tensor

    @classmethod
    def empty(cls, dims: lq_dims, device="cuda") -> "State":
        B, Hv, dk, dv = dims.batch, dims.heads_v, dims.d_k, dims.d_v
        r, W = dims.n_comp, dims.window
        g = dk if dims.gate == LQ_GATE_DIAG else 1
        kw = {"device": device}
        return cls(
            dims,
            torch.zeros((B, Hv, dv, dk * CODE_BITS[dims.code] // 8), dtype=torch.uint8, **kw),
            torch.zeros((B, Hv, dv), dtype=torch.float32, **kw),
            torch.zeros((B, Hv, dk), dtype=torch.float32, **kw),
            torch.zeros((B, Hv, max(r, 1), dk), dtype=torch.float16, **kw),
            torch.zeros((B, Hv, max(r, 1), dv), dtype=torch.float16, **kw),
            torch.zeros((B, Hv, W, dk), dtype=torch.float16, **kw),
            torch.zeros((B, Hv, W, dv), dtype=torch.float16, **kw),
            torch.zeros((B, Hv, W, g), dtype=torch.float16, **kw),
            torch.zeros((B, Hv), dtype=torch.int32, **kw),
            torch.zeros((4,), dtype=torch.int32, **kw),
        )

    def struct(self) -> lq_state:
        return lq_state(*[getattr(self, f).data_ptr() for f in FIELDS])

    def requests(self, b0: int, b1: int) -> "State":
        """Requests b0 .. b1-1 as views into this state (every array starts at
        tile b0 * heads_v; the error word is shared), with dims for b1 - b0
        requests: a group that runs on its own schedule or stream."""
        if not 0 <= b0 < b1 <= self.dims.batch:
            raise ValueError(f"request range [{b0}, {b1}) outside [0, {self.dims.batch})")
        d = lq_dims.from_buffer_copy(self.dims)
        d.batch = b1 - b0
        return State(d, *[self.err if f == "err" else getattr(self, f)[b0:b1] for f in FIELDS])

    def nbytes(self) -> int:
        return sum(getattr(self, f).numel() * getattr(self, f).element_size() for f in FIELDS)


def leapquant_quantize_state(dims: lq_dims, S: torch.Tensor, st: State, stream=None):
    _check_state(dims, st)
    _need(S, dims.batch * dims.heads_v * dims.d_v * dims.d_k * 4, "S", torch.float32)
    s = st.struct()
    _check(_lib().leapquant_quantize_state(C.byref(dims), _ptr(S), C.byref(s), _stream(stream)),
           "leapquant_quantize_state")


def leapquant_decode_step(dims: lq_dims, st: State, q, k, v, alpha, beta, o, stream=None):
    _check_state(dims, st)
    _check_tokens(dims, q, k, v, alpha, beta, o)
    s = st.struct()
    _check(_lib().leapquant_decode_step(C.byref(dims), C.byref(s), _ptr(q), _ptr(k), _ptr(v),
                                        _ptr(alpha), _ptr(beta), _ptr(o), _stream(stream)),
           "leapquant_decode_step")


def leapquant_decode_step_commit(dims: lq_dims, st: State, q, k, v, alpha, beta, o, stream=None):
    """Decode step, then the commit of every tile whose window it filled, in one
    launch."""
    _check_state(dims, st)
    _check_tokens(dims, q, k, v, alpha, beta, o)
    s = st.struct()
    _check(_lib().leapquant_decode_step_commit(C.byref(dims), C.byref(s), _ptr(q), _ptr(k), _ptr(v),
                                               _ptr(alpha), _ptr(beta), _ptr(o), _stream(stream)),
           "leapquant_decode_step_commit")


def leapquant_decode_step_general(dims: lq_dims, st: State, q, k, b, v, alpha, beta, o,
                                  stream=None):
    """Decode step with the read vectors b [B][heads_v][d_k] given (dims.rule
    must be LQ_RULE_GENERAL)."""
    _check_state(dims, st)
    _check_tokens(dims, q, k, v, alpha, beta, o)
    _check_read(dims, b)
    s = st.struct()
    _check(_lib().leapquant_decode_step_general(C.byref(dims), C.byref(s), _ptr(q), _ptr(k), _ptr(b),
                                                _ptr(v), _ptr(alpha), _ptr(beta), _ptr(o),
                                                _stream(stream)),
           "leapquant_decode_step_general")


def leapquant_window_commit(dims: lq_dims, st: State, mask=None, stream=None):
    _check_state(dims, st)
    if mask is not None:
        _need(mask, dims.batch * 4, "mask")
    s = st.struct()
    _check(_lib().leapquant_window_commit(C.byref(dims), C.byref(s), _ptr(mask), _stream(stream)),
           "leapquant_window_commit")


def leapquant_baseline_step(dims: lq_dims, S, state_dtype: int, q, k, v, alpha, beta, o,
                            stream=None):
    width = 2 if state_dtype == LQ_STATE_BF16 else 4
    _need(S, dims.batch * dims.heads_v * dims.d_v * dims.d_k * width, "S",
          torch.bfloat16 if state_dtype == LQ_STATE_BF16 else torch.float32)
    _check_tokens(dims, q, k, v, alpha, beta, o)
    _check(_lib().leapquant_baseline_step(C.byref(dims), _ptr(S), state_dtype, _ptr(q), _ptr(k),
                                          _ptr(v), _ptr(alpha), _ptr(beta), _ptr(o),
                                          _stream(stream)),
           "leapquant_baseline_step")


def leapquant_baseline_step_general(dims: lq_dims, S, state_dtype: int, q, k, b, v, alpha, beta, o,
                                    stream=None):
    width = 2 if state_dtype == LQ_STATE_BF16 else 4
    _need(S, dims.batch * dims.heads_v * dims.d_v * dims.d_k * width, "S",
          torch.bfloat16 if state_dtype == LQ_STATE_BF16 else torch.float32)
    _check_tokens(dims, q, k, v, alpha, beta, o)
    _check_read(dims, b)
    _check(_lib().leapquant_baseline_step_general(C.byref(dims), _ptr(S), state_dtype, _ptr(q),
                                                  _ptr(k), _ptr(b), _ptr(v), _ptr(alpha), _ptr(beta),
                                                  _ptr(o), _stream(stream)),
           "leapquant_baseline_step_general")


def leapquant_dequantize_state(dims: lq_dims, st: State, S_out, stream=None):
    _check_state(dims, st)
    _need(S_out, dims.batch * dims.heads_v * dims.d_v * dims.d_k * 4, "S_out", torch.float32)
    s = st.struct()
    _check(_lib().leapquant_dequantize_state(C.byref(dims), C.byref(s), _ptr(S_out),
                                             _stream(stream)),
           "leapquant_dequantize_state")


def leapquant_check_error(st: State, stream=None) -> int:
    """Synchronise, return the sticky device error bits and clear them."""
    s = st.struct()
    bits = C.c_int32(0)
    status = _lib().leapquant_check_error(C.byref(s), _stream(stream), C.byref(bits))
    if status not in (LQ_OK, LQ_EDEVICE):
        raise LeapQuantError(status, "leapquant_check_error")
    return bits.value


class Prepared:
    """A call with its ctypes arguments built once, for tight timing loops."""

    def __init__(self, fn, *args):
        self.fn, self.args = fn, args

    def __call__(self):
        status = self.fn(*self.args)
        if status != LQ_OK:
            raise LeapQuantError(status, self.fn.__name__)


def prepare_decode(dims, st: State, q, k, v, alpha, beta, o, stream=None) -> Prepared:
    _check_state(dims, st)
    _check_tokens(dims, q, k, v, alpha, beta, o)
    s = st.struct()
    st._keep = s
    return Prepared(_lib().leapquant_decode_step, C.byref(dims), C.byref(s), _ptr(q), _ptr(k),
                    _ptr(v), _ptr(alpha), _ptr(beta), _ptr(o), _stream(stream))


def prepare_commit(dims, st: State, mask=None, stream=None) -> Prepared:
    _check_state(dims, st)
    if mask is not None:
        _need(mask, dims.batch * 4, "mask")
    s = st.struct()
    st._keep_c = s
    return Prepared(_lib().leapquant_window_commit, C.byref(dims), C.byref(s), _ptr(mask),
                    _stream(stream))
