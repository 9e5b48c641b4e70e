"""Sub-step streams of the instances that split a token (App. A).

A model whose erase direction differs from its write key, or that applies
several delta-rule steps per token, runs as a sequence of steps of the general
recurrence S_t = D_t S_{t-1} + k~_t (v_t - S_{t-1}^T b_t)^T.  These helpers
turn raw per-token model inputs into such sub-step streams, in the layout of the
oracle's batched drivers ([tiles][steps][...], float32); the GPU tests transpose
the same arrays to the library's step-major layout.  Nothing here computes any
part of the quantized method.

RWKV7, transition Diag(w) - kappa (a . kappa)^T, then the write k v^T: two
sub-steps per token, both under the general rule with the per-channel gate:
  erase: D = Diag(w), write key kappa (beta = 1), b = a . kappa, v = 0;
  write: D = I, write key k (beta = 1), b = 0, v = v.
Both sub-steps take the token's receptance r as the query; the token's output
is that of the write sub-step.

DeltaProduct with n sub-steps (scalar gate, delta rule): sub-step j applies
(I - beta_j k_j k_j^T) and writes beta_j k_j v_j^T; the token's scalar gate
(Gated DeltaProduct) is the decay of the first sub-step, the others take 1.
"""
from __future__ import annotations

import numpy as np


def rwkv7_raw(rng: np.random.Generator, tiles: int, T: int, dk: int, dv: int) -> dict:
    """Per-token RWKV7 inputs, [tiles][T][...] float32: decay w = exp(-e^-0.5
    sigmoid(z)) in (0.545, 1) per key channel, in-context rate a = sigmoid(z),
    removal key kappa, key k and receptance r unit-norm Gaussian, value v
    ~ N(0, I).  One draw of 5 x d_k + d_v normals per token."""
    z = rng.standard_normal((tiles, T, 5 * dk + dv), dtype=np.float32)
    zk = z[..., :5 * dk].reshape(tiles, T, 5, dk)
    one = np.float32(1.0)
    sig = one / (one + np.exp(-zk[:, :, :2]))
    unit = zk[:, :, 2:] / np.sqrt(np.einsum("tsjd,tsjd->tsj", zk[:, :, 2:], zk[:, :, 2:]))[..., None]
    return {
        "w": np.exp(np.float32(-np.exp(-0.5)) * sig[:, :, 0]),
        "a": np.ascontiguousarray(sig[:, :, 1]),
        "kappa": np.ascontiguousarray(unit[:, :, 0]),
        "k": np.ascontiguousarray(unit[:, :, 1]),
        "r": np.ascontiguousarray(unit[:, :, 2]),
        "v": np.ascontiguousarray(z[..., 5 * dk:]),
    }


def _interleave(x0, x1):
    """[tiles][T][...] pair -> [tiles][2T][...], sub-step 2t from x0, 2t+1 from x1."""
    out = np.empty((x0.shape[0], 2 * x0.shape[1]) + x0.shape[2:], np.float32)
    out[:, 0::2], out[:, 1::2] = x0, x1
    return out


def rwkv7_substeps(raw: dict) -> dict:
    """Two general-rule sub-steps per token (per-channel gate)."""
    w, a, kap, k, r, v = (raw[n] for n in ("w", "a", "kappa", "k", "r", "v"))
    tiles, T = w.shape[:2]
    one = np.ones_like(w)
    return {
        "q": _interleave(r, r),
        "k": _interleave(kap, k),
        "b": _interleave((a * kap).astype(np.float32), np.zeros_like(kap)),
        "v": _interleave(np.zeros_like(v), v),
        "alpha": _interleave(w, one),
        "beta": _interleave(np.ones((tiles, T), np.float32), np.ones((tiles, T), np.float32)),
    }


def deltaproduct_substeps(tok: dict, n: int) -> dict:
    """n delta-rule sub-steps per token from per-sub-step q, k, v, beta
    ([tiles][T*n][...]) and a per-token scalar gate alpha ([tiles][T][1])."""
    tiles, Tn = tok["k"].shape[:2]
    T = Tn // n
    alpha = np.ones((tiles, Tn, 1), np.float32)
    alpha[:, 0::n] = tok["alpha"].reshape(tiles, T, 1)
    return {"q": tok["q"], "k": tok["k"], "v": tok["v"], "beta": tok["beta"], "alpha": alpha}


def step_major(x: np.ndarray, batch: int, heads: int) -> np.ndarray:
    """[tiles][steps][...] -> [steps][batch][heads][...] (tiles = batch * heads)."""
    x = np.moveaxis(np.asarray(x), 1, 0)
    return np.ascontiguousarray(x.reshape((x.shape[0], batch, heads) + x.shape[2:]))
