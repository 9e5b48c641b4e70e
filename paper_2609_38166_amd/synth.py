"""Seeded synthetic decode workloads.

This module only draws inputs: token streams (q, k, v, beta, decay), the
outlier pattern injected into the initial state, and the workload shapes.  It
holds none of the method's arithmetic, so both the HIP path (tests, benchmark)
and the CPU oracle (tests) can be fed from it.

Distributions (stand-ins for the hidden states of the paper's GDN / KDA models,
whose weights and datasets are not available), all computed in float32:
  q, k  ~ N(0, I_d), then L2-normalised (the models normalise q and k);
  v     ~ N(0, I_d);
  beta  = sigmoid(N(0, 1));
  decay = exp(-0.1 * softplus(N(0, 1))): one scalar per token for the scalar
          gate, d_k independent draws per token for the per-channel gate
          (Workload.gate_scale replaces 0.1 for a long-memory variant).

Every tile (request b, value head h) owns two independent PCG64 streams seeded
from SeedSequence([seed, phase, kind, b, head]): kind 0 is the key stream of
key head h_k (q then k per token), kind 1 the value stream of value head h_v
(v, beta-logit, decay-logit(s) per token).  Phase 0 drives the prefill that
builds the initial state, phase 1 the decode steps, phase 2 the outliers.  Any
tile can therefore be regenerated on its own, and drawing a trajectory in
chunks gives the same numbers as drawing it at once.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace

import numpy as np

GATE_SCALAR, GATE_DIAG = 0, 1
CODE_INT8, CODE_E4M3, CODE_INT4, CODE_INT6, CODE_BF16 = 0, 1, 2, 3, 4
PHASE_PREFILL, PHASE_DECODE, PHASE_OUTLIER = 0, 1, 2


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    heads_v: int
    heads_k: int
    steps: int                # decode tokens
    window: int               # W
    n_comp: int               # r
    gate: int
    code: int = CODE_INT8
    dk: int = 128
    dv: int = 128
    prefill: int = 512        # tokens of the unquantized prefill that builds the initial state
    power_iters: int = 4
    smooth: int = 1           # residual smoothing on (1) or c = 1 (0)
    rule: int = 0             # read vector: delta rule (0), b_t = 0 (1), given with the token (2)
    outliers: str = "all"     # "all": every tile; "frac": 5 % of tiles; "none"
    outlier_factor: float = 20.0
    gate_scale: float = 0.1           # decay = exp(-gate_scale * softplus(N(0, 1)))
    seed: int = 20260000
    extra: dict = field(default_factory=dict)

    @property
    def tiles(self) -> int:
        return self.batch * self.heads_v

    @property
    def g(self) -> int:
        return self.dk if self.gate == GATE_DIAG else 1

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# The workload shapes of the evaluation: a tiny GDN case, a Qwen3-Next-like GDN
# layer with grouped key heads, the Kimi-Linear-like KDA layer (the headline
# throughput case), a large-batch GDN stress case and a long trace.
WORKLOADS = {
    "gdn_tiny": Workload("gdn_tiny", 4, 4, 4, 256, 16, 4, GATE_SCALAR, seed=20260000),
    "gdn_qwen3next": Workload("gdn_qwen3next", 64, 32, 16, 1024, 64, 8, GATE_SCALAR, seed=20260001),
    "kda_kimi": Workload("kda_kimi", 256, 32, 32, 512, 64, 8, GATE_DIAG, seed=20260002),
    "gdn_stress": Workload("gdn_stress", 1024, 32, 32, 128, 32, 8, GATE_SCALAR, outliers="frac",
                           seed=20260003),
    "gdn_long": Workload("gdn_long", 32, 16, 16, 32768, 128, 8, GATE_SCALAR, seed=20260004),
    # 8192 cached prefix snapshots x 32 heads, quantized in bulk
    "bulk_quantize": Workload("bulk_quantize", 8192, 32, 32, 0, 1, 8, GATE_SCALAR, seed=20260005),
}
# the KDA layer with the lower-bit residual codes (same inputs, r = 8)
WORKLOADS["kda_kimi_int4"] = WORKLOADS["kda_kimi"].with_(name="kda_kimi_int4", code=CODE_INT4)
WORKLOADS["kda_kimi_int6"] = WORKLOADS["kda_kimi"].with_(name="kda_kimi_int6", code=CODE_INT6)
# the per-window BF16 state (no Compensator Tokens, no smoothing) at the headline shape
WORKLOADS["kda_kimi_bf16w"] = WORKLOADS["kda_kimi"].with_(name="kda_kimi_bf16w", code=CODE_BF16, n_comp=0,
                                                          smooth=0)


def _threads(n=None) -> int:
    return max(1, min(n or (os.cpu_count() or 1), 16))


def _gen(*words) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(w) for w in words])))


def vtile_index(wl: Workload, b: int, hv: int) -> int:
    return b * wl.heads_v + hv


def khead_of(wl: Workload, hv: int) -> int:
    """Key head read by value head hv: consecutive value heads share one key head."""
    return hv // (wl.heads_v // wl.heads_k)


class Streams:
    """Token streams of one phase for a set of value-head tiles.

    ``draw(n)`` returns the next n tokens of every stream, step-major:
      q, k      float32 [n][n_ktiles][dk]  (one row per distinct (b, key head))
      v         float32 [n][n_vtiles][dv]
      alpha     float32 [n][n_vtiles][g]
      beta      float32 [n][n_vtiles]
    ``ktile_of_vtile[i]`` maps value tile i to its key tile column.
    """

    def __init__(self, wl: Workload, phase: int, vtiles=None, threads=None):
        self.wl = wl
        if vtiles is None:
            vtiles = range(wl.tiles)
        self.vtiles = np.asarray(list(vtiles), dtype=np.int64)
        bs, hvs = self.vtiles // wl.heads_v, self.vtiles % wl.heads_v
        keys = sorted({(int(b), khead_of(wl, int(h))) for b, h in zip(bs, hvs)})
        self.ktiles = keys
        kidx = {kt: i for i, kt in enumerate(keys)}
        self.ktile_of_vtile = np.array([kidx[(int(b), khead_of(wl, int(h)))] for b, h in zip(bs, hvs)])
        self._kg = [_gen(wl.seed, phase, 0, b, hk) for b, hk in keys]
        self._vg = [_gen(wl.seed, phase, 1, int(b), int(h)) for b, h in zip(bs, hvs)]
        self._pool = ThreadPoolExecutor(_threads(threads))

    def draw(self, n: int) -> dict:
        wl = self.wl
        nk, nv = len(self._kg), len(self._vg)
        q = np.empty((n, nk, wl.dk), np.float32)
        k = np.empty((n, nk, wl.dk), np.float32)
        v = np.empty((n, nv, wl.dv), np.float32)
        beta = np.empty((n, nv), np.float32)
        alpha = np.empty((n, nv, wl.g), np.float32)

        def fill_k(lo, hi):
            buf = np.empty((hi - lo, n, 2, wl.dk), np.float32)
            for i in range(lo, hi):
                self._kg[i].standard_normal((n, 2, wl.dk), dtype=np.float32, out=buf[i - lo])
            buf /= np.sqrt(np.einsum("stjd,stjd->stj", buf, buf))[..., None]
            q[:, lo:hi] = buf[:, :, 0].transpose(1, 0, 2)
            k[:, lo:hi] = buf[:, :, 1].transpose(1, 0, 2)

        def fill_v(lo, hi):
            buf = np.empty((hi - lo, n, wl.dv + 1 + wl.g), np.float32)
            for i in range(lo, hi):
                self._vg[i].standard_normal(buf.shape[1:], dtype=np.float32, out=buf[i - lo])
            v[:, lo:hi] = buf[:, :, :wl.dv].transpose(1, 0, 2)
            zb = buf[:, :, wl.dv]
            beta[:, lo:hi] = (np.float32(1.0) / (np.float32(1.0) + np.exp(-zb))).T
            za = buf[:, :, wl.dv + 1:]
            # softplus(z) = max(z, 0) + log1p(exp(-|z|))
            sp = np.maximum(za, np.float32(0.0)) + np.log1p(np.exp(-np.abs(za)))
            alpha[:, lo:hi] = np.exp(np.float32(-wl.gate_scale) * sp).transpose(1, 0, 2)

        def spans(total, per=64):
            return [(lo, min(lo + per, total)) for lo in range(0, total, per)]

        futs = [self._pool.submit(fill_k, lo, hi) for lo, hi in spans(nk)]
        futs += [self._pool.submit(fill_v, lo, hi) for lo, hi in spans(nv)]
        for f in futs:
            f.result()
        return {"q": q, "k": k, "v": v, "beta": beta, "alpha": alpha}

    def close(self):
        self._pool.shutdown()


def tile_major(wl: Workload, st: Streams, tok: dict) -> dict:
    """Per value-tile arrays [vtiles][n][...] with q, k repeated for heads sharing a key head."""
    kv = st.ktile_of_vtile
    return {"q": np.ascontiguousarray(tok["q"][:, kv].transpose(1, 0, 2)),
            "k": np.ascontiguousarray(tok["k"][:, kv].transpose(1, 0, 2)),
            "v": np.ascontiguousarray(tok["v"].transpose(1, 0, 2)),
            "alpha": np.ascontiguousarray(tok["alpha"].transpose(1, 0, 2)),
            "beta": np.ascontiguousarray(tok["beta"].T)}


def step_major_full(wl: Workload, tok: dict) -> dict:
    """Views for a full-batch stream set (vtiles = all tiles in order):
    q, k [n][B][Hk][dk]; v [n][B][Hv][dv]; alpha [n][B][Hv](*[dk]); beta [n][B][Hv]."""
    n = tok["v"].shape[0]
    B, Hv, Hk = wl.batch, wl.heads_v, wl.heads_k
    out = {
        "q": tok["q"].reshape(n, B, Hk, wl.dk),
        "k": tok["k"].reshape(n, B, Hk, wl.dk),
        "v": tok["v"].reshape(n, B, Hv, wl.dv),
        "beta": tok["beta"].reshape(n, B, Hv),
    }
    a = tok["alpha"]
    out["alpha"] = a.reshape(n, B, Hv, wl.dk) if wl.gate == GATE_DIAG else a.reshape(n, B, Hv)
    return out


def outliers(wl: Workload, vtiles=None) -> dict:
    """Outlier lines injected into the initial state.

    Per tile: two distinct key rows and two distinct value columns.  Mode
    "all": every tile, factor `outlier_factor` on each line.  Mode "frac":
    a tile is chosen with probability 0.05 and each of its four lines gets an
    independent factor U[10, 50].  Returns row_f [tiles][dk] and col_f
    [tiles][dv]; the factor at (k, v) is max(row_f[k], col_f[v]) (an "or"
    mask, so a crossing is scaled once, not twice).
    """
    if vtiles is None:
        vtiles = range(wl.tiles)
    vtiles = list(vtiles)
    row_f = np.ones((len(vtiles), wl.dk), np.float32)
    col_f = np.ones((len(vtiles), wl.dv), np.float32)
    if wl.outliers == "none":
        return {"row_f": row_f, "col_f": col_f}
    for i, t in enumerate(vtiles):
        b, h = divmod(int(t), wl.heads_v)
        rng = _gen(wl.seed, PHASE_OUTLIER, 2, b, h)
        pick = rng.random()
        rows = rng.choice(wl.dk, 2, replace=False)
        cols = rng.choice(wl.dv, 2, replace=False)
        if wl.outliers == "frac":
            f = rng.uniform(10.0, 50.0, size=4)
            if pick >= 0.05:
                continue
        else:
            f = np.full(4, wl.outlier_factor)
        row_f[i, rows] = f[:2]
        col_f[i, cols] = f[2:]
    return {"row_f": row_f, "col_f": col_f}


def outlier_factor(out: dict) -> np.ndarray:
    """Dense factor F[tiles][dk][dv] = max(row_f[k], col_f[v])."""
    return np.maximum(out["row_f"][:, :, None], out["col_f"][:, None, :])


def bulk_states(wl: Workload, n_tiles: int, first: int = 0, threads=None) -> np.ndarray:
    """Cached prefix states for the bulk-quantize workload, S^T layout [n][dv][dk].

    A cached state is a decayed sum of rank-one writes with a few dominant
    directions; it is drawn directly (no recurrence): 16 rank-one terms with
    geometrically falling weight plus N(0, 0.05^2) noise, then the outlier
    lines of the tile.  Tile t uses SeedSequence([seed, 3, t]).
    """
    out = np.empty((n_tiles, wl.dv, wl.dk), np.float32)
    w = 0.8 ** np.arange(16)

    def one(i):
        t = first + i
        rng = _gen(wl.seed, 3, t)
        a = rng.standard_normal((16, wl.dk))
        b = rng.standard_normal((16, wl.dv))
        a /= np.linalg.norm(a, axis=1, keepdims=True)
        s = (b.T * w) @ a + 0.05 * rng.standard_normal((wl.dv, wl.dk))
        rows = rng.choice(wl.dk, 2, replace=False)
        cols = rng.choice(wl.dv, 2, replace=False)
        f = np.ones((wl.dv, wl.dk))
        f[:, rows] = wl.outlier_factor
        f[cols, :] = wl.outlier_factor
        out[i] = (s * f).astype(np.float32)

    with ThreadPoolExecutor(_threads(threads)) as ex:
        list(ex.map(one, range(n_tiles)))
    return out
