"""Pins of the CPU oracle against what the paper and the mathematics fix.

Recurrence (Sec. 3.1 Eq. (general), App. A): the native GDN / KDA updates, the
additive rows, the general read-vector rule and the split-token instances
(RWKV7 as erase + write, DeltaProduct as n Householder sub-steps) against
explicit matrix forms, the delta-rule write, degenerate gates.  Quantizer (Secs. 3.3-3.4, App. B.3):
exhaustive code search, error bounds, scaling / sign / permutation symmetry,
Eckart-Young optimality of the fitted tokens.  Window method (Sec. 3.2,
App. B.1-B.3): unrolling equals the recurrence, W=1 without tokens is the naive
per-step scheme (Eq. (naive)), readout form equals dense form, the deviation
recursion (Eq. (deviation)) holds with errors only at window ends.
"""
import numpy as np
import pytest

from tests import brute


def rel(a, b):
    return float(np.linalg.norm(np.asarray(a) - np.asarray(b)) / max(np.linalg.norm(b), 1e-300))


def unit(rng, d):
    x = rng.standard_normal(d)
    return (x / np.linalg.norm(x)).astype(np.float32)


def f32(x):
    return np.asarray(x, dtype=np.float32)


# --------------------------------------------------------------------------- O1

@pytest.mark.parametrize("gate", [0, 1])
def test_recurrence_equals_native_gdn_kda(O, gate):
    """GDN: a(I - b k k^T) S + b k v^T;  KDA: (I - b k k^T) Diag(a) S + b k v^T."""
    rng = np.random.default_rng(10 + gate)
    dk, dv = 16, 12
    cfg = O.make_cfg(dk=dk, dv=dv, gate=gate)
    S = rng.standard_normal((dk, dv))
    for _ in range(5):
        q, k, v = unit(rng, dk), unit(rng, dk), f32(rng.standard_normal(dv))
        beta = np.float32(rng.uniform(0.1, 0.9))
        a = f32(rng.uniform(0.5, 1.0, dk if gate else 1))
        kk, bb = k.astype(np.float64), np.float64(beta)
        D = np.diag(a.astype(np.float64)) if gate else a[0] * np.eye(dk)
        P = np.eye(dk) - bb * np.outer(kk, kk)
        native = (D @ P @ S if not gate else P @ D @ S) + bb * np.outer(kk, v.astype(np.float64))
        S_new, o = O.recurrent_step(cfg, S, q, k, v, a, beta)
        assert rel(S_new, native) < 1e-13
        assert rel(o, native.T @ q.astype(np.float64)) < 1e-13
        S = native


@pytest.mark.parametrize("gate", [0, 1])
def test_additive_instances_native_forms(O, gate):
    """Rows of the instance table with b_t = 0 (App. A): S_t = D_t S + k~ v^T with no
    read of the previous state -- Mamba2 (scalar decay), GLA / RWKV6 / HGRN2
    (per-channel decay); with D = I and beta = 1 the state of linear attention is
    the plain sum of k v^T."""
    rng = np.random.default_rng(14 + gate)
    dk, dv = 16, 12
    cfg = O.make_cfg(dk=dk, dv=dv, gate=gate, rule=O.RULE_ADD)
    S = rng.standard_normal((dk, dv))
    for _ in range(5):
        q, k, v = unit(rng, dk), unit(rng, dk), f32(rng.standard_normal(dv))
        beta = np.float32(rng.uniform(0.1, 0.9))
        a = f32(rng.uniform(0.5, 1.0, dk if gate else 1))
        D = np.diag(a.astype(np.float64)) if gate else a[0] * np.eye(dk)
        native = D @ S + np.float64(beta) * np.outer(k.astype(np.float64), v.astype(np.float64))
        S_new, o = O.recurrent_step(cfg, S, q, k, v, a, beta)
        assert rel(S_new, native) < 1e-13
        assert rel(o, native.T @ q.astype(np.float64)) < 1e-13
        S = native
    # linear attention: D = I, beta = 1 -> S_T = S_0 + sum_t k_t v_t^T
    cl = O.make_cfg(dk=dk, dv=dv, gate=0, rule=O.RULE_ADD)
    S0 = rng.standard_normal((dk, dv))
    S, acc = S0.copy(), S0.copy()
    for _ in range(6):
        q, k, v = unit(rng, dk), unit(rng, dk), f32(rng.standard_normal(dv))
        S, _ = O.recurrent_step(cl, S, q, k, v, f32([1.0]), 1.0)
        acc += np.outer(k.astype(np.float64), v.astype(np.float64))
    assert rel(S, acc) < 1e-14


@pytest.mark.parametrize("gate", [0, 1])
def test_general_rule_special_cases(O, gate):
    """General rule (read vector given): b = D_t k reproduces the delta rule (up
    to the fp32 rounding of the product a k), b = 0 the additive rule exactly,
    in the recurrence, the dense window step and the readout form from a
    quantized base (exact records, so that no FP16 rounding of a correction can
    flip on that last-bit difference)."""
    rng = np.random.default_rng(17 + gate)
    dk, dv = 16, 12
    cg, cd, ca = (O.make_cfg(dk=dk, dv=dv, gate=gate, n_comp=2, window=8, round_records=0, rule=r)
                  for r in (O.RULE_GENERAL, O.RULE_DELTA, O.RULE_ADD))
    S = _state(rng, dk, dv)
    rep = O.quantize(cg, S)
    ra, rk, ru = [], [], []
    for _ in range(4):
        q, k, v = unit(rng, dk), unit(rng, dk), f32(rng.standard_normal(dv))
        beta = np.float32(rng.uniform(0.1, 0.9))
        a = f32(rng.uniform(0.5, 1.0, dk if gate else 1))
        bk = f32(a * k)
        z = np.zeros(dk, np.float32)
        for fn in (O.recurrent_step, O.window_step):
            g1, g0 = fn(cg, S, q, k, v, a, beta, b=bk), fn(cd, S, q, k, v, a, beta)
            assert rel(g1[0], g0[0]) < 1e-6 and rel(g1[1], g0[1]) < 1e-6
            z1, z0 = fn(cg, S, q, k, v, a, beta, b=z), fn(ca, S, q, k, v, a, beta)
            assert np.array_equal(z1[0], z0[0]) and np.array_equal(z1[1], z0[1])
        recs = (np.array(ra), np.array(rk), np.array(ru)) if ra else (None, None, None)
        o1, n1 = O.readout_step(cg, rep, None, *recs, q, k, v, a, beta, b=bk)
        o0, n0 = O.readout_step(cd, rep, None, *recs, q, k, v, a, beta)
        assert rel(o1, o0) < 1e-6 and rel(n1[2], n0[2]) < 1e-6
        oz, nz = O.readout_step(cg, rep, None, *recs, q, k, v, a, beta, b=z)
        oa, na = O.readout_step(ca, rep, None, *recs, q, k, v, a, beta)
        assert np.array_equal(oz, oa) and np.array_equal(nz[2], na[2])
        ra.append(n0[0]), rk.append(n0[1]), ru.append(n0[2])
        S = O.window_step(cd, S, q, k, v, a, beta)[0]


def test_rwkv7_two_substeps_native_transition(O):
    """RWKV7 (App. A): the erase sub-step (general rule, b = a.kappa, v = 0)
    followed by the pure write (b = 0, D = I) is one token of the native
    transition S_t = (Diag(w) - kappa (a.kappa)^T) S_{t-1} + k v^T, o_t = S_t^T r,
    written here as explicit d_k x d_k matrices.  Checked on the recurrence and
    on both forms of the per-window method (quantization off, exact records),
    with windows that end between the two sub-steps of a token."""
    from tests import instances
    rng = np.random.default_rng(18)
    dk, dv, tiles, T = 16, 12, 2, 11
    raw = instances.rwkv7_raw(rng, tiles, T, dk, dv)
    tok = instances.rwkv7_substeps(raw)
    S0 = rng.standard_normal((tiles, dk, dv))
    o_nat = np.zeros((tiles, T, dv))
    S_nat = S0.copy()
    for i in range(tiles):
        S = S0[i]
        for t in range(T):
            w, a, kap, k, r, v = (raw[n][i, t].astype(np.float64) for n in ("w", "a", "kappa", "k", "r", "v"))
            bvec = f32(raw["a"][i, t] * raw["kappa"][i, t]).astype(np.float64)
            assert np.allclose(bvec, a * kap, rtol=1e-7)
            S = (np.diag(w) - np.outer(kap, bvec)) @ S + np.outer(k, v)
            o_nat[i, t] = S.T @ r
        S_nat[i] = S
    cfg_b = O.make_cfg(dk=dk, dv=dv, gate=1, rule=O.RULE_GENERAL)
    o_ref, S_ref = O.run_baseline(cfg_b, S0, tok, mode=O.STATE_EXACT)
    assert rel(o_ref[:, 1::2], o_nat) < 1e-13
    assert rel(S_ref, S_nat) < 1e-13
    for W in (5, 8):
        cfg = O.make_cfg(dk=dk, dv=dv, window=W, n_comp=2, gate=1, quantize=0, round_records=0,
                         rule=O.RULE_GENERAL)
        for run in (O.run_dense, O.run_readout):
            res = run(cfg, S0, tok, snapshots=False)
            assert rel(res["o"][:, 1::2], o_nat) < 1e-12
            assert rel(res["S_final"], S_nat) < 1e-12
    # the pin separates the plausible misreading that reads b against the decayed
    # state, (D S)^T b, from the paper's S^T b
    Sw = S0[0]
    for t in range(T):
        w, kap, k, v = (raw[n][0, t].astype(np.float64) for n in ("w", "kappa", "k", "v"))
        bvec = f32(raw["a"][0, t] * raw["kappa"][0, t]).astype(np.float64)
        A = np.diag(w) @ Sw
        Sw = A - np.outer(kap, A.T @ bvec) + np.outer(k, v)
    assert rel(Sw, S_nat[0]) > 1e-3


def test_deltaproduct_substeps_native_householder_product(O):
    """DeltaProduct (App. A), n = 3 delta-rule sub-steps per token with the
    token's scalar gate on the first: S_t = a_t P_n..P_1 S_{t-1} + sum_j
    P_n..P_{j+1} beta_j k_j v_j^T with P_j = I - beta_j k_j k_j^T, as explicit
    matrix products.  Recurrence and both window forms."""
    from tests import instances
    rng = np.random.default_rng(19)
    dk, dv, tiles, T, n = 16, 12, 2, 7, 3
    q = rng.standard_normal((tiles, T * n, dk))
    k = rng.standard_normal((tiles, T * n, dk))
    sub = {"q": f32(q / np.linalg.norm(q, axis=-1, keepdims=True)),
           "k": f32(k / np.linalg.norm(k, axis=-1, keepdims=True)),
           "v": f32(rng.standard_normal((tiles, T * n, dv))),
           "beta": f32(rng.uniform(0.0, 2.0, (tiles, T * n))),      # negative eigenvalues allowed
           "alpha": f32(rng.uniform(0.6, 1.0, (tiles, T, 1)))}
    tok = instances.deltaproduct_substeps(sub, n)
    S0 = rng.standard_normal((tiles, dk, dv))
    o_nat, S_nat = np.zeros((tiles, T, dv)), S0.copy()
    for i in range(tiles):
        S = S0[i]
        for t in range(T):
            js = range(t * n, (t + 1) * n)
            Ps = [np.eye(dk) - np.float64(sub["beta"][i, j]) *
                  np.outer(sub["k"][i, j].astype(np.float64), sub["k"][i, j].astype(np.float64)) for j in js]
            prod = np.eye(dk)
            for P in Ps:
                prod = P @ prod
            Snew = np.float64(sub["alpha"][i, t, 0]) * prod @ S
            for m, j in enumerate(js):
                tail = np.eye(dk)
                for P in Ps[m + 1:]:
                    tail = P @ tail
                Snew += tail @ (np.float64(sub["beta"][i, j]) * np.outer(sub["k"][i, j].astype(np.float64),
                                                                          sub["v"][i, j].astype(np.float64)))
            S = Snew
            o_nat[i, t] = S.T @ sub["q"][i, t * n + n - 1].astype(np.float64)
        S_nat[i] = S
    cfg_b = O.make_cfg(dk=dk, dv=dv, gate=0)
    o_ref, S_ref = O.run_baseline(cfg_b, S0, tok, mode=O.STATE_EXACT)
    assert rel(o_ref[:, n - 1::n], o_nat) < 1e-12
    assert rel(S_ref, S_nat) < 1e-12
    cfg = O.make_cfg(dk=dk, dv=dv, window=4, n_comp=2, gate=0, quantize=0, round_records=0)
    for run in (O.run_dense, O.run_readout):
        res = run(cfg, S0, tok, snapshots=False)
        assert rel(res["o"][:, n - 1::n], o_nat) < 1e-12
        assert rel(res["S_final"], S_nat) < 1e-12


def test_delta_rule_writes_value_exactly(O):
    """alpha = 1, beta = 1, |k| = 1: after the write S^T k = v (the delta rule)."""
    rng = np.random.default_rng(11)
    cfg = O.make_cfg(dk=32, dv=24)
    S = rng.standard_normal((32, 24))
    k, q, v = unit(rng, 32), unit(rng, 32), f32(rng.standard_normal(24))
    S_new, _ = O.recurrent_step(cfg, S, q, k, v, f32([1.0]), 1.0)
    kk = k.astype(np.float64)
    err = S_new.T @ kk - v.astype(np.float64) * (kk @ kk) - (1 - kk @ kk) * (S.T @ kk)
    assert np.max(np.abs(err)) < 1e-12


def test_degenerate_gates(O):
    rng = np.random.default_rng(12)
    cfg = O.make_cfg(dk=8, dv=8, gate=1)
    S = rng.standard_normal((8, 8))
    q, k, v = unit(rng, 8), unit(rng, 8), f32(rng.standard_normal(8))
    a = f32(rng.uniform(0.3, 1, 8))
    S1, o = O.recurrent_step(cfg, S, q, k, v, a, 0.0)             # beta = 0: pure decay
    assert np.array_equal(S1, a.astype(np.float64)[:, None] * S)
    S2, _ = O.recurrent_step(cfg, S, q, k, v, f32(np.ones(8)), 0.0)  # identity: state unchanged
    assert np.array_equal(S2, S)
    # KDA with equal channels is GDN
    cg = O.make_cfg(dk=8, dv=8, gate=0)
    S3, o3 = O.recurrent_step(cg, S, q, k, v, f32([0.7]), 0.4)
    S4, o4 = O.recurrent_step(cfg, S, q, k, v, f32(np.full(8, 0.7)), 0.4)
    assert np.array_equal(S3, S4) and np.array_equal(o3, o4)


def test_state_rounding_modes(O):
    rng = np.random.default_rng(13)
    cfg = O.make_cfg(dk=16, dv=16)
    S = rng.standard_normal((16, 16))
    q, k, v = unit(rng, 16), unit(rng, 16), f32(rng.standard_normal(16))
    S32, _ = O.recurrent_step(cfg, S, q, k, v, f32([0.9]), 0.5, mode=O.STATE_F32)
    assert np.array_equal(S32, S32.astype(np.float32).astype(np.float64))
    Sb, _ = O.recurrent_step(cfg, S, q, k, v, f32([0.9]), 0.5, mode=O.STATE_BF16)
    bits = Sb.astype(np.float32).view(np.uint32)
    assert np.all(bits & 0xFFFF == 0)
    Se, _ = O.recurrent_step(cfg, S, q, k, v, f32([0.9]), 0.5)
    assert rel(Sb, Se) < 4e-3 and rel(S32, Se) < 1e-6


# --------------------------------------------------------------------------- O2

def _state(rng, dk, dv, outliers=True):
    S = sum(np.outer(rng.standard_normal(dk), rng.standard_normal(dv)) * 0.7 ** i for i in range(6))
    S = S + 0.3 * rng.standard_normal((dk, dv))
    if outliers:
        S[rng.choice(dk, 2, replace=False), :] *= 20
        S[:, rng.choice(dv, 2, replace=False)] *= 20
    return S


QMAX = {O_CODE: q for O_CODE, q in ((0, 127), (2, 7), (3, 31))}   # INT8, INT4, INT6


@pytest.mark.parametrize("code", [0, 2, 3])
@pytest.mark.parametrize("smooth", [0, 1])
@pytest.mark.parametrize("r", [0, 2])
def test_quantizer_matches_bruteforce(O, smooth, r, code):
    """Tiny tiles: every code is the nearest of all 2*qmax+1 integer codes
    (exhaustive; qmax = 127, 31, 7 for 8, 6, 4 bits), and the tokens /
    smoothing / scales agree with an independent float64 statement."""
    rng = np.random.default_rng(20 + smooth + 2 * r + 5 * code)
    for dk, dv in ((4, 4), (8, 4), (8, 8)):
        S = _state(rng, dk, dv, outliers=False)
        cfg = O.make_cfg(dk=dk, dv=dv, n_comp=r, power_iters=3, smooth=smooth, code=code)
        rep = O.quantize(cfg, S)
        Zb, db, cb, Kb, Ub = brute.quantize(S, r, 3, bool(smooth), qmax=QMAX[code])
        assert np.allclose(rep.Kt, Kb, rtol=0, atol=0) and np.allclose(rep.Ut, Ub, rtol=1e-3, atol=1e-6)
        assert np.array_equal(rep.c, cb)
        assert np.array_equal(rep.delta, db)
        Z = rep.Z.view(np.int8).astype(int)
        # codes may differ only where x/delta sits on a rounding boundary to fp32 precision
        M = S - rep.Kt.T @ rep.Ut
        t = (M / rep.c.astype(np.float64)[:, None]) / (rep.delta.astype(np.float64)[None, :])
        near_tie = np.abs(np.abs(t - np.floor(t)) - 0.5) < 1e-5
        assert np.all((Z == Zb) | near_tie)


@pytest.mark.parametrize("code", [0, 1, 2, 3])
def test_quantizer_error_bounds_and_extremes(O, code):
    rng = np.random.default_rng(30 + code)
    S = _state(rng, 128, 128)
    cfg = O.make_cfg(n_comp=8 if code == 2 else 4, code=code)
    rep = O.quantize(cfg, S)
    M = S - rep.Kt.T @ rep.Ut                     # residual the codes represent
    Rc = M / rep.c.astype(np.float64)[:, None]
    if code != 1:
        q = QMAX[code]
        Z = rep.Z.view(np.int8).astype(np.float64)
        assert np.all(np.abs(Z) <= q)
        # every column reaches +-qmax at its largest-magnitude entry
        assert np.all(np.abs(Z).max(axis=0) == q)
        err = np.abs(Rc - Z * rep.delta.astype(np.float64))
        assert np.all(err <= rep.delta.astype(np.float64) * (0.5 + 1e-5))
    else:
        vals = O.e4m3_to_f32(rep.Z).astype(np.float64)
        assert np.all(np.isfinite(vals)) and np.all(np.abs(vals).max(axis=0) == 448.0)
        x = Rc / rep.delta.astype(np.float64)
        # nearest e4m3 value: relative error at most half a 3-bit ulp (or half the
        # subnormal step 2^-9 near zero)
        bound = np.maximum(np.abs(x) * 2.0 ** -4, 2.0 ** -10) * (1 + 1e-5)
        assert np.all(np.abs(x - vals) <= bound)
    deq = O.dequantize(cfg, rep)
    assert rel(deq, S) < {0: 0.01, 1: 0.03, 2: 0.15, 3: 0.03}[code]


def test_quantizer_power_of_four_scaling(O):
    """Q(4^e S): identical codes and tokens' key vectors; c, delta scale by 2^e,
    value vectors by 4^e -- every step is an exact power-of-two scaling."""
    rng = np.random.default_rng(40)
    S = _state(rng, 128, 128)
    cfg = O.make_cfg(n_comp=4)
    a = O.quantize(cfg, S)
    for e in (-2, 3):
        b = O.quantize(cfg, S * 4.0 ** e)
        assert np.array_equal(a.Z, b.Z)
        assert np.array_equal(a.Kt, b.Kt)
        assert np.array_equal(a.Ut * 4.0 ** e, b.Ut)
        assert np.array_equal(a.c * np.float32(2.0 ** e), b.c)
        assert np.array_equal(a.delta * np.float32(2.0 ** e), b.delta)


def test_quantizer_sign_symmetry(O):
    rng = np.random.default_rng(41)
    S = _state(rng, 128, 128)
    cfg = O.make_cfg(n_comp=4)
    a, b = O.quantize(cfg, S), O.quantize(cfg, -S)
    assert np.array_equal(a.Z.view(np.int8), -b.Z.view(np.int8))
    assert np.array_equal(a.Kt, b.Kt) and np.array_equal(a.Ut, -b.Ut)
    assert np.array_equal(a.c, b.c) and np.array_equal(a.delta, b.delta)


def test_quantizer_permutation_equivariance(O):
    rng = np.random.default_rng(42)
    S = _state(rng, 128, 128)
    cfg = O.make_cfg(n_comp=4)
    pk, pv = rng.permutation(128), rng.permutation(128)
    a, b = O.quantize(cfg, S), O.quantize(cfg, S[pk][:, pv])
    Za, Zb = a.Z.view(np.int8), b.Z.view(np.int8)
    assert np.mean(Za[pk][:, pv] == Zb) > 0.9999
    assert rel(b.Kt.T @ b.Ut, (a.Kt.T @ a.Ut)[pk][:, pv]) < 1e-6
    assert np.allclose(a.c[pk], b.c, rtol=1e-6) and np.allclose(a.delta[pv], b.delta, rtol=1e-6)


def test_compensators_reach_eckart_young(O):
    """With many power-iteration sweeps the r tokens are the best rank-r
    approximation (Sec. 3.3: the argmin over rank-one / rank-r factors)."""
    rng = np.random.default_rng(43)
    U, _ = np.linalg.qr(rng.standard_normal((128, 128)))
    V, _ = np.linalg.qr(rng.standard_normal((128, 128)))
    sig = np.concatenate([[40, 25, 15, 9, 5.5], 3.0 * 0.97 ** np.arange(123)])
    S = (U * sig) @ V.T
    for r in (1, 4):
        cfg = O.make_cfg(n_comp=r, power_iters=400)
        rep = O.quantize(cfg, S)
        u, s, vt = np.linalg.svd(S)
        best = (u[:, :r] * s[:r]) @ vt[:r]
        assert rel(rep.Kt.T @ rep.Ut, best) < 2e-3       # FP16 rounding of the factors
        resid = np.linalg.norm(S - rep.Kt.T @ rep.Ut)
        assert abs(resid / np.sqrt(np.sum(s[r:] ** 2)) - 1) < 2e-3


def test_compensators_configured_iters_near_optimal(O):
    """Diagnostic of the configured 4 sweeps on outlier states: the residual is
    within a few percent of the Eckart-Young bound."""
    rng = np.random.default_rng(44)
    for _ in range(3):
        S = _state(rng, 128, 128)
        for r in (4, 8):
            rep = O.quantize(O.make_cfg(n_comp=r, power_iters=4), S)
            s = np.linalg.svd(S, compute_uv=False)
            resid = np.linalg.norm(S - rep.Kt.T @ rep.Ut)
            assert resid <= 1.10 * np.sqrt(np.sum(s[r:] ** 2))


def test_rank_one_state_recovered(O):
    rng = np.random.default_rng(45)
    a, b = rng.standard_normal(128), rng.standard_normal(128) * 3
    S = np.outer(a, b)
    rep = O.quantize(O.make_cfg(n_comp=1), S)
    assert rel(rep.Kt.T @ rep.Ut, S) < 1e-3          # FP16 factors
    assert rel(O.dequantize(O.make_cfg(n_comp=1), rep), S) < 1e-5   # codes absorb the rest


def test_zero_state_and_zero_columns(O):
    cfg = O.make_cfg(n_comp=4)
    rep = O.quantize(cfg, np.zeros((128, 128)))
    assert not rep.Z.any() and not rep.delta.any() and not rep.Kt.any() and not rep.Ut.any()
    assert np.array_equal(O.dequantize(cfg, rep), np.zeros((128, 128)))
    rng = np.random.default_rng(46)
    S = rng.standard_normal((128, 128))
    S[:, [3, 77]] = 0
    rep = O.quantize(O.make_cfg(n_comp=0), S)
    assert rep.delta[3] == 0 and rep.delta[77] == 0 and not rep.Z[:, [3, 77]].any()


def test_smoothing_balances_rows(O):
    """c_k is the square root of the key row's mean |R|: a residual whose rows have
    constant magnitude m_k gets c_k = sqrt(m_k), flat rows give constant c, and
    smoothing lowers the reconstruction error of a row-imbalanced residual."""
    rng = np.random.default_rng(47)
    m = np.exp(rng.uniform(-3, 3, 128))
    S = m[:, None] * np.sign(rng.standard_normal((128, 128)))
    rep = O.quantize(O.make_cfg(n_comp=0), S)
    assert np.allclose(rep.c, np.sqrt(m).astype(np.float32), rtol=1e-7)
    flat = np.sign(rng.standard_normal((128, 128))) * 0.25
    assert np.all(O.quantize(O.make_cfg(n_comp=0), flat).c == np.float32(0.5))
    T = rng.standard_normal((128, 128)) * m[:, None]
    e1 = rel(O.dequantize(O.make_cfg(n_comp=0, smooth=1), O.quantize(O.make_cfg(n_comp=0, smooth=1), T)), T)
    e0 = rel(O.dequantize(O.make_cfg(n_comp=0, smooth=0), O.quantize(O.make_cfg(n_comp=0, smooth=0), T)), T)
    assert e1 < e0


# --------------------------------------------------------------------------- O3 / O4

def _tokens(rng, tiles, T, dk, dv, gate):
    g = dk if gate else 1
    q = rng.standard_normal((tiles, T, dk))
    k = rng.standard_normal((tiles, T, dk))
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    return {"q": f32(q), "k": f32(k), "v": f32(rng.standard_normal((tiles, T, dv))),
            "alpha": f32(np.exp(-0.1 * np.logaddexp(0, rng.standard_normal((tiles, T, g))))),
            "beta": f32(1 / (1 + np.exp(-rng.standard_normal((tiles, T)))))}


@pytest.mark.parametrize("gate", [0, 1])
@pytest.mark.parametrize("W", [1, 3, 16])
@pytest.mark.parametrize("rule", [0, 1, 2])
def test_window_unrolling_equals_recurrence(O, gate, W, rule):
    """Quantization off and exact records: the per-window method (both forms) is
    the recurrence itself (Eq. (window) follows from Eq. (record) by induction),
    for the delta rule, the b_t = 0 rows of the instance table and the general
    read vector."""
    rng = np.random.default_rng(50 + W + gate + 7 * rule)
    dk = dv = 32
    S0 = rng.standard_normal((3, dk, dv))
    tok = _tokens(rng, 3, 37, dk, dv, gate)
    if rule == 2:
        tok["b"] = f32(0.7 * rng.standard_normal((3, 37, dk)) / np.sqrt(dk))
    cfg = O.make_cfg(dk=dk, dv=dv, window=W, n_comp=2, gate=gate, quantize=0, round_records=0,
                     rule=rule)
    o_ref, S_ref = O.run_baseline(cfg, S0, tok, mode=O.STATE_EXACT)
    for run in (O.run_dense, O.run_readout):
        res = run(cfg, S0, tok, snapshots=False)
        assert rel(res["o"], o_ref) < 1e-12
        assert rel(res["S_final"], S_ref) < 1e-12
    res32 = O.run_readout(cfg, S0, tok, snapshots=False, prec=32)
    assert rel(res32["o"], o_ref) < 2e-5


@pytest.mark.parametrize("smooth", [0, 1])
def test_window_one_without_tokens_is_naive_per_step(O, smooth):
    """W = 1, r = 0, exact records: Eq. (naive) -- decay and delta update from the
    dequantized previous state, then re-quantize after every token."""
    rng = np.random.default_rng(60 + smooth)
    dk = dv = 32
    S0 = rng.standard_normal((1, dk, dv))
    tok = _tokens(rng, 1, 12, dk, dv, 0)
    cfg = O.make_cfg(dk=dk, dv=dv, window=1, n_comp=0, smooth=smooth, round_records=0)
    res = O.run_dense(cfg, S0, tok)
    S = O.dequantize(cfg, O.quantize(cfg, S0[0]))
    for t in range(12):
        q, k, v = (tok[n][0, t].astype(np.float64) for n in ("q", "k", "v"))
        a, b = np.float64(tok["alpha"][0, t, 0]), np.float64(tok["beta"][0, t])
        Snew = a * S + np.outer(b * k, v - S.T @ (a * k))
        o = Snew.T @ q
        assert rel(res["o"][0, t], o) < 1e-12
        rep = O.quantize(cfg, Snew)
        assert np.array_equal(rep.Z, res["Z"][0, t + 1])
        S = O.dequantize(cfg, rep)


@pytest.mark.parametrize("gate,code,r,smooth", [(0, 0, 4, 1), (1, 0, 8, 1), (0, 1, 8, 1),
                                                (1, 0, 0, 0), (0, 0, 2, 0)])
def test_readout_form_equals_dense_form(O, gate, code, r, smooth):
    """Buffered readout (App. B.2-B.3) from the fixed quantized base equals the
    dense step-by-step window, at every token and every window end (the delta
    rule, and the b_t = 0 rule on the odd cases)."""
    rng = np.random.default_rng(70 + gate + 2 * code + r)
    dk = dv = 64
    S0 = _state(rng, dk, dv)[None].repeat(2, 0) * rng.uniform(0.5, 2, (2, 1, 1))
    tok = _tokens(rng, 2, 45, dk, dv, gate)
    cfg = O.make_cfg(dk=dk, dv=dv, window=16, n_comp=r, gate=gate, code=code, smooth=smooth,
                     rule=(r + code + gate) % 2)
    d, b = O.run_dense(cfg, S0, tok), O.run_readout(cfg, S0, tok)
    assert rel(b["o"], d["o"]) < 1e-10
    assert np.mean(b["Z"] == d["Z"]) > 0.9999
    assert rel(b["S_final"], d["S_final"]) < 1e-10
    assert np.array_equal(b["rec_len"], d["rec_len"])
    n = int(d["rec_len"][0])
    assert rel(b["rec_u"][:, :n], d["rec_u"][:, :n]) < 1e-12


@pytest.mark.parametrize("gate", [0, 1])
def test_readout_form_equals_dense_form_general_rule(O, gate):
    """The same agreement under the general rule: RWKV7 sub-steps (per-channel
    gate) and, for the scalar gate, read vectors drawn independently of the key."""
    from tests import instances
    rng = np.random.default_rng(75 + gate)
    dk = dv = 64
    S0 = _state(rng, dk, dv)[None].repeat(2, 0) * rng.uniform(0.5, 2, (2, 1, 1))
    if gate:
        tok = instances.rwkv7_substeps(instances.rwkv7_raw(rng, 2, 23, dk, dv))
    else:
        tok = _tokens(rng, 2, 46, dk, dv, 0)
        tok["b"] = f32(0.8 * rng.standard_normal((2, 46, dk)) / np.sqrt(dk))
    cfg = O.make_cfg(dk=dk, dv=dv, window=16, n_comp=4, gate=gate, rule=O.RULE_GENERAL)
    d, b = O.run_dense(cfg, S0, tok), O.run_readout(cfg, S0, tok)
    assert rel(b["o"], d["o"]) < 1e-10
    assert np.mean(b["Z"] == d["Z"]) > 0.9999
    assert rel(b["S_final"], d["S_final"]) < 1e-10
    n = int(d["rec_len"][0])
    assert rel(b["rec_u"][:, :n], d["rec_u"][:, :n]) < 1e-12


def test_window_trajectory_matches_bruteforce(O):
    """A 3-window trajectory on 4x4 and 8x8 tiles equals the independent float64
    brute-force statement (exhaustive code search)."""
    rng = np.random.default_rng(80)
    for d in (4, 8):
        S0 = _state(rng, d, d, outliers=False)
        tok = _tokens(rng, 1, 9, d, d, 1)
        cfg = O.make_cfg(dk=d, dv=d, window=3, n_comp=1, power_iters=3, gate=1)
        res = O.run_dense(cfg, S0[None], tok)
        toks = [{n: tok[n][0, t] for n in ("q", "k", "v", "alpha", "beta")} for t in range(9)]
        outs, reps = brute.window_trajectory(S0, toks, 3, 1, 3, True)
        assert rel(res["o"][0], outs) < 1e-9
        for s, rp in enumerate(reps):
            assert np.mean(res["Z"][0, s].view(np.int8) == rp[0]) >= 0.95
            assert rel(res["Kt"][0, s].T @ res["Ut"][0, s], rp[3].T @ rp[4]) < 1e-6


def test_reconstruct_equals_dense_window_end(O):
    rng = np.random.default_rng(90)
    dk = dv = 32
    cfg = O.make_cfg(dk=dk, dv=dv, window=64, n_comp=2, gate=1)
    S0 = _state(rng, dk, dv)
    rep = O.quantize(cfg, S0)
    S = O.dequantize(cfg, rep)
    tok = _tokens(rng, 1, 7, dk, dv, 1)
    ra, rk, ru = [], [], []
    for t in range(7):
        S, _, (a, k, u) = O.window_step(cfg, S, tok["q"][0, t], tok["k"][0, t], tok["v"][0, t],
                                        tok["alpha"][0, t], tok["beta"][0, t])
        ra.append(a), rk.append(k), ru.append(u)
    R = O.reconstruct(cfg, rep, None, np.array(ra), np.array(rk), np.array(ru))
    assert rel(R, S) < 1e-12


def test_deviation_recursion(O):
    """App. B.1: E_t = D_t E_{t-1} - k~_t (E_{t-1}^T b_t)^T + eps_t, and under
    per-window quantization eps_t = 0 except at window ends."""
    rng = np.random.default_rng(91)
    dk = dv = 16
    W, T = 4, 13
    cfg = O.make_cfg(dk=dk, dv=dv, window=W, n_comp=1, gate=1, round_records=0)
    ex = O.make_cfg(dk=dk, dv=dv, gate=1)
    S0 = _state(rng, dk, dv)
    tok = _tokens(rng, 1, T, dk, dv, 1)
    F = S0.copy()                                          # FP reference trajectory
    S = O.dequantize(cfg, O.quantize(cfg, S0))            # window trajectory
    E = S - F
    for t in range(T):
        q, k, v, a, b = (tok[n][0, t] for n in ("q", "k", "v", "alpha", "beta"))
        F, _ = O.recurrent_step(ex, F, q, k, v, a, b)
        S_pre, _, _ = O.window_step(cfg, S, q, k, v, a, b)   # S_t before quantization
        if (t + 1) % W == 0:
            S_new = O.dequantize(cfg, O.quantize(cfg, S_pre))
        else:
            S_new = S_pre
        eps = S_new - S_pre
        kk, aa = k.astype(np.float64), a.astype(np.float64)
        pred = aa[:, None] * E - np.outer(np.float64(b) * kk, E.T @ (aa * kk)) + eps
        E = S_new - F
        assert np.max(np.abs(E - pred)) <= 1e-12 * max(1.0, np.abs(F).max())
        if (t + 1) % W:
            assert not eps.any()
        else:
            assert np.abs(eps).max() > 0
        S = S_new


def test_per_window_drifts_less_than_per_step(O):
    """The paper's central observation (Sec. 3.2): quantizing once per window keeps
    the state far closer to the FP32 trajectory than re-quantizing every token."""
    rng = np.random.default_rng(92)
    dk = dv = 64
    S0 = np.stack([_state(rng, dk, dv) for _ in range(4)])
    tok = _tokens(rng, 4, 256, dk, dv, 0)
    d_step, _ = O.run_drift(O.make_cfg(dk=dk, dv=dv, window=1, n_comp=0, smooth=0), S0, tok, 64)
    d_win, _ = O.run_drift(O.make_cfg(dk=dk, dv=dv, window=16, n_comp=4), S0, tok, 64)
    assert np.mean(d_win) < 0.5 * np.mean(d_step)


# --------------------------------------------------------------------------- BF16 state (code 4)

def _bf16(x):
    """fp32 -> bf16 (round to nearest even) -> float64, by torch (not the oracle)."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).to(
        torch.float64).numpy()


def test_bf16_state_quantizer_is_bf16_rounding(O):
    """Code 4 keeps the state itself in BF16: the window-end quantizer is the
    round-to-nearest-even BF16 rounding of the fp32 value, with unit scales and no
    smoothing.  Checked against torch's conversion, ties and subnormals included."""
    import torch
    rng = np.random.default_rng(120)
    dk = dv = 32
    S = rng.standard_normal((dk, dv)) * np.exp(rng.uniform(-30, 30, (dk, dv)))
    b = np.float32(rng.standard_normal(64)).view(np.uint32)
    ties = ((b & 0xFFFF0000) | 0x8000).view(np.float32)          # exactly half-way between two bf16
    S.flat[:64] = ties
    S.flat[64:72] = np.float32([1e-39, -3e-40, 0.0, -0.0, 1e-45, 3.4e38, -1.17e-38, 7e-39])
    cfg = O.make_cfg(dk=dk, dv=dv, n_comp=0, code=O.CODE_BF16)
    rep = O.quantize(cfg, S)
    ref = torch.from_numpy(S.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert rep.Z.dtype == np.uint16 and np.array_equal(rep.Z, ref)
    assert np.all(rep.delta == 1.0) and np.all(rep.c == 1.0)
    assert np.array_equal(O.dequantize(cfg, rep), _bf16(S.astype(np.float32)))


@pytest.mark.parametrize("gate", [0, 1])
@pytest.mark.parametrize("W", [1, 5])
def test_bf16_per_window_is_recurrence_rounded_at_window_ends(O, gate, W):
    """The per-window BF16 state (Sec. 3.2, the BF16 rows of the ablation): the
    unquantized recurrence, written out with the explicit delta-rule formulas,
    with the state rounded to BF16 through fp32 at the start and after every W
    tokens (exact records, so only the window-end rounding differs from the
    recurrence)."""
    rng = np.random.default_rng(121 + gate + W)
    dk = dv = 32
    T = 3 * W + 2
    S0 = rng.standard_normal((1, dk, dv))
    tok = _tokens(rng, 1, T, dk, dv, gate)
    cfg = O.make_cfg(dk=dk, dv=dv, window=W, n_comp=0, gate=gate, code=O.CODE_BF16, smooth=0,
                     round_records=0)
    res = O.run_dense(cfg, S0, tok, snapshots=True)
    S = _bf16(S0[0].astype(np.float32))
    assert np.array_equal(O.dequantize(cfg, O.Rep(res["Z"][0, 0], res["delta"][0, 0], res["c"][0, 0],
                                                  np.zeros((0, dk)), np.zeros((0, dv)))), S)
    for t in range(T):
        q, k, v = (tok[n][0, t].astype(np.float64) for n in ("q", "k", "v"))
        a = tok["alpha"][0, t].astype(np.float64)
        b = np.float64(tok["beta"][0, t])
        A = (a[:, None] if gate else a[0]) * S
        S = A + np.outer(b * k, v - A.T @ k)
        assert rel(res["o"][0, t], S.T @ q) < 1e-12
        if (t + 1) % W == 0:
            S = _bf16(S.astype(np.float32))
            bits = (S.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
            assert np.array_equal(res["Z"][0, (t + 1) // W], bits)


def test_bf16_per_step_is_the_bf16_baseline(O):
    """W = 1 with exact records: the per-window BF16 state after every token is
    the per-step BF16 baseline's state (the state rounded to BF16 after each
    update), bit for bit."""
    rng = np.random.default_rng(125)
    dk = dv = 32
    S0 = _bf16(rng.standard_normal((2, dk, dv)).astype(np.float32))
    tok = _tokens(rng, 2, 17, dk, dv, 1)
    cfg = O.make_cfg(dk=dk, dv=dv, window=1, n_comp=0, gate=1, code=O.CODE_BF16, round_records=0)
    res = O.run_dense(cfg, S0, tok, snapshots=False)
    _, S_b = O.run_baseline(cfg, S0, tok, mode=O.STATE_BF16)
    assert np.array_equal(res["S_final"], S_b)


@pytest.mark.parametrize("gate", [0, 1])
def test_bf16_readout_form_equals_dense_form(O, gate):
    rng = np.random.default_rng(126 + gate)
    dk = dv = 64
    S0 = _state(rng, dk, dv)[None].repeat(2, 0)
    tok = _tokens(rng, 2, 40, dk, dv, gate)
    cfg = O.make_cfg(dk=dk, dv=dv, window=16, n_comp=0, gate=gate, code=O.CODE_BF16, smooth=0)
    d, b = O.run_dense(cfg, S0, tok), O.run_readout(cfg, S0, tok)
    assert rel(b["o"], d["o"]) < 1e-10
    assert np.mean(b["Z"] == d["Z"]) > 0.9999
    assert rel(b["S_final"], d["S_final"]) < 1e-10


# --------------------------------------------------------------------------- drift (App. B.1)

def test_drift_is_zero_without_quantization(O):
    """Quantization off and exact records: in the fp32 build the window path and
    the fp32 recurrence take the same operations, so the drift is exactly 0."""
    rng = np.random.default_rng(130)
    dk = dv = 32
    S0 = rng.standard_normal((3, dk, dv)).astype(np.float32).astype(np.float64)
    tok = _tokens(rng, 3, 64, dk, dv, 1)
    cfg = O.make_cfg(dk=dk, dv=dv, window=16, n_comp=4, gate=1, quantize=0, round_records=0)
    drift, odrift = O.run_drift(cfg, S0, tok, 8, prec=32)
    assert drift.shape == (3, 8) and not drift.any() and not odrift.any()


@pytest.mark.parametrize("gate", [0, 1])
def test_drift_bookkeeping_against_explicit_fp32_recurrence(O, gate):
    """run_drift's sampled drift equals ||S_window(t) - F(t)|| / ||F(t)|| with the
    window state taken from the dense trajectory after t tokens and F the fp32
    recurrence written out here (fp64 update, rounded to fp32 after every token),
    at window ends and inside windows; and likewise for the outputs."""
    rng = np.random.default_rng(131 + gate)
    dk = dv = 16
    T, W, every = 12, 3, 2
    S0 = rng.standard_normal((1, dk, dv)).astype(np.float32).astype(np.float64)
    tok = _tokens(rng, 1, T, dk, dv, gate)
    cfg = O.make_cfg(dk=dk, dv=dv, window=W, n_comp=1, gate=gate)
    drift, odrift = O.run_drift(cfg, S0, tok, every)
    F = S0[0].copy()
    for t in range(T):
        q, k, v = (tok[n][0, t].astype(np.float64) for n in ("q", "k", "v"))
        a = tok["alpha"][0, t].astype(np.float64)
        A = (a[:, None] if gate else a[0]) * F
        F = (A + np.outer(np.float64(tok["beta"][0, t]) * k, v - A.T @ k)).astype(np.float32).astype(np.float64)
        if (t + 1) % every == 0:
            sub = {n_: x[:, :t + 1] for n_, x in tok.items()}
            win = O.run_dense(cfg, S0, sub, snapshots=False)
            Sw, ow = win["S_final"][0], win["o"][0, t]
            assert abs(drift[0, (t + 1) // every - 1] - rel(Sw, F)) <= 1e-12 * rel(Sw, F)
            assert abs(odrift[0, (t + 1) // every - 1] - rel(ow, F.T @ q)) <= 1e-12 * rel(ow, F.T @ q)
