"""Pins for the fp64 oracle against things other than itself.

Each test checks the oracle against a library routine (numpy float64
matmul, numpy.quantile), brute force in pure Python on tiny shapes, closed
forms, exact algebraic identities of the method (Eq. 1 == Eq. 5, the
shared-index property of Eq. 4, index set = all / empty), or exact
metamorphic relations. Shapes are non-square so a transposed operand fails.
"""
import math

import numpy as np
import pytest

from workloads import WORKLOADS, bf16_round, bf16_to_f32
from workloads.synth import T_CALIB, make_layer, make_predictor, make_tokens

import oracle


def f64(a):
    return bf16_to_f32(a).astype(np.float64)


def small_layer(d_model=24, d_ff=40, sigma=0.3, B=3, seed=7):
    L = make_layer(900 + seed, d_model, d_ff, sigma)
    x = make_tokens(900 + seed, B, d_model)
    return x, L


def np_reference(x, L):
    """Independent numpy float64 evaluation of Sec. 3 quantities."""
    X, G, U, D = f64(x), f64(L["W_gate"]), f64(L["W_up"]), f64(L["W_down"])
    u = X @ U.T
    g = X @ G.T
    h = g / (1.0 + np.exp(-g))
    s = u * h
    return u, g, h, s, s @ D


# --------------------------------------------------------------- dense, Eq. (1)

@pytest.mark.parametrize("shape", [(24, 40, 3), (256, 688, 2), (8, 16, 1)])
def test_dense_matches_numpy_float64(shape):
    dm, dff, B = shape
    x, L = small_layer(dm, dff, 0.3 if dm < 100 else 0.02, B)
    y = oracle.dense(x, L["W_gate"], L["W_up"], L["W_down"])
    *_, yr = np_reference(x, L)
    assert y.shape == (B, dm)
    np.testing.assert_allclose(y, yr, rtol=1e-12, atol=1e-14 * np.abs(yr).max())


def test_coefficients_match_numpy_float64():
    x, L = small_layer()
    u, g, s = oracle.coefficients(x, L["W_gate"], L["W_up"])
    ur, gr, hr, sr, _ = np_reference(x, L)
    np.testing.assert_allclose(u, ur, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(g, gr, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(s, sr, rtol=1e-12, atol=1e-15)


def test_one_hot_input_closed_form():
    """x = e_j: u[i] = W_up[i, j] exactly; with a large gate column, SiLU(g) = g exactly
    in double (e^-g underflows next to 1), so s[i] = W_up[i, j] * W_gate[i, j] and
    y = sum_i s[i] W_down^T[i]."""
    dm, dff, j = 16, 12, 5
    rng = np.random.default_rng(3)
    Wg = rng.standard_normal((dff, dm)).astype(np.float32)
    Wg[:, j] = 64.0 + np.arange(dff, dtype=np.float32)   # g = 64..75: exp(-g) < 2^-92
    L = {"W_gate": bf16_round(Wg),
         "W_up": bf16_round(rng.standard_normal((dff, dm)).astype(np.float32)),
         "W_down": bf16_round(rng.standard_normal((dff, dm)).astype(np.float32))}
    xo = np.zeros(dm, np.float32)
    xo[j] = 1.0
    x = bf16_round(xo)[None]
    u, g, s = oracle.coefficients(x, L["W_gate"], L["W_up"])
    np.testing.assert_array_equal(u[0], f64(L["W_up"])[:, j])
    np.testing.assert_array_equal(g[0], f64(L["W_gate"])[:, j])
    np.testing.assert_array_equal(s[0], f64(L["W_up"])[:, j] * f64(L["W_gate"])[:, j])
    y = oracle.dense(x, L["W_gate"], L["W_up"], L["W_down"])
    expect = np.zeros(dm)
    for i in range(dff):  # ascending, as the oracle sums
        expect += s[0, i] * f64(L["W_down"])[i]
    np.testing.assert_array_equal(y[0], expect)


# ------------------------------------------------------------------ SiLU

def test_silu_closed_forms():
    assert oracle.silu(0.0) == 0.0
    assert oracle.silu(100.0) == 100.0
    assert oracle.silu(-1000.0) == 0.0 or abs(oracle.silu(-1000.0)) < 1e-300
    assert not math.isnan(oracle.silu(-1e6))
    for z in (-7.5, -1.0, -0.25, 0.5, 2.0, 9.0):
        assert oracle.silu(z) == pytest.approx(z / (1.0 + math.exp(-z)), rel=1e-15)
    # SiLU(z) - SiLU(-z) = z (sigmoid(z) + sigmoid(-z) = 1)
    for z in (0.3, 1.7, 4.0):
        assert oracle.silu(z) - oracle.silu(-z) == pytest.approx(z, rel=1e-15)


# -------------------------------------------------- brute force on tiny shapes

def brute(x, L, mode, thld, A_t=None, B_t=None):
    """Pure-Python loops straight from Sec. 3 / Eq. (5) / Eq. (6)."""
    X, G, U, D = (f64(a).tolist() for a in (x, L["W_gate"], L["W_up"], L["W_down"]))
    B, dm, dff = len(X), len(X[0]), len(U)

    def dot(a, b):
        t = 0.0
        for p, q in zip(a, b):
            t += p * q
        return t

    def silu(z):
        return z / (1.0 + math.exp(-z)) if z >= 0 else z * math.exp(z) / (1.0 + math.exp(z))

    u = [[dot(X[b], U[i]) for i in range(dff)] for b in range(B)]
    g = [[dot(X[b], G[i]) for i in range(dff)] for b in range(B)]
    s = [[u[b][i] * silu(g[b][i]) for i in range(dff)] for b in range(B)]
    if mode == "mono":
        c = [[abs(v) for v in row] for row in u]
    elif mode == "dual_ideal":
        c = [[abs(v) for v in row] for row in s]
    else:
        A, Bm = f64(A_t).tolist(), f64(B_t).tolist()
        lat = [[dot(X[b], A[r]) for r in range(len(A))] for b in range(B)]
        c = [[dot(lat[b], Bm[i]) for i in range(dff)] for b in range(B)]
    idx = [i for i in range(dff) if any(c[b][i] > thld for b in range(B))]
    y = [[0.0] * dm for _ in range(B)]
    for b in range(B):
        for i in idx:
            for j in range(dm):
                y[b][j] += s[b][i] * D[i][j]
    return np.array(idx, dtype=np.int32), np.array(y)


@pytest.mark.parametrize("mode", ["mono", "dual_ideal", "dual_pred"])
@pytest.mark.parametrize("B", [1, 3])
def test_variants_match_brute_force(mode, B):
    dm, dff, dr = 8, 16, 4
    L = make_layer(950, dm, dff, 0.5)
    P = make_predictor(950, dm, dr, dff, 0.5)
    x = make_tokens(950, B, dm)
    if mode == "mono":
        c = np.abs(oracle.coefficients(x, L["W_gate"], L["W_up"])[0])
    elif mode == "dual_ideal":
        c = np.abs(oracle.coefficients(x, L["W_gate"], L["W_up"])[2])
    else:
        c = oracle.predictor(x, P["A_t"], P["B_t"])[1]
    thld = float(np.float32(np.quantile(c[0], 0.6)))
    idx_b, y_b = brute(x, L, mode, thld, P["A_t"], P["B_t"])
    if mode == "mono":
        idx, y, _ = oracle.ffn_mono(x, L["W_gate"], L["W_up"], L["W_down"], thld)
    elif mode == "dual_ideal":
        idx, y, _ = oracle.ffn_dual_ideal(x, L["W_gate"], L["W_up"], L["W_down"], thld)
    else:
        idx, y, _ = oracle.ffn_dual_pred(x, L["W_gate"], L["W_up"], L["W_down"], P["A_t"],
                                         P["B_t"], thld)
    np.testing.assert_array_equal(idx, idx_b)
    assert 0 < len(idx) < dff
    np.testing.assert_allclose(y, y_b, rtol=1e-12, atol=1e-13)


# ------------------------------------- identities of the method (Eq. 1, 4, 5)

@pytest.mark.parametrize("variant", ["mono", "dual_ideal"])
def test_all_indices_reproduce_dense_bitwise(variant):
    """thld = -inf selects every neuron: Eq. (5) over all i is Eq. (1)."""
    x, L = small_layer(B=2)
    fn = oracle.ffn_mono if variant == "mono" else oracle.ffn_dual_ideal
    idx, y, _ = fn(x, L["W_gate"], L["W_up"], L["W_down"], -np.inf)
    np.testing.assert_array_equal(idx, np.arange(40))
    np.testing.assert_array_equal(y, oracle.dense(x, L["W_gate"], L["W_up"], L["W_down"]))


def test_pred_all_indices_reproduce_dense():
    x, L = small_layer(B=2)
    P = make_predictor(907, 24, 6, 40, 0.3)
    idx, y, _ = oracle.ffn_dual_pred(x, L["W_gate"], L["W_up"], L["W_down"], P["A_t"], P["B_t"],
                                     -np.inf)
    assert len(idx) == 40
    np.testing.assert_array_equal(y, oracle.dense(x, L["W_gate"], L["W_up"], L["W_down"]))


@pytest.mark.parametrize("variant", ["mono", "dual_ideal"])
def test_empty_index_gives_zero(variant):
    x, L = small_layer()
    fn = oracle.ffn_mono if variant == "mono" else oracle.ffn_dual_ideal
    idx, y, _ = fn(x, L["W_gate"], L["W_up"], L["W_down"], np.inf)
    assert len(idx) == 0
    np.testing.assert_array_equal(y, 0.0)


def test_shared_index_property():
    """Eq. (4): masking s outside IDX then a dense down product equals the gathered
    evaluation where gate, up and down are all restricted to IDX."""
    x, L = small_layer(B=2)
    *_, s, _ = np_reference(x, L)
    idx = np.array([1, 4, 5, 9, 17, 33, 39], dtype=np.int32)
    y_g, s_c = oracle.ffn_on_idx(x, L["W_gate"], L["W_up"], L["W_down"], idx)
    masked = np.zeros_like(s)
    masked[:, idx] = s[:, idx]
    np.testing.assert_allclose(y_g, masked @ f64(L["W_down"]), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(s_c, s[:, idx], rtol=1e-13, atol=1e-16)


def test_dropped_terms_are_the_residual():
    """y_dense - y_sparse = sum over i not in IDX of s_i W_down^T[i], within the a-priori
    fp64 summation bound gamma_n * sum |s_i W_ij|."""
    w = WORKLOADS["tiny_256x688"]
    L = w.layer()
    x = w.tokens(2)
    _, _, s = oracle.coefficients(x, L["W_gate"], L["W_up"])
    thld = float(np.float32(np.quantile(np.abs(s[0]), 0.9)))
    idx, y_sp, _ = oracle.ffn_dual_ideal(x, L["W_gate"], L["W_up"], L["W_down"], thld)
    drop = np.setdiff1d(np.arange(w.d_ff), idx).astype(np.int32)
    y_drop = oracle.combine(s, L["W_down"], drop)
    y_dense = oracle.dense(x, L["W_gate"], L["W_up"], L["W_down"])
    n = w.d_ff
    gamma = n * 2.0 ** -53 / (1 - n * 2.0 ** -53)
    bound = 3 * gamma * (np.abs(s) @ np.abs(f64(L["W_down"])))
    assert np.all(np.abs(y_dense - y_sp - y_drop) <= bound)
    assert np.abs(y_drop).max() > 1e3 * bound.max()  # the check is not vacuous


def test_union_over_batch():
    x, L = small_layer(B=3)
    u = oracle.coefficients(x, L["W_gate"], L["W_up"])[0]
    thld = float(np.quantile(np.abs(u), 0.8))
    idx, _, _ = oracle.ffn_mono(x, L["W_gate"], L["W_up"], L["W_down"], thld)
    per = [set(oracle.ffn_mono(x[b:b + 1], L["W_gate"], L["W_up"], L["W_down"], thld)[0].tolist())
           for b in range(3)]
    assert set(idx.tolist()) == set().union(*per)
    assert list(idx) == sorted(idx)
    same = np.repeat(x[:1], 3, axis=0)
    idx3, y3, _ = oracle.ffn_mono(same, L["W_gate"], L["W_up"], L["W_down"], thld)
    idx1, y1, _ = oracle.ffn_mono(x[:1], L["W_gate"], L["W_up"], L["W_down"], thld)
    np.testing.assert_array_equal(idx3, idx1)
    for b in range(3):
        np.testing.assert_array_equal(y3[b], y1[0])


def test_union_tokens_use_their_own_coefficients():
    """Every token uses all rows of the shared IDX with its own s_b[i]."""
    x, L = small_layer(B=2)
    *_, s, _ = np_reference(x, L)
    thld = float(np.quantile(np.abs(s), 0.85))
    idx, y, _ = oracle.ffn_dual_ideal(x, L["W_gate"], L["W_up"], L["W_down"], thld)
    for b in range(2):
        np.testing.assert_allclose(y[b], s[b, idx] @ f64(L["W_down"])[idx], rtol=1e-12,
                                   atol=1e-15)


# -------------------------------------------------------- metamorphic (exact)

def test_metamorphic_relations_mono():
    x, L = small_layer(B=2)
    u = oracle.coefficients(x, L["W_gate"], L["W_up"])[0]
    thld = float(np.float32(np.quantile(np.abs(u), 0.7)))
    idx, y, _ = oracle.ffn_mono(x, L["W_gate"], L["W_up"], L["W_down"], thld)

    # W_down x 2 -> y x 2 exactly (power-of-two scaling of bf16 is exact)
    D2 = bf16_round(2 * f64(L["W_down"]).astype(np.float32))
    idx2, y2, _ = oracle.ffn_mono(x, L["W_gate"], L["W_up"], D2, thld)
    np.testing.assert_array_equal(idx2, idx)
    np.testing.assert_array_equal(y2, 2 * y)

    # W_up x 2 with thld x 2 -> same IDX, y x 2
    U2 = bf16_round(2 * f64(L["W_up"]).astype(np.float32))
    idx3, y3, _ = oracle.ffn_mono(x, L["W_gate"], U2, L["W_down"], 2 * thld)
    np.testing.assert_array_equal(idx3, idx)
    np.testing.assert_array_equal(y3, 2 * y)

    # W_up -> -W_up: same IDX (|u| unchanged), y -> -y
    Un = bf16_round(-f64(L["W_up"]).astype(np.float32))
    idx4, y4, _ = oracle.ffn_mono(x, L["W_gate"], Un, L["W_down"], thld)
    np.testing.assert_array_equal(idx4, idx)
    np.testing.assert_array_equal(y4, -y)

    # W_gate -> -W_gate changes SiLU asymmetrically: y must change (guards a dropped gate)
    Gn = bf16_round(-f64(L["W_gate"]).astype(np.float32))
    _, y5, _ = oracle.ffn_mono(x, Gn, L["W_up"], L["W_down"], thld)
    assert np.abs(y5 - y).max() > 1e-3 * np.abs(y).max()


@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "dual_pred"])
def test_neuron_permutation(variant):
    """Permuting neurons (rows of all matrices, and of B_t) permutes IDX and leaves y
    unchanged up to summation order."""
    dm, dff, dr = 24, 40, 6
    x, L = small_layer(dm, dff)
    P = make_predictor(908, dm, dr, dff, 0.3)
    perm = np.random.default_rng(5).permutation(dff)
    Lp = {k: v[perm].copy() for k, v in L.items()}
    Pp = {"A_t": P["A_t"], "B_t": P["B_t"][perm].copy()}

    def run(LL, PP, thld):
        if variant == "mono":
            return oracle.ffn_mono(x, LL["W_gate"], LL["W_up"], LL["W_down"], thld)
        if variant == "dual_ideal":
            return oracle.ffn_dual_ideal(x, LL["W_gate"], LL["W_up"], LL["W_down"], thld)
        return oracle.ffn_dual_pred(x, LL["W_gate"], LL["W_up"], LL["W_down"], PP["A_t"],
                                    PP["B_t"], thld)

    coef = {"mono": lambda: np.abs(oracle.coefficients(x, L["W_gate"], L["W_up"])[0]),
            "dual_ideal": lambda: np.abs(oracle.coefficients(x, L["W_gate"], L["W_up"])[2]),
            "dual_pred": lambda: oracle.predictor(x, P["A_t"], P["B_t"])[1]}[variant]()
    thld = float(np.quantile(coef, 0.75))
    idx, y, _ = run(L, P, thld)
    idxp, yp, _ = run(Lp, Pp, thld)
    np.testing.assert_array_equal(np.sort(perm[idxp]), idx)
    np.testing.assert_allclose(yp, y, rtol=1e-12, atol=1e-14)
    assert 0 < len(idx) < dff


# ------------------------------------------------------------- thresholds

def test_quantile_matches_numpy_linear():
    rng = np.random.default_rng(11)
    for n in (1, 2, 7, 688, 11008):
        v = rng.standard_normal(n)
        for k in (0.0, 0.1, 0.5, 0.7, 0.9, 0.99, 1.0):
            assert oracle.quantile_linear(k, v) == pytest.approx(
                np.quantile(v, k, method="linear"), rel=1e-15, abs=1e-300)
    v = np.array([3.0, 1.0, 1.0, 1.0, 2.0])  # ties
    assert oracle.quantile_linear(0.5, v) == np.quantile(v, 0.5)


@pytest.mark.parametrize("n,k", [(688, 0.9), (11008, 0.9), (11008, 0.7), (11008, 0.5),
                                 (14336, 0.9), (28672, 0.7)])
def test_count_law_of_per_token_threshold(n, k):
    """For distinct values, #{|c| > Quantile(k, |c|)} = n - 1 - floor(k (n - 1))."""
    c = np.abs(np.random.default_rng(n).standard_normal(n))
    q = oracle.quantile_linear(k, c)
    idx = oracle.select(c, q, use_abs=True)
    assert len(idx) == n - 1 - math.floor(k * (n - 1))


def test_select_is_strict_and_signed():
    c = np.array([[-3.0, 1.0, 2.0, -2.0, 2.5]])
    np.testing.assert_array_equal(oracle.select(c, 2.0, use_abs=True), [0, 4])
    np.testing.assert_array_equal(oracle.select(c, 2.0, use_abs=False), [4])
    np.testing.assert_array_equal(oracle.select(c, -2.5, use_abs=False), [1, 2, 3, 4])
    with pytest.raises(ValueError):
        oracle.select(c, float("nan"))


def test_calibration_is_mean_of_per_token_quantiles():
    w = WORKLOADS["tiny_256x688"]
    L = w.layer()
    X = w.tokens(16, purpose=T_CALIB)
    ur, gr, hr, sr, _ = np_reference(X, L)
    for variant, c in (("mono", np.abs(ur)), ("dual_ideal", np.abs(sr)), ("cats", np.abs(hr))):
        t, q = oracle.calibrate(variant, X, 0.9, W_gate=L["W_gate"], W_up=L["W_up"])
        qr = np.quantile(c, 0.9, axis=1, method="linear")
        np.testing.assert_allclose(q, qr, rtol=1e-12)
        assert t == pytest.approx(qr.mean(), rel=1e-12)
    P = make_predictor(w.wid, w.d_model, 32, w.d_ff, 0.02)
    t, q = oracle.calibrate("dual_pred", X, 0.9, A_t=P["A_t"], B_t=P["B_t"])
    sh = (f64(X) @ f64(P["A_t"]).T) @ f64(P["B_t"]).T
    np.testing.assert_allclose(q, np.quantile(sh, 0.9, axis=1), rtol=1e-10)


def test_calibrated_threshold_realises_about_k_on_held_out_tokens():
    w = WORKLOADS["tiny_256x688"]
    L = w.layer()
    t, _ = oracle.calibrate("mono", w.tokens(64, purpose=T_CALIB), 0.9, W_up=L["W_up"])
    x = w.tokens(32)
    u = oracle.coefficients(x, L["W_gate"], L["W_up"])[0]
    realised = 1.0 - np.mean(np.abs(u) > np.float32(t))
    assert abs(realised - 0.9) < 0.02


# --------------------------------------------------------- predictor, stack

def test_predictor_matches_numpy():
    x, _ = small_layer()
    P = make_predictor(909, 24, 6, 40, 0.3)
    lat, sh = oracle.predictor(x, P["A_t"], P["B_t"])
    np.testing.assert_allclose(lat, f64(x) @ f64(P["A_t"]).T, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(sh, lat @ f64(P["B_t"]).T, rtol=1e-12, atol=1e-15)


def test_residual_rmsnorm_closed_form():
    h = np.full(64, 3.0)
    h2, r = oracle.residual_rmsnorm(h, np.full(64, 1.0), eps=0.0)
    np.testing.assert_array_equal(h2, 4.0)
    np.testing.assert_allclose(r, 1.0, rtol=1e-15)
    h = np.array([3.0, -4.0])
    _, r = oracle.residual_rmsnorm(h, None, eps=0.0)
    np.testing.assert_allclose(r, h / math.sqrt(12.5), rtol=1e-15)
    # eps inside the root, comparable to mean(h^2): 1 / sqrt(1 + 3) = 1/2 exactly
    _, r = oracle.residual_rmsnorm(np.ones(16), None, eps=3.0)
    np.testing.assert_array_equal(r, 0.5)


def test_bad_arguments_are_rejected():
    x, L = small_layer()
    with pytest.raises(ValueError):
        oracle.ffn_mono(x, L["W_gate"], L["W_up"], L["W_down"], float("nan"))
    with pytest.raises(ValueError):
        oracle.combine(np.zeros((1, 40)), L["W_down"], np.array([40], dtype=np.int32))
    with pytest.raises(TypeError):
        oracle.dense(x.astype(np.int16), L["W_gate"], L["W_up"], L["W_down"])


# ------------------------------------------- per-token threshold (Eq. 6, per token)

def _brute_cs(x, L, mode, A_t=None, B_t=None):
    """Coefficient vectors c_b and s_b by pure-Python loops (Sec. 3, Sec. 4)."""
    X, G, U = (f64(a).tolist() for a in (x, L["W_gate"], L["W_up"]))

    def dot(a, b):
        t = 0.0
        for p, q in zip(a, b):
            t += p * q
        return t

    def silu(z):
        return z / (1.0 + math.exp(-z)) if z >= 0 else z * math.exp(z) / (1.0 + math.exp(z))

    B, dff = len(X), len(U)
    u = [[dot(X[b], U[i]) for i in range(dff)] for b in range(B)]
    s = [[u[b][i] * silu(dot(X[b], G[i])) for i in range(dff)] for b in range(B)]
    if mode == "mono":
        c = [[abs(v) for v in row] for row in u]
    elif mode == "dual_ideal":
        c = [[abs(v) for v in row] for row in s]
    else:
        A, Bm = f64(A_t).tolist(), f64(B_t).tolist()
        lat = [[dot(X[b], A[r]) for r in range(len(A))] for b in range(B)]
        c = [[dot(lat[b], Bm[i]) for i in range(dff)] for b in range(B)]
    return c, s


def _brute_quantile(v, k):
    w = sorted(v)
    h = k * (len(w) - 1)
    lo = math.floor(h)
    hi = min(lo + 1, len(w) - 1)
    return w[lo] + (h - lo) * (w[hi] - w[lo])


@pytest.mark.parametrize("mode", ["mono", "dual_ideal", "dual_pred"])
@pytest.mark.parametrize("B,k", [(1, 0.75), (3, 0.5), (2, 0.9)])
def test_topk_matches_brute_force(mode, B, k):
    dm, dff, dr = 8, 16, 4
    L = make_layer(960, dm, dff, 0.5)
    P = make_predictor(960, dm, dr, dff, 0.5)
    x = make_tokens(960, B, dm)
    c, s = _brute_cs(x, L, mode, P["A_t"], P["B_t"])
    q = [_brute_quantile(c[b], k) for b in range(B)]
    idx_b = [i for i in range(dff) if any(c[b][i] > q[b] for b in range(B))]
    D = f64(L["W_down"]).tolist()
    y_b = [[sum(s[b][i] * D[i][j] for i in idx_b) for j in range(dm)] for b in range(B)]
    pred = mode == "dual_pred"
    idx, y, qo = oracle.ffn_topk(mode, x, L["W_gate"], L["W_up"], L["W_down"], k,
                                 A_t=P["A_t"] if pred else None, B_t=P["B_t"] if pred else None)
    np.testing.assert_array_equal(idx, idx_b)
    np.testing.assert_allclose(qo, q, rtol=1e-13, atol=0)
    np.testing.assert_allclose(y, np.array(y_b), rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("mode", ["mono", "dual_ideal"])
def test_topk_count_law_and_constant_threshold_equivalence(mode):
    """Batch 1: |IDX| = n - 1 - floor(k (n - 1)) for distinct coefficients, and the
    result equals the constant-threshold path run at that token's quantile."""
    w = WORKLOADS["tiny_256x688"]
    L = w.layer()
    x = w.tokens(1)
    k = 0.9
    idx, y, q = oracle.ffn_topk(mode, x, L["W_gate"], L["W_up"], L["W_down"], k)
    n = w.d_ff
    assert len(idx) == n - 1 - math.floor(k * (n - 1))
    fn = oracle.ffn_mono if mode == "mono" else oracle.ffn_dual_ideal
    idx_c, y_c, _ = fn(x, L["W_gate"], L["W_up"], L["W_down"], q[0])
    np.testing.assert_array_equal(idx, idx_c)
    np.testing.assert_array_equal(y, y_c)


def test_topk_identical_tokens_and_extremes():
    w = WORKLOADS["tiny_256x688"]
    L = w.layer()
    x = w.tokens(1)
    idx1, y1, q1 = oracle.ffn_topk("mono", x, L["W_gate"], L["W_up"], L["W_down"], 0.8)
    idx3, y3, q3 = oracle.ffn_topk("mono", np.repeat(x, 3, axis=0), L["W_gate"], L["W_up"],
                                   L["W_down"], 0.8)
    np.testing.assert_array_equal(idx1, idx3)
    np.testing.assert_array_equal(q3, np.repeat(q1, 3))
    for b in range(3):
        np.testing.assert_array_equal(y3[b], y1[0])
    idx, y, _ = oracle.ffn_topk("mono", x, L["W_gate"], L["W_up"], L["W_down"], 1.0)
    assert len(idx) == 0 and not y.any()          # nothing exceeds the maximum
    idx, _, _ = oracle.ffn_topk("mono", x, L["W_gate"], L["W_up"], L["W_down"], 0.0)
    assert len(idx) == w.d_ff - 1                 # everything but the minimum


# ------------------------------------------------------ CATS coefficient (Eq. 6a)

@pytest.mark.parametrize("B", [1, 3])
def test_cats_matches_brute_force(B):
    """CATS keeps {i : |SiLU(x.W_gate)[i]| > thld} (union over the batch)."""
    dm, dff = 8, 16
    L = make_layer(970, dm, dff, 0.5)
    x = make_tokens(970, B, dm)
    X, G, U, D = (f64(a).tolist() for a in (x, L["W_gate"], L["W_up"], L["W_down"]))

    def dot(a, b):
        t = 0.0
        for p, q in zip(a, b):
            t += p * q
        return t

    def silu(z):
        return z / (1.0 + math.exp(-z)) if z >= 0 else z * math.exp(z) / (1.0 + math.exp(z))

    h = [[silu(dot(X[b], G[i])) for i in range(dff)] for b in range(B)]
    u = [[dot(X[b], U[i]) for i in range(dff)] for b in range(B)]
    thld = float(np.float32(np.quantile(np.abs(h[0]), 0.6)))
    idx_b = [i for i in range(dff) if any(abs(h[b][i]) > thld for b in range(B))]
    y_b = [[sum(u[b][i] * h[b][i] * D[i][j] for i in idx_b) for j in range(dm)] for b in range(B)]
    idx, y, hc = oracle.ffn_cats(x, L["W_gate"], L["W_up"], L["W_down"], thld, want_coef=True)
    np.testing.assert_array_equal(idx, idx_b)
    np.testing.assert_allclose(y, np.array(y_b), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(hc, np.array(h), rtol=1e-14, atol=0)
    # CATS through the per-token path with the CATS coefficient
    idx_t, _, q = oracle.ffn_topk("cats", x, L["W_gate"], L["W_up"], L["W_down"], 0.5)
    for b in range(B):
        assert q[b] == np.quantile(np.abs(h[b]), 0.5)


# --------------------------------------- ternary predictor (Sec. 6, TernaryLinear)

def _tern_small(B, seed=980, dm=8, dff=16):
    from workloads import make_ternary

    L = make_layer(seed, dm, dff, 0.5)
    T = make_ternary(seed, dm, dff)
    x = make_tokens(seed, B, dm)
    return x, L, T


@pytest.mark.parametrize("B", [1, 3])
def test_ternary_matches_brute_force(B):
    """s_hat = x . theta with theta in {-1, 0, +1}, then the predictor's signed
    threshold and the gather, by pure-Python loops."""
    x, L, T = _tern_small(B)
    dm, dff = T.shape[1], T.shape[0]
    X, G, U, D = (f64(a).tolist() for a in (x, L["W_gate"], L["W_up"], L["W_down"]))
    th = T.tolist()  # theta_t[i][j] = theta[j][i]

    def silu(z):
        return z / (1.0 + math.exp(-z)) if z >= 0 else z * math.exp(z) / (1.0 + math.exp(z))

    shat = []
    for b in range(B):
        row = []
        for i in range(dff):
            t = 0.0
            for j in range(dm):
                if th[i][j] == 1:
                    t += X[b][j]
                elif th[i][j] == -1:
                    t -= X[b][j]
            row.append(t)
        shat.append(row)
    thld = float(np.float32(np.quantile(shat[0], 0.6)))
    idx_b = [i for i in range(dff) if any(shat[b][i] > thld for b in range(B))]
    s = [[sum(X[b][j] * U[i][j] for j in range(dm)) * silu(sum(X[b][j] * G[i][j] for j in range(dm)))
          for i in range(dff)] for b in range(B)]
    y_b = [[sum(s[b][i] * D[i][j] for i in idx_b) for j in range(dm)] for b in range(B)]
    idx, y, c = oracle.ffn_dual_tern(x, L["W_gate"], L["W_up"], L["W_down"], T, thld,
                                     want_coef=True)
    np.testing.assert_array_equal(idx, idx_b)
    assert 0 < len(idx) < dff
    np.testing.assert_array_equal(c, np.array(shat))
    np.testing.assert_allclose(y, np.array(y_b), rtol=1e-12, atol=1e-13)


def test_ternary_equals_low_rank_with_identity_and_theta():
    """theta_A = I and theta_B = theta make the low-rank predictor the ternary one:
    identical index sets, scores and outputs (the low-rank oracle is pinned above)."""
    x, L, T = _tern_small(3, seed=981, dm=24, dff=40)
    dm, dff = T.shape[1], T.shape[0]
    A_t = bf16_round(np.eye(dm, dtype=np.float32))
    B_t = bf16_round(T.astype(np.float32))          # [d_ff][d_rank = d_model]
    sh_t = oracle.ternary_predictor(x, T)
    _, sh_p = oracle.predictor(x, A_t, B_t)
    np.testing.assert_array_equal(sh_t, sh_p)
    thld = float(np.float32(np.median(sh_t)))
    a = oracle.ffn_dual_tern(x, L["W_gate"], L["W_up"], L["W_down"], T, thld)
    b = oracle.ffn_dual_pred(x, L["W_gate"], L["W_up"], L["W_down"], A_t, B_t, thld)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


def test_ternary_closed_forms():
    x, L, _ = _tern_small(2, seed=982, dm=24, dff=40)
    dm, dff = 24, 40
    X = f64(x)
    # one-hot theta columns: s_hat_i = x_{j(i)}; negated: -x_{j(i)}
    T = np.zeros((dff, dm), dtype=np.int8)
    cols = np.arange(dff) % dm
    T[np.arange(dff), cols] = 1
    np.testing.assert_array_equal(oracle.ternary_predictor(x, T), X[:, cols])
    np.testing.assert_array_equal(oracle.ternary_predictor(x, -T), -X[:, cols])
    # all +1: the sum of the token; all zero: 0, so thld 0 keeps nothing (strict)
    ones = np.ones((dff, dm), dtype=np.int8)
    np.testing.assert_allclose(oracle.ternary_predictor(x, ones),
                               np.repeat(X.sum(axis=1, keepdims=True), dff, axis=1), rtol=1e-15)
    zero = np.zeros((dff, dm), dtype=np.int8)
    idx, y, _ = oracle.ffn_dual_tern(x, L["W_gate"], L["W_up"], L["W_down"], zero, 0.0)
    assert len(idx) == 0 and not y.any()
    with pytest.raises(ValueError):
        bad = zero.copy()
        bad[0, 0] = 2
        oracle.ffn_dual_tern(x, L["W_gate"], L["W_up"], L["W_down"], bad, 0.0)


def test_ternary_calibration_and_per_token_path():
    """The ternary score through calibration (mean of per-token quantiles of the
    signed score) and the per-token path, against numpy.quantile of brute-force scores."""
    x, L, T = _tern_small(3, seed=983, dm=24, dff=40)
    X = f64(x)
    shat = X @ T.astype(np.float64).T
    k = 0.7
    qs = [np.quantile(shat[b], k) for b in range(3)]
    tau, q = oracle.calibrate("dual_tern", x, k, theta_t=T)
    np.testing.assert_allclose(q, qs, rtol=1e-14)
    assert tau == pytest.approx(np.mean(qs), rel=1e-14)
    idx, _, qo = oracle.ffn_topk("dual_tern", x, L["W_gate"], L["W_up"], L["W_down"], k, theta_t=T)
    np.testing.assert_allclose(qo, qs, rtol=1e-14)
    want = [i for i in range(40) if any(shat[b][i] > qs[b] for b in range(3))]
    np.testing.assert_array_equal(idx, want)


def test_thread_count_does_not_change_results():
    """The oracle's OpenMP loops split independent rows and columns, each summed by
    one thread in ascending order: one thread and many give the same bits."""
    L = make_layer(2200, 64, 264, 0.05)
    X = make_tokens(2201, 3, 64)
    n = oracle.num_threads()
    try:
        outs = []
        for t in (1, max(n, 2)):
            oracle.set_num_threads(t)
            assert oracle.num_threads() == t
            outs.append(oracle.ffn_mono(X, L["W_gate"], L["W_up"], L["W_down"], np.float32(0.3)))
            outs.append(oracle.dense(X, L["W_gate"], L["W_up"], L["W_down"]))
    finally:
        oracle.set_num_threads(n)
    (i1, y1, _), d1, (i2, y2, _), d2 = outs
    assert np.array_equal(i1, i2) and np.array_equal(y1, y2) and np.array_equal(d1, d2)
