"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Same seeded inputs on both sides; IDX compared exactly except for neurons
within the relative band of thld, y compared against the oracle evaluated
on the GPU's IDX (a flipped boundary neuron moves y by more than the y
tolerance, so the y check is made on the set the GPU actually used), the
compact coefficients against the oracle's, and the dense coefficient
vector against the oracle within an fp32 dot-product bound.
"""
import math

import numpy as np
import pytest

from workloads import WORKLOADS, bf16_to_f32, make_layer, make_predictor, make_tokens
from workloads.synth import bf16_round
from workloads.synth import T_CALIB

from gpu_support import (COEF_TOL, check_idx, check_s, check_y, coef_max, dev_bf16, dot_bound)

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import oracle  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_17701_amd import binding

    binding.load_library()
    torch.cuda.set_device(0)


def f64(a):
    return bf16_to_f32(a).astype(np.float64)


class Layer:
    """A layer's weights on host (bf16 bits) and device; T: an optional ternary
    predictor theta_t (int8, kept on the host, packed on the device)."""

    def __init__(self, L, P=None, T=None):
        self.h = dict(L)
        if P:
            self.h.update(P)
        self.d = {k: dev_bf16(v) for k, v in self.h.items()}
        self.d_ff, self.d_model = self.h["W_up"].shape
        self.d_rank = self.h["A_t"].shape[0] if P else 0
        if T is not None:
            from paper_2505_17701_amd import binding as cd

            self.h["theta_t"] = T
            packed = cd.countdown_ternary_pack(T)
            self.d["theta_p"] = torch.from_numpy(packed.view(np.int32)).to("cuda")


def run_gpu(plan, variant, layer, x, thld):
    from paper_2505_17701_amd import binding as cd

    xd = dev_bf16(x)
    D = layer.d
    if variant == "mono":
        y = cd.countdown_ffn_mono(plan, xd, D["W_gate"], D["W_up"], D["W_down"], thld)
    elif variant == "dual_ideal":
        y = cd.countdown_ffn_dual(plan, xd, D["W_gate"], D["W_up"], D["W_down"], thld)
    elif variant == "dual_pred":
        y = cd.countdown_ffn_dual(plan, xd, D["W_gate"], D["W_up"], D["W_down"], thld,
                                  A_t=D["A_t"], B_t=D["B_t"])
    elif variant == "dense":
        y = cd.countdown_ffn_dense(plan, xd, D["W_gate"], D["W_up"], D["W_down"])
    elif variant == "cats":
        y = cd.countdown_ffn_cats(plan, xd, D["W_gate"], D["W_up"], D["W_down"], thld)
    elif variant == "dual_tern":
        y = cd.countdown_ffn_tern(plan, xd, D["W_gate"], D["W_up"], D["W_down"], D["theta_p"],
                                  thld)
    else:
        raise ValueError(variant)
    idx, s_c, coef = cd.countdown_export_active(plan)
    return (y.cpu().numpy().astype(np.float64), idx.cpu().numpy(), s_c.cpu().numpy(),
            None if coef is None else coef.cpu().numpy())


def run_oracle(variant, layer, x, thld):
    H = layer.h
    if variant == "mono":
        return oracle.ffn_mono(x, H["W_gate"], H["W_up"], H["W_down"], thld, want_coef=True)
    if variant == "dual_ideal":
        return oracle.ffn_dual_ideal(x, H["W_gate"], H["W_up"], H["W_down"], thld, want_coef=True)
    if variant == "dual_pred":
        return oracle.ffn_dual_pred(x, H["W_gate"], H["W_up"], H["W_down"], H["A_t"], H["B_t"],
                                    thld, want_coef=True)
    if variant == "dense":
        idx = np.arange(layer.d_ff, dtype=np.int32)
        return idx, oracle.dense(x, H["W_gate"], H["W_up"], H["W_down"]), None
    if variant == "cats":
        return oracle.ffn_cats(x, H["W_gate"], H["W_up"], H["W_down"], thld, want_coef=True)
    if variant == "dual_tern":
        return oracle.ffn_dual_tern(x, H["W_gate"], H["W_up"], H["W_down"], H["theta_t"], thld,
                                    want_coef=True)
    raise ValueError(variant)


def compare(plan, variant, layer, x, thld, label, check_coef=True):
    """Full parity check of one call; returns (n_active_gpu, n_flips, y_rel_err)."""
    x = np.atleast_2d(x)
    return check_call(variant, layer, x, thld, run_gpu(plan, variant, layer, x, thld), label,
                      check_coef)


def check_call(variant, layer, x, thld, gpu_out, label, check_coef=True):
    """Parity of one GPU call's outputs (y, IDX, compact s, coefficients) against the
    oracle on the same bf16 input x; returns (n_active_gpu, n_flips, y_rel_err)."""
    x = np.atleast_2d(x)
    y_g, idx_g, s_g, coef_g = gpu_out
    idx_o, y_o, coef_o = run_oracle(variant, layer, x, thld)
    H = layer.h
    if variant == "dense":
        np.testing.assert_array_equal(idx_g, np.arange(layer.d_ff))
        flips = 0
    else:
        flips = check_idx(idx_g, idx_o, coef_max(variant, coef_o), thld, label)
    # y and s on the GPU's own index set
    y_on, s_on = oracle.ffn_on_idx(x, H["W_gate"], H["W_up"], H["W_down"], idx_g)
    rel = check_y(y_g, y_on, label)
    if flips == 0 and variant != "dense":
        check_y(y_g, y_o, label + " (oracle IDX)")
    check_s(s_g, s_on, label)
    if check_coef and coef_g is not None and coef_o is not None:
        xf = f64(x)
        if variant == "mono":
            bound = COEF_TOL * dot_bound(xf, f64(H["W_up"]))
        elif variant == "dual_ideal":
            u, g, _ = oracle.coefficients(x, H["W_gate"], H["W_up"])
            su = np.array([[oracle.silu(v) for v in row] for row in g]) if g.size < 5000 else \
                g / (1.0 + np.exp(-g))
            bound = COEF_TOL * (dot_bound(xf, f64(H["W_up"])) * np.abs(su)
                                + np.abs(u) * dot_bound(xf, f64(H["W_gate"])))
        elif variant == "cats":
            # h = SiLU(g): |dh| <= max|SiLU'| |dg|, max|SiLU'| < 1.1
            bound = COEF_TOL * 1.1 * dot_bound(xf, f64(H["W_gate"]))
        elif variant == "dual_tern":
            bound = COEF_TOL * dot_bound(xf, H["theta_t"].astype(np.float64))
        else:
            lat = oracle.predictor(x, H["A_t"], H["B_t"])[0]
            bound = COEF_TOL * (np.abs(lat) @ np.abs(f64(H["B_t"])).T
                                + dot_bound(xf, f64(H["A_t"])) @ np.abs(f64(H["B_t"])).T)
        err = np.abs(coef_g[: x.shape[0]] - coef_o)
        assert np.all(err <= bound + 1e-30), f"{label}: coefficient error {err.max():.3e}"
    return len(idx_g), flips, rel


def plan_for(layer, max_batch=1, keep_coef=True):
    from paper_2505_17701_amd import binding as cd

    return cd.Plan(layer.d_model, layer.d_ff, max_batch, layer.d_rank, keep_coef=keep_coef)


def calibrated(variant, layer, wid, k, T=32, outlier_frac=0.0):
    X = make_tokens(wid, T, layer.d_model, purpose=T_CALIB, outlier_frac=outlier_frac)
    H = layer.h
    t, _ = oracle.calibrate(variant, X, k, W_gate=H["W_gate"], W_up=H["W_up"],
                            A_t=H.get("A_t"), B_t=H.get("B_t"))
    return float(np.float32(t))


# --------------------------------------------------------------- small shapes

@pytest.fixture(scope="module")
def tiny():
    w = WORKLOADS["tiny_256x688"]
    return w, Layer(w.layer())


@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "cats"])
def test_tiny_parity_calibrated(tiny, variant):
    w, layer = tiny
    thld = calibrated(variant, layer, w.wid, 0.9, T=64)
    plan = plan_for(layer)
    X = w.tokens(16)
    for t in range(16):
        n, flips, _ = compare(plan, variant, layer, X[t:t + 1], thld, f"tiny {variant} tok{t}")
        assert 20 < n < 140


@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "cats"])
@pytest.mark.parametrize("B", [2, 3, 5, 8])
def test_tiny_batch_union(tiny, variant, B):
    w, layer = tiny
    thld = calibrated(variant, layer, w.wid, 0.9, T=64)
    plan = plan_for(layer, max_batch=8)
    X = w.tokens(B)
    n, _, _ = compare(plan, variant, layer, X, thld, f"tiny {variant} B={B}")
    assert n > 69


@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "cats"])
def test_all_rows_equals_dense_and_none_gives_zero(tiny, variant):
    w, layer = tiny
    plan = plan_for(layer, max_batch=2)
    X = w.tokens(2)
    n, _, _ = compare(plan, variant, layer, X, -math.inf, f"{variant} -inf")
    assert n == layer.d_ff
    y_all = run_gpu(plan, variant, layer, X, -math.inf)[0]
    y_dense = run_gpu(plan, "dense", layer, X, 0.0)[0]
    np.testing.assert_allclose(y_all, y_dense, rtol=0, atol=1e-5 * np.abs(y_dense).max())
    y0, idx0, _, _ = run_gpu(plan, variant, layer, X, math.inf)
    assert len(idx0) == 0 and np.all(y0 == 0.0)


@pytest.mark.parametrize("B", [1, 2, 4])
def test_dense_parity(tiny, B):
    w, layer = tiny
    plan = plan_for(layer, max_batch=4)
    compare(plan, "dense", layer, w.tokens(B), 0.0, f"dense B={B}")


def _summation_atol(layer, idx, x):
    """fp32 bound on the difference of two orders of the sum of y over the active rows:
    2 (n + 8) units of 2^-24 of the largest sum of |s_i W_down[i, j]| (n terms, plus
    the lane and workgroup sums; each order within half of it)."""
    H = layer.h
    _, s_on = oracle.ffn_on_idx(np.atleast_2d(x), H["W_gate"], H["W_up"], H["W_down"], idx)
    yabs = np.abs(s_on) @ np.abs(f64(H["W_down"])[idx])
    return 2 * (len(idx) + 8) * 2.0 ** -24 * float(yabs.max()) + 1e-30


@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "cats", "dual_pred"])
def test_metamorphic_relations(tiny, variant):
    """Exact relations of the method, checked on the kernels alone (Eq. 5 and 6): W_down
    doubled gives the same IDX and 2y; W_up negated gives the same IDX and -y (|u|, |s|,
    |SiLU(g)| and the predictor score are unchanged bit for bit); a permutation of the neurons permutes IDX and leaves
    y unchanged up to the order of the sum."""
    w, layer = tiny
    if variant == "dual_pred":  # the predictor reads neither W_up nor W_down
        layer = Layer(w.layer(), make_predictor(w.wid, layer.d_model, 64, layer.d_ff, 0.02))
    thld = calibrated(variant, layer, w.wid, 0.9, T=64)
    X = w.tokens(2)
    plan = plan_for(layer, max_batch=2)
    y, idx, _, _ = run_gpu(plan, variant, layer, X, thld)
    assert 0 < len(idx) < layer.d_ff
    atol = _summation_atol(layer, idx, X)
    H = layer.h

    doubled = Layer(dict(H, W_down=bf16_round(2.0 * bf16_to_f32(H["W_down"]))))
    y2, idx2, _, _ = run_gpu(plan, variant, doubled, X, thld)
    np.testing.assert_array_equal(idx2, idx)
    np.testing.assert_allclose(y2, 2.0 * y, rtol=0, atol=2.0 * atol)

    negated = Layer(dict(H, W_up=H["W_up"] ^ np.uint16(0x8000)))
    yn, idxn, _, _ = run_gpu(plan, variant, negated, X, thld)
    np.testing.assert_array_equal(idxn, idx)
    np.testing.assert_allclose(yn, -y, rtol=0, atol=atol)

    perm = np.random.default_rng(17).permutation(layer.d_ff)  # new row j = old row perm[j]
    permuted = Layer({k: np.ascontiguousarray(v[perm]) if v.shape[0] == layer.d_ff else v
                      for k, v in H.items()})  # neuron-major matrices (A_t is not)
    yp, idxp, _, _ = run_gpu(plan, variant, permuted, X, thld)
    np.testing.assert_array_equal(np.sort(perm[idxp]), idx)
    np.testing.assert_allclose(yp, y, rtol=0, atol=atol)


def test_single_active_row(tiny):
    w, layer = tiny
    x = w.tokens(1)
    u = oracle.coefficients(x, layer.h["W_gate"], layer.h["W_up"])[0][0]
    top = np.sort(np.abs(u))
    thld = float(np.float32((top[-1] + top[-2]) / 2))
    plan = plan_for(layer)
    n, flips, _ = compare(plan, "mono", layer, x, thld, "single row")
    assert n == 1 and flips == 0


@pytest.mark.parametrize("d_model,d_ff,B", [(264, 1000, 3), (1032, 520, 2), (8, 8, 1),
                                            (2056, 4104, 7), (512, 16, 4), (8192, 1048, 1),
                                            (1544, 2056, 2), (4096, 776, 1), (4160, 1000, 4),
                                            (4160, 1000, 1), (6152, 520, 1)])
@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "dual_pred", "cats"])
def test_ragged_shapes(d_model, d_ff, B, variant):
    L = make_layer(700 + d_model, d_model, d_ff, 0.05)
    P = make_predictor(700 + d_model, d_model, 16, d_ff, 0.05) if variant == "dual_pred" else None
    layer = Layer(L, P)
    x = make_tokens(700 + d_model, B, d_model)
    if variant == "dual_pred":
        c = oracle.predictor(x, P["A_t"], P["B_t"])[1]
    else:
        u, g, s = oracle.coefficients(x, L["W_gate"], L["W_up"])
        c = np.abs({"mono": u, "dual_ideal": s, "cats": g / (1.0 + np.exp(-g))}[variant])
    thld = float(np.float32(np.quantile(c, 0.7)))
    from paper_2505_17701_amd import binding as cd

    plan = plan_for(layer, max_batch=cd.max_batch_for(d_model))
    compare(plan, variant, layer, x, thld, f"ragged {d_model}x{d_ff} B={B} {variant}")


@pytest.mark.parametrize("d_rank", [8, 32, 128, 512, 1024])
@pytest.mark.parametrize("B", [1, 4, 8])
def test_predictor_ranks(d_rank, B):
    """Every predictor rank the plan accepts, through the v_dot2 (B <= 4) and MFMA
    (B 8) predictor kernels; rank 1024 stages the latent in LDS instead of
    registers. Signed 0.8-quantile threshold of the oracle's scores."""
    dm, dff = 512, 1040
    L = make_layer(900 + d_rank, dm, dff, 0.05)
    P = make_predictor(900 + d_rank, dm, d_rank, dff, 0.05)
    layer = Layer(L, P)
    x = make_tokens(901 + d_rank, B, dm)
    thld = float(np.float32(np.quantile(oracle.predictor(x, P["A_t"], P["B_t"])[1], 0.8)))
    plan = plan_for(layer, max_batch=8)
    n, flips, rel = compare(plan, "dual_pred", layer, x, thld, f"rank {d_rank} B={B}")
    assert n > 0
    print(f"rank {d_rank} B={B}: n={n} flips={flips} rel_err={rel:.2e}", flush=True)


@pytest.mark.parametrize("B", [2, 3, 4])
@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "dual_pred", "cats", "dual_tern"])
def test_widest_token_tile(variant, B):
    """d_model 8192 at 2-4 tokens: the LDS token copy that two tokens of this width
    take, batch x d_model at the plan's limit of 32768 (64 KB of LDS), and the MFMA
    down kernel at its widest rows."""
    from workloads import make_ternary

    dm, dff = 8192, 1048
    L = make_layer(960 + B, dm, dff, 0.02)
    P = make_predictor(960 + B, dm, 64, dff, 0.02) if variant == "dual_pred" else None
    T = make_ternary(960 + B, dm, dff) if variant == "dual_tern" else None
    layer = Layer(L, P, T)
    x = make_tokens(961 + B, B, dm)
    if variant == "dual_pred":
        c = oracle.predictor(x, P["A_t"], P["B_t"])[1]
    elif variant == "dual_tern":
        c = oracle.ternary_predictor(x, T)
    else:
        u, g, s = oracle.coefficients(x, L["W_gate"], L["W_up"])
        c = np.abs({"mono": u, "dual_ideal": s, "cats": g / (1.0 + np.exp(-g))}[variant])
    thld = float(np.float32(np.quantile(c, 0.85)))
    plan = plan_for(layer, max_batch=4)
    n, flips, rel = compare(plan, variant, layer, x, thld, f"8192 B={B} {variant}")
    assert n > 0
    print(f"8192 B={B} {variant}: n={n} flips={flips} rel_err={rel:.2e}", flush=True)


def test_plan_reuse_with_shrinking_batch(tiny):
    w, layer = tiny
    thld = calibrated("mono", layer, w.wid, 0.9, T=64)
    plan = plan_for(layer, max_batch=8)
    for B in (8, 3, 1, 5, 2, 1):
        compare(plan, "mono", layer, w.tokens(B), thld, f"reuse B={B}")


def test_nondefault_stream_and_repeatability(tiny):
    from paper_2505_17701_amd import binding as cd

    w, layer = tiny
    thld = calibrated("dual_ideal", layer, w.wid, 0.9, T=64)
    plan = plan_for(layer, max_batch=2, keep_coef=False)
    X = dev_bf16(w.tokens(2))
    D = layer.d
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        y1 = cd.countdown_ffn_dual(plan, X, D["W_gate"], D["W_up"], D["W_down"], thld)
        i1 = cd.countdown_export_active(plan)[0].clone()
        y2 = cd.countdown_ffn_dual(plan, X, D["W_gate"], D["W_up"], D["W_down"], thld)
        i2 = cd.countdown_export_active(plan)[0].clone()
    s.synchronize()
    assert torch.equal(i1, i2)
    torch.testing.assert_close(y1, y2, rtol=0, atol=1e-6 * float(y1.abs().max()))


def test_phase_selection(tiny):
    """Coefficient-only then down-only calls reproduce the full call; a down-only call
    needs a previous coefficient kernel on the plan, run on the same batch."""
    from paper_2505_17701_amd import binding as cd

    w, layer = tiny
    thld = calibrated("mono", layer, w.wid, 0.9, T=64)
    D = layer.d
    X = dev_bf16(w.tokens(2))
    plan = plan_for(layer, max_batch=2, keep_coef=False)
    y_full = cd.countdown_ffn_mono(plan, X, D["W_gate"], D["W_up"], D["W_down"], thld)
    cd.countdown_plan_set_phases(plan, cd.CD_PHASE_COEF)
    y_c = torch.full_like(y_full, float("nan"))
    cd.countdown_ffn_mono(plan, X, D["W_gate"], D["W_up"], D["W_down"], thld, y=y_c)
    torch.cuda.synchronize()
    assert torch.all(y_c == 0)  # the coefficient kernel zeroes y for the down kernel
    cd.countdown_plan_set_phases(plan, cd.CD_PHASE_DOWN)
    for _ in range(2):
        y_d = torch.zeros_like(y_full)
        cd.countdown_ffn_mono(plan, X, D["W_gate"], D["W_up"], D["W_down"], thld, y=y_d)
        torch.testing.assert_close(y_d, y_full, rtol=0, atol=1e-6 * float(y_full.abs().max()))
    # the coefficient kernel ran on two tokens: a down-only call on one is refused
    with pytest.raises(cd.CountdownError):
        cd.countdown_ffn_mono(plan, X[:1], D["W_gate"], D["W_up"], D["W_down"], thld)
    cd.countdown_plan_set_phases(plan, cd.CD_PHASE_ALL)
    torch.testing.assert_close(
        cd.countdown_ffn_mono(plan, X, D["W_gate"], D["W_up"], D["W_down"], thld), y_full,
        rtol=0, atol=1e-6 * float(y_full.abs().max()))
    fresh = plan_for(layer, keep_coef=False)
    cd.countdown_plan_set_phases(fresh, cd.CD_PHASE_DOWN)
    with pytest.raises(cd.CountdownError):
        cd.countdown_ffn_mono(fresh, X[:1], D["W_gate"], D["W_up"], D["W_down"], thld)
    for bad in (0, 4, 7):
        with pytest.raises(cd.CountdownError):
            cd.countdown_plan_set_phases(fresh, bad)


def test_bad_calls_raise(tiny):
    from paper_2505_17701_amd import binding as cd

    w, layer = tiny
    plan = plan_for(layer, max_batch=2)
    D = layer.d
    X = dev_bf16(w.tokens(3))
    with pytest.raises(cd.CountdownError):
        cd.countdown_ffn_mono(plan, X, D["W_gate"], D["W_up"], D["W_down"], 0.5)  # B > max_batch
    with pytest.raises(cd.CountdownError):
        cd.countdown_ffn_mono(plan, X[:1], D["W_gate"], D["W_up"], D["W_down"], float("nan"))
    # one predictor matrix only: the binding's shape check (no rank-0 A_t exists) or the
    # library's rule rejects it
    with pytest.raises((cd.CountdownError, ValueError)):
        cd.countdown_ffn_dual(plan, X[:1], D["W_gate"], D["W_up"], D["W_down"], 0.5,
                              A_t=D["W_up"], B_t=None)


def test_outputs_overlapping_inputs_are_rejected(tiny):
    """y sharing memory with x or a weight matrix, and per-token thresholds sharing
    memory with y, are rejected on the host: nothing is launched."""
    from paper_2505_17701_amd import binding as cd

    w, layer = tiny
    plan = plan_for(layer, max_batch=2)
    D = layer.d
    dm = plan.d_model
    x = dev_bf16(w.tokens(2))
    raw = torch.zeros(2 * dm * 4, dtype=torch.uint8, device="cuda")
    y_over_x = raw.view(torch.float32).view(2, dm)
    x_in = raw[: 2 * dm * 2].view(torch.bfloat16).view(2, dm)
    x_in.copy_(x)
    with pytest.raises(cd.CountdownError):
        cd.countdown_ffn_mono(plan, x_in, D["W_gate"], D["W_up"], D["W_down"], 0.5, y=y_over_x)
    up_before = D["W_up"].clone()
    y_in_up = D["W_up"].view(-1).view(torch.float32)[dm: 3 * dm].view(2, dm)
    for call in (lambda: cd.countdown_ffn_mono(plan, x, D["W_gate"], D["W_up"], D["W_down"],
                                               0.5, y=y_in_up),
                 lambda: cd.countdown_ffn_dense(plan, x, D["W_gate"], D["W_up"], D["W_down"],
                                                y=y_in_up),
                 lambda: cd.countdown_ffn_topk(plan, 0, x, D["W_gate"], D["W_up"], D["W_down"],
                                               0.9, y=y_in_up)):
        with pytest.raises(cd.CountdownError):
            call()
    y = torch.empty(2, dm, dtype=torch.float32, device="cuda")
    with pytest.raises(cd.CountdownError):
        cd.countdown_ffn_topk(plan, 0, x, D["W_gate"], D["W_up"], D["W_down"], 0.9, y=y,
                              thld_out=y.view(-1).view(torch.float64)[:2])
    torch.cuda.synchronize()
    assert torch.equal(D["W_up"], up_before)
    # the same call with separate outputs goes through
    q = torch.empty(2, dtype=torch.float64, device="cuda")
    cd.countdown_ffn_topk(plan, 0, x, D["W_gate"], D["W_up"], D["W_down"], 0.9, y=y, thld_out=q)
    torch.cuda.synchronize()


# ------------------------------------------------------------- calibration

@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "dual_pred", "cats"])
def test_calibration_matches_oracle(variant):
    from paper_2505_17701_amd import binding as cd

    dm, dff = 512, 1376
    L = make_layer(811, dm, dff, 0.02)
    P = make_predictor(811, dm, 64, dff, 0.02) if variant == "dual_pred" else None
    layer = Layer(L, P)
    X = make_tokens(811, 20, dm, purpose=T_CALIB)
    t_o, q_o = oracle.calibrate(variant, X, 0.9, W_gate=L["W_gate"], W_up=L["W_up"],
                                A_t=P and P["A_t"], B_t=P and P["B_t"])
    plan = cd.Plan(dm, dff, 8, layer.d_rank, keep_coef=True)
    v = {"mono": cd.CD_VARIANT_MONO, "dual_ideal": cd.CD_VARIANT_DUAL_IDEAL,
         "dual_pred": cd.CD_VARIANT_DUAL_PRED, "cats": cd.CD_VARIANT_CATS}[variant]
    D = layer.d
    thld, q = cd.countdown_calibrate(plan, v, dev_bf16(X), 0.9, W_gate=D["W_gate"], W_up=D["W_up"],
                                     A_t=D.get("A_t"), B_t=D.get("B_t"))
    q = q.cpu().numpy()
    np.testing.assert_allclose(q, q_o, rtol=2e-5)
    assert abs(float(thld.item()) - t_o) <= 2e-5 * abs(t_o)
    assert float(thld.item()) == float(np.float32(q.mean()))  # fp64 mean, fp32 rounding


def test_calibration_selects_exact_order_statistics():
    """On the GPU's own fp32 coefficients the per-token quantile is exactly the
    linear interpolation between the order statistics (numpy sort)."""
    from paper_2505_17701_amd import binding as cd

    dm, dff = 256, 688
    L = make_layer(812, dm, dff, 0.02)
    layer = Layer(L)
    X = make_tokens(812, 6, dm, purpose=T_CALIB)
    plan = cd.Plan(dm, dff, 8, 0, keep_coef=True)
    D = layer.d
    for k in (0.0, 0.5, 0.9, 0.999, 1.0):
        _, q = cd.countdown_calibrate(plan, cd.CD_VARIANT_MONO, dev_bf16(X), k, W_up=D["W_up"])
        y = cd.countdown_ffn_mono(plan, dev_bf16(X), D["W_gate"], D["W_up"], D["W_down"],
                                  math.inf)
        coef = cd.countdown_export_active(plan)[2].cpu().numpy().astype(np.float64)
        for t in range(6):
            v = np.sort(np.abs(coef[t]))
            h = k * (dff - 1)
            lo = min(int(math.floor(h)), dff - 1)
            hi = min(lo + 1, dff - 1)
            assert q[t].item() == v[lo] + (h - lo) * (v[hi] - v[lo])
        del y


def test_graph_replay_matches_eager(tiny):
    """FFN calls captured in a HIP graph and replayed several times, with eager work
    between the replays, give the eager results every time."""
    from paper_2505_17701_amd import binding as cd

    w, layer = tiny
    thld_m = calibrated("mono", layer, w.wid, 0.9, T=64)
    thld_d = calibrated("dual_ideal", layer, w.wid, 0.9, T=64)
    pm, pd = plan_for(layer, keep_coef=False), plan_for(layer, keep_coef=False)
    X = dev_bf16(w.tokens(4))
    D = layer.d
    ys = [torch.empty((1, layer.d_model), dtype=torch.float32, device="cuda") for _ in range(8)]

    def calls():
        for t in range(4):
            cd.countdown_ffn_mono(pm, X[t:t + 1], D["W_gate"], D["W_up"], D["W_down"], thld_m,
                                  y=ys[t])
            cd.countdown_ffn_dual(pd, X[t:t + 1], D["W_gate"], D["W_up"], D["W_down"], thld_d,
                                  y=ys[4 + t])

    calls()
    torch.cuda.synchronize()
    eager = [y.clone() for y in ys]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        calls()
    for rep in range(3):
        for y in ys:
            y.fill_(float("nan"))
        cd.countdown_ffn_dense(pm, X[:1], D["W_gate"], D["W_up"], D["W_down"])  # eager work
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for y, e in zip(ys, eager):
            torch.testing.assert_close(y, e, rtol=0, atol=1e-6 * float(e.abs().max()) + 1e-30)


def test_graph_replay_all_paths():
    """Graph replay of the batch-8 predictor (MFMA gather and MFMA down projection),
    the ternary predictor and the per-token path, against their eager results."""
    from paper_2505_17701_amd import binding as cd
    from workloads import make_ternary

    dm, dff = 1024, 2056
    L = make_layer(830, dm, dff, 0.03)
    P = make_predictor(830, dm, 64, dff, 0.05)
    T = make_ternary(830, dm, dff)
    layer = Layer(L, P, T)
    D = layer.d
    X = dev_bf16(make_tokens(830, 16, dm))
    th_p = calibrated("dual_pred", layer, 830, 0.7, T=32)
    th_t = float(np.float32(oracle.calibrate("dual_tern", make_tokens(830, 32, dm, purpose=T_CALIB),
                                             0.7, theta_t=T)[0]))
    plans = [cd.Plan(dm, dff, 8, 64) for _ in range(4)]
    ys = [torch.empty((8, dm), dtype=torch.float32, device="cuda") for _ in range(4)]

    def calls():
        cd.countdown_ffn_dual(plans[0], X[:8], D["W_gate"], D["W_up"], D["W_down"], th_p,
                              A_t=D["A_t"], B_t=D["B_t"], y=ys[0])
        cd.countdown_ffn_tern(plans[1], X[8:16], D["W_gate"], D["W_up"], D["W_down"],
                              D["theta_p"], th_t, y=ys[1])
        cd.countdown_ffn_topk(plans[2], cd.CD_VARIANT_MONO, X[2:6], D["W_gate"], D["W_up"],
                              D["W_down"], 0.9, y=ys[2][:4])
        cd.countdown_ffn_tern_topk(plans[3], X[5:6], D["W_gate"], D["W_up"], D["W_down"],
                                   D["theta_p"], 0.8, y=ys[3][:1])

    calls()
    torch.cuda.synchronize()
    eager = [y.clone() for y in ys]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        calls()
    for rep in range(3):
        for y in ys:
            y.fill_(float("nan"))
        cd.countdown_ffn_dual(plans[0], X[8:16], D["W_gate"], D["W_up"], D["W_down"], th_p,
                              A_t=D["A_t"], B_t=D["B_t"])  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, (y, e) in enumerate(zip(ys, eager)):
            rows = (8, 8, 4, 1)[k]
            torch.testing.assert_close(y[:rows], e[:rows], rtol=0,
                                       atol=1e-6 * float(e[:rows].abs().max()) + 1e-30)
    for p in plans:
        p.close()


def test_stream_read_measurement_aid():
    """countdown_stream_read reads a buffer without touching it or the sink (all-zero
    data folds to 0) and rejects sizes that are not whole 16-byte chunks."""
    from paper_2505_17701_amd import binding as cd

    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    for n in (8, 4096 * 8 + 8, 3 << 20):  # bf16 elements: one chunk, a ragged wave, 6 MiB
        buf = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
        cd.countdown_stream_read(buf, sink)
        torch.cuda.synchronize()
        assert int(sink.item()) == 0 and not buf.any()
    with pytest.raises(cd.CountdownError):
        cd.countdown_stream_read(torch.zeros(7, dtype=torch.uint8, device="cuda"), sink)
    with pytest.raises(cd.CountdownError):
        cd.countdown_stream_read(torch.zeros(64, dtype=torch.uint8, device="cuda")[1:17], sink)
