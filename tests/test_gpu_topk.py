"""GPU parity of the per-token threshold path (countdown_ffn_topk): each
token's threshold is the linear-interpolation k-quantile of its own
coefficients, IDX the union of the neurons above their token's threshold.
Checked against oracle.ffn_topk: thresholds, IDX (bit-exact outside a band
around each token's threshold), y on the GPU's index set, and the count law
d_ff - 1 - floor(k (d_ff - 1)) at batch 1."""
import math

import numpy as np
import pytest

import oracle
from gpu_support import IDX_BAND, check_s, check_y, dev_bf16
from test_gpu_parity import Layer, f64
from workloads import WORKLOADS, make_layer, make_predictor, make_tokens
from workloads.synth import bf16_round

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

VID = {"mono": 0, "dual_ideal": 1, "dual_pred": 2, "cats": 4}
Q_TOL = 1e-5  # relative to max(|q|, rms(c)): fp32 coefficients against fp64


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def oracle_coef(variant, layer, x):
    H = layer.h
    if variant == "dual_pred":
        return oracle.predictor(x, H["A_t"], H["B_t"])[1]
    if variant == "dual_tern":
        return oracle.ternary_predictor(x, H["theta_t"])
    u, g, s = oracle.coefficients(x, H["W_gate"], H["W_up"])
    return np.abs({"mono": u, "dual_ideal": s, "cats": g / (1.0 + np.exp(-g))}[variant])


def run_topk(variant, layer, x, k):
    from paper_2505_17701_amd import binding as cd

    B = x.shape[0]
    plan = cd.Plan(layer.d_model, layer.d_ff, max_batch=B, d_rank=layer.d_rank)
    q = torch.zeros(B, dtype=torch.float64, device="cuda")
    D = layer.d
    if variant == "dual_tern":
        y = cd.countdown_ffn_tern_topk(plan, dev_bf16(x), D["W_gate"], D["W_up"], D["W_down"],
                                       D["theta_p"], k, thld_out=q)
    else:
        y = cd.countdown_ffn_topk(plan, VID[variant], dev_bf16(x), D["W_gate"], D["W_up"],
                                  D["W_down"], k, A_t=D.get("A_t"), B_t=D.get("B_t"), thld_out=q)
    idx, s_c, _ = cd.countdown_export_active(plan)
    out = (y.cpu().numpy().astype(np.float64), idx.cpu().numpy(), s_c.cpu().numpy(),
           q.cpu().numpy())
    plan.close()
    return out


def check_topk(variant, layer, x, k, label):
    x = np.atleast_2d(x)
    B = x.shape[0]
    y_g, idx_g, s_g, q_g = run_topk(variant, layer, x, k)
    H = layer.h
    idx_o, y_o, q_o = oracle.ffn_topk(variant, x, H["W_gate"], H["W_up"], H["W_down"], k,
                                      A_t=H.get("A_t"), B_t=H.get("B_t"),
                                      theta_t=H.get("theta_t"))
    c = oracle_coef(variant, layer, x)
    scale = np.maximum(np.abs(q_o), np.sqrt(np.mean(c * c, axis=1)))
    assert np.all(np.abs(q_g - q_o) <= Q_TOL * scale), f"{label}: thresholds {q_g} vs {q_o}"
    # IDX: equal except neurons within the band of their own token's threshold
    assert np.all(np.diff(idx_g) > 0), f"{label}: IDX not ascending"
    diff = np.setxor1d(idx_g, idx_o)
    band = IDX_BAND * scale + np.abs(q_g - q_o)
    near = np.zeros(layer.d_ff, dtype=bool)
    for b in range(B):
        near |= np.abs(c[b] - q_o[b]) <= band[b]
    assert near[diff].all(), f"{label}: {np.count_nonzero(~near[diff])} IDX differences outside the band"
    y_on, s_on = oracle.ffn_on_idx(x, H["W_gate"], H["W_up"], H["W_down"], idx_g)
    rel = check_y(y_g, y_on, label)
    if len(diff) == 0:
        check_y(y_g, y_o, label + " (oracle IDX)")
    check_s(s_g, s_on, label)
    return len(idx_g), len(diff), rel


def small(variant, dm, dff, seed):
    L = make_layer(1200 + seed, dm, dff, 0.03)
    P = make_predictor(1200 + seed, dm, 64, dff, 0.05) if variant == "dual_pred" else None
    return Layer(L, P)


@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "dual_pred", "cats"])
@pytest.mark.parametrize("shape", [(256, 688, 1, 0.9), (1032, 1000, 3, 0.75), (4096, 1376, 2, 0.5),
                                   (2048, 776, 8, 0.9), (264, 16, 1, 0.5)])
def test_topk_small(variant, shape):
    dm, dff, B, k = shape
    layer = small(variant, dm, dff, dm + dff)
    x = make_tokens(1300 + dm, B, dm)
    n, flips, rel = check_topk(variant, layer, x, k, f"topk {variant} {shape}")
    if B == 1 and flips == 0:
        assert n == dff - 1 - math.floor(k * (dff - 1)), (n, dff, k)


@pytest.mark.parametrize("k", [0.0, 1.0])
def test_topk_extremes(k):
    layer = small("mono", 512, 520, 3)
    x = make_tokens(1400, 2, 512)
    y_g, idx_g, _, q_g = run_topk("mono", layer, x, k)
    if k == 1.0:
        assert len(idx_g) == 0 and not y_g.any()
    else:
        # each token drops only its own minimum; the union drops what both minima share
        assert len(idx_g) >= layer.d_ff - 2


@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "dual_pred", "cats"])
@pytest.mark.parametrize("shape", [(8, 8, 0.5), (8, 16384, 0.9), (4096, 8, 0.3), (520, 24, 0.6),
                                   (1544, 9000, 0.1), (3080, 16384, 0.95)])
def test_topk_single_token_edges(variant, shape):
    """One token takes the one-launch kernels (select with gather, or for ideal
    D select with down projection) at their smallest and largest shapes: 8
    columns or neurons, 16384 neurons, a 520-column row (one 8-column chunk past
    512), 90% active."""
    dm, dff, k = shape
    layer = small(variant, dm, dff, 7 * dm + dff)
    x = make_tokens(1500 + dm + dff, 1, dm)
    n, flips, rel = check_topk(variant, layer, x, k, f"one token {variant} {shape}")
    if flips == 0:
        assert n == dff - 1 - math.floor(k * (dff - 1)), (n, dff, k)


@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "cats"])
@pytest.mark.parametrize("k", [0.0, 1.0])
def test_topk_extremes_single_token(variant, k):
    """k = 1 keeps nothing (y = 0); k = 0 keeps every neuron but the token's minimum."""
    layer = small(variant, 512, 520, 5)
    x = make_tokens(1401, 1, 512)
    if k == 1.0:
        y_g, idx_g, _, _ = run_topk(variant, layer, x, k)
        assert len(idx_g) == 0 and not y_g.any()
    else:
        n, flips, rel = check_topk(variant, layer, x, k, f"one token {variant} k=0")
        assert n == layer.d_ff - 1 or flips, n


def test_topk_count_law_llama7b():
    w = WORKLOADS["llama7b_4096x11008"]
    layer = Layer(w.layer())
    for t, k in enumerate((0.9, 0.7, 0.5)):
        x = w.tokens(t + 1)[t:t + 1]
        n, flips, rel = check_topk("mono", layer, x, k, f"7b mono topk k={k}")
        assert n == w.d_ff - 1 - math.floor(k * (w.d_ff - 1)), (n, k)
        print(f"7b topk k={k}: n={n} flips={flips} rel={rel:.2e}", flush=True)
    n, flips, rel = check_topk("dual_ideal", layer, w.tokens(2), 0.9, "7b dual topk B=2")
    print(f"7b dual topk B=2: n={n} flips={flips} rel={rel:.2e}", flush=True)
    # one token: select, flags and down projection in one launch
    n, flips, rel = check_topk("dual_ideal", layer, w.tokens(4)[3:4], 0.9, "7b dual topk B=1")
    if flips == 0:
        assert n == w.d_ff - 1 - math.floor(0.9 * (w.d_ff - 1)), n
    print(f"7b dual topk B=1: n={n} flips={flips} rel={rel:.2e}", flush=True)


def test_topk_predictor_batch():
    w = WORKLOADS["llama3_8b_4096x14336_pred"]
    layer = Layer(w.layer(), w.predictor())
    for B in (1, 4):
        n, flips, rel = check_topk("dual_pred", layer, w.tokens(B), 0.9, f"8b pred topk B={B}")
        print(f"8b pred topk B={B}: n={n} flips={flips} rel={rel:.2e}", flush=True)


@pytest.mark.parametrize("variant", ["mono", "cats", "dual_ideal", "dual_pred", "dual_tern"])
@pytest.mark.parametrize("shape", [(4096, 11008, 0.9, None), (4096, 14336, 0.9, None),
                                   (512, 16384, 0.8, None), (256, 32768, 0.7, None),
                                   (1032, 1000, 0.75, None), (264, 16, 0.5, None),
                                   (1024, 11008, 0.7, "cluster"), (256, 4104, 0.5, "all")])
def test_batch1_single_launch_matches_batch2_kernels(variant, shape):
    """A single token (d_model <= 4096, d_ff <= 16384) runs its select, flags and
    gather in one launch (every workgroup selects, then gathers its own slice of
    neurons, with the loads of neurons known to be active after the select's
    first pass issued there), and for ideal D its select, flags and down
    projection; two tokens run a select kernel and a gather kernel. A token
    alone and the same token twice give the same bits (coefficients, threshold,
    IDX and s) and the same y to fp32 rounding. "cluster" (most coefficients
    within a relative 2^-8 of each other, with ties) and "all" (every
    coefficient equal) send the select through its radix passes."""
    from paper_2505_17701_amd import binding as cd
    from workloads import make_ternary

    dm, dff, k, dup = shape
    if dup and variant == "dual_tern":
        pytest.skip("ternary weights take three values: no clustered scores to build")
    L = make_layer(2200 + dm, dm, dff, 0.03)
    P = make_predictor(2200 + dm, dm, 64, dff, 0.05) if variant == "dual_pred" else None
    T = make_ternary(2200 + dm, dm, dff) if variant == "dual_tern" else None
    if dup:  # the matrix whose rows set the coefficient
        W = {"mono": L["W_up"], "cats": L["W_gate"], "dual_ideal": L["W_up"],
             "dual_pred": P["B_t"] if P else None}[variant]
        rows = np.arange(dff) % 16 != 0 if dup == "cluster" else np.arange(dff) >= 0
        W[rows] = W[0]
        if dup == "cluster":
            small = (np.arange(dff) % 64 - 32).astype(np.float32) * np.float32(2.0 ** -18)
            W[rows, 0] = bf16_round(small[rows])
    layer = Layer(L, P, T=T)
    x = make_tokens(2201 + dm, 1, dm)
    D = layer.d
    plan = cd.Plan(dm, dff, max_batch=2, d_rank=layer.d_rank, keep_coef=True)
    got = []
    for X in (x, np.concatenate([x, x])):
        B = X.shape[0]
        q = torch.zeros(B, dtype=torch.float64, device="cuda")
        if variant == "dual_tern":
            y = cd.countdown_ffn_tern_topk(plan, dev_bf16(X), D["W_gate"], D["W_up"], D["W_down"],
                                           D["theta_p"], k, thld_out=q)
        else:
            y = cd.countdown_ffn_topk(plan, VID[variant], dev_bf16(X), D["W_gate"], D["W_up"],
                                      D["W_down"], k, A_t=D.get("A_t"), B_t=D.get("B_t"),
                                      thld_out=q)
        idx, s_c, coef = cd.countdown_export_active(plan)
        got.append((q.cpu().numpy(), idx.cpu().numpy(), s_c.cpu().numpy(), coef.cpu().numpy(),
                    y.cpu().numpy().astype(np.float64)))
    (q1, i1, s1, c1, y1), (q2, i2, s2, c2, y2) = got
    assert np.array_equal(c1[0], c2[0]) and np.array_equal(c2[0], c2[1]), "coefficients"
    assert q1[0] == q2[0] == q2[1], (q1, q2)
    assert np.array_equal(i1, i2), (len(i1), len(i2))
    assert np.array_equal(s1[0], s2[0]) and np.array_equal(s2[0], s2[1]), "s"
    scale = max(np.abs(y2).max(), 1e-30)
    assert np.abs(y1[0] - y2[0]).max() <= 1e-5 * scale, "y"
    assert np.abs(y2[0] - y2[1]).max() <= 1e-5 * scale, "y of the two tokens"
    plan.close()


@pytest.mark.parametrize("variant", ["mono", "cats"])
def test_topk_wide_rows_single_token(variant):
    """Rows of 8192 columns at batch 1 (16 loads per lane and row in the
    coefficient kernel, d_ff above the one-launch limit's slices): the dense
    coefficients, the select and the gather."""
    layer = small(variant, 8192, 1048, 5)
    x = make_tokens(1320, 1, 8192)
    n, flips, rel = check_topk(variant, layer, x, 0.8, f"wide topk {variant}")
    if flips == 0:
        assert n == 1048 - 1 - math.floor(0.8 * 1047), n


def test_topk_rejects():
    from paper_2505_17701_amd import binding as cd

    layer = small("mono", 256, 688, 1)
    plan = cd.Plan(256, 688, max_batch=1)
    x = dev_bf16(make_tokens(1500, 1, 256))
    D = layer.d
    for bad in ({"k": 1.5}, {"k": float("nan")}, {"variant": 3}):
        kw = {"k": 0.9, "variant": 0}
        kw.update(bad)
        with pytest.raises(cd.CountdownError):
            cd.countdown_ffn_topk(plan, kw["variant"], x, D["W_gate"], D["W_up"], D["W_down"],
                                  kw["k"])
    big = cd.Plan(256, 32776, max_batch=1)
    Lb = Layer(make_layer(1501, 256, 32776, 0.03))
    with pytest.raises(cd.CountdownError):
        cd.countdown_ffn_topk(big, 0, x, Lb.d["W_gate"], Lb.d["W_up"], Lb.d["W_down"], 0.9)


def test_cif_caf_masks_match_oracle():
    """The masks behind CIF / CAF (per-token |s|, |u|, |h| quantile sets) from the GPU
    equal the oracle's up to neurons at their token's threshold; the metrics agree."""
    from paper_2505_17701_amd.metrics import cif_caf, masks_on_gpu

    w = WORKLOADS["tiny_256x688"]
    layer = Layer(w.layer())
    X = w.tokens(8)
    k = 0.7
    S, U, H = masks_on_gpu(layer.d, dev_bf16(X), k)
    ref = []
    for variant in ("dual_ideal", "mono", "cats"):
        m = np.zeros((8, w.d_ff), dtype=bool)
        for t in range(8):
            idx, _, _ = oracle.ffn_topk(variant, X[t:t + 1], layer.h["W_gate"], layer.h["W_up"],
                                        layer.h["W_down"], k)
            m[t, idx] = True
        ref.append(m)
    for got, want, name in zip((S, U, H), ref, "SUH"):
        mism = np.count_nonzero(got != want)
        assert mism <= 2, f"mask {name}: {mism} differences"
    a, b = cif_caf(S, U, H), cif_caf(*ref)
    for key in a:
        assert abs(a[key] - b[key]) <= 2e-3, (key, a[key], b[key])
    print({k2: round(v, 3) for k2, v in a.items()}, flush=True)
