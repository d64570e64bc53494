"""The per-token quantile selection on the GPU's own coefficients: for every
row length the select kernels handle (16 or 32 keys per thread, and the
LDS-keyed kernel past 32768), with distinct and with repeated values, |c| and
signed, each quantile must be exactly the linear interpolation between the
order statistics of the fp32 coefficients (numpy sort)."""
import math

import numpy as np
import pytest

from gpu_support import dev_bf16
from test_gpu_parity import Layer
from test_gpu_topk import check_topk
from workloads import make_layer, make_predictor, make_tokens
from workloads.synth import T_CALIB, bf16_round

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def exact_quantile(v, k):
    v = np.sort(v)
    n = len(v)
    h = k * (n - 1)
    lo = min(int(math.floor(h)), n - 1)
    hi = min(lo + 1, n - 1)
    return v[lo] + (h - lo) * (v[hi] - v[lo])


@pytest.mark.parametrize("dm,dff,dup", [(256, 688, None), (64, 16384, None), (64, 16392, "pairs"),
                                        (64, 32768, None), (64, 32776, None),
                                        (128, 20000, "pairs"), (64, 11008, "all"),
                                        (64, 11008, "cluster"), (64, 28672, "cluster")])
def test_select_exact_order_statistics(dm, dff, dup):
    """dup: "pairs" makes every |u| value appear twice; "all" makes every row
    equal, so all coefficients of a token tie; "cluster" gives 15/16 of the
    rows one shared body and a small varying first weight, so most
    coefficients of a token lie within a relative 2^-8 of each other, with
    many ties: both put far more keys than the candidate list holds into the
    select's first-pass bins, and the exact result then comes from its later
    radix passes."""
    from paper_2505_17701_amd import binding as cd

    L = make_layer(1900 + dff % 97, dm, dff, 0.05)
    W = L["W_up"]
    if dup == "pairs":
        W[1::2] = W[0::2][: dff // 2]
    elif dup == "all":
        W[:] = W[0]
    elif dup == "cluster":
        rows = np.arange(dff) % 16 != 0
        W[rows] = W[0]
        # first weight of each clustered row: 64 distinct bf16 values in [-2^-13, 2^-13)
        small = (np.arange(dff) % 64 - 32).astype(np.float32) * np.float32(2.0 ** -18)
        W[rows, 0] = bf16_round(small[rows])
    layer = Layer(L)
    T = 5
    X = make_tokens(1901, T, dm, purpose=T_CALIB)
    plan = cd.Plan(dm, dff, 8, 0, keep_coef=True)
    D = layer.d
    xd = dev_bf16(X)
    cd.countdown_ffn_mono(plan, xd, D["W_gate"], D["W_up"], D["W_down"], math.inf)
    coef = cd.countdown_export_active(plan)[2].cpu().numpy().astype(np.float64)[:T]
    if dup == "pairs":
        assert np.array_equal(np.abs(coef[:, 0::2][:, : dff // 2]), np.abs(coef[:, 1::2]))
    elif dup == "all":
        assert (np.abs(coef) == np.abs(coef[:, :1])).all()
    elif dup == "cluster":
        c = np.abs(coef[:, rows])
        assert (c.max(axis=1) - c.min(axis=1) < 2.0 ** -8 * c.max(axis=1)).all()
        assert all(len(np.unique(r)) > 16 for r in c)
    for k in (0.0, 0.3, 0.5, 0.9, 0.999, 1.0):
        _, q = cd.countdown_calibrate(plan, cd.CD_VARIANT_MONO, xd, k, W_up=D["W_up"])
        q = q.cpu().numpy()
        for t in range(T):
            assert q[t] == exact_quantile(np.abs(coef[t]), k), (dff, dup, k, t)
    plan.close()


@pytest.mark.parametrize("dff,cluster", [(688, False), (20000, False), (11008, True),
                                         (20000, True)])
def test_select_signed_scores(dff, cluster):
    """The predictor's signed score: the quantile of the signed values. With
    cluster, 15/16 of the B_t rows share one body and differ in a small first
    entry, so most scores of a token lie within a relative 2^-8 of each other
    (with ties): the select's later radix passes on signed keys."""
    from paper_2505_17701_amd import binding as cd

    dm, dr = 64, 8
    L = make_layer(1950, dm, dff, 0.05)
    P = make_predictor(1950, dm, dr, dff, 0.3)
    if cluster:
        Bt = P["B_t"]
        rows = np.arange(dff) % 16 != 0
        Bt[rows] = Bt[0]
        small = (np.arange(dff) % 64 - 32).astype(np.float32) * np.float32(2.0 ** -19)
        Bt[rows, 0] = bf16_round(small[rows])
    layer = Layer(L, P)
    T = 4
    X = make_tokens(1951, T, dm, purpose=T_CALIB)
    plan = cd.Plan(dm, dff, 8, dr, keep_coef=True)
    D = layer.d
    xd = dev_bf16(X)
    cd.countdown_ffn_dual(plan, xd, D["W_gate"], D["W_up"], D["W_down"], math.inf,
                          A_t=D["A_t"], B_t=D["B_t"])
    coef = cd.countdown_export_active(plan)[2].cpu().numpy().astype(np.float64)[:T]
    if cluster:
        c = coef[:, rows]
        assert (c.max(axis=1) - c.min(axis=1) < 2.0 ** -8 * np.abs(c).max(axis=1)).all()
        assert all(len(np.unique(r)) > 8 for r in c)
    else:
        assert (coef < 0).any() and (coef > 0).any()
    for k in (0.1, 0.5, 0.9):
        _, q = cd.countdown_calibrate(plan, cd.CD_VARIANT_DUAL_PRED, xd, k, A_t=D["A_t"],
                                      B_t=D["B_t"])
        q = q.cpu().numpy()
        for t in range(T):
            assert q[t] == exact_quantile(coef[t], k), (dff, cluster, k, t)
    plan.close()


@pytest.mark.parametrize("shape", [(512, 24584, 2, 0.9), (256, 32768, 1, 0.7)])
def test_topk_long_rows(shape):
    """The per-token path with 32 keys per thread of the select (d_ff > 16384)."""
    dm, dff, B, k = shape
    layer = Layer(make_layer(1960 + B, dm, dff, 0.03))
    x = make_tokens(1961, B, dm)
    n, flips, rel = check_topk("mono", layer, x, k, f"long topk {shape}")
    if B == 1 and flips == 0:
        assert n == dff - 1 - math.floor(k * (dff - 1))


@pytest.mark.parametrize("variant", ["mono", "cats", "dual_ideal", "dual_pred"])
@pytest.mark.parametrize("dup", [None, "pairs", "all", "cluster"])
def test_per_token_call_exact_order_statistics(variant, dup):
    """The per-token FFN call's own select (|c| keys, or signed keys for the
    predictor score): on six calls in a row of one plan, with batch sizes and
    k that change from call to call, every token's threshold is exactly the
    interpolated order statistic of the coefficients the call wrote. "all"
    (every coefficient of a token equal) and "cluster" (most within a relative
    2^-8, with ties) put thousands of keys into one first-pass bin, so the
    radix passes finish those."""
    from paper_2505_17701_amd import binding as cd

    dm, dff, dr = 64, 11008, 8
    L = make_layer(1970, dm, dff, 0.05)
    P = make_predictor(1970, dm, dr, dff, 0.3) if variant == "dual_pred" else None
    # the matrix whose rows set the coefficient (for ideal D both factors)
    mats = {"mono": [L["W_up"]], "cats": [L["W_gate"]], "dual_ideal": [L["W_up"], L["W_gate"]],
            "dual_pred": [P["B_t"] if P is not None else None]}[variant]
    rows = np.arange(dff) % 16 != 0
    for W in mats:
        if dup == "pairs":
            W[1::2] = W[0::2][: dff // 2]
        elif dup == "all":
            W[:] = W[0]
        elif dup == "cluster":
            W[rows] = W[0]
    if dup == "cluster":  # a small varying first weight in the coefficient's own matrix
        W = mats[0]
        small = (np.arange(dff) % 64 - 32).astype(np.float32) * np.float32(2.0 ** -18)
        W[rows, 0] = bf16_round(small[rows])
    layer = Layer(L, P)
    D = layer.d
    vid = {"mono": cd.CD_VARIANT_MONO, "cats": cd.CD_VARIANT_CATS,
           "dual_ideal": cd.CD_VARIANT_DUAL_IDEAL, "dual_pred": cd.CD_VARIANT_DUAL_PRED}[variant]
    plan = cd.Plan(dm, dff, 8, dr if variant == "dual_pred" else 0, keep_coef=True)
    signed = variant == "dual_pred"
    for call, (B, k) in enumerate([(5, 0.9), (3, 0.5), (8, 0.0), (1, 1.0), (2, 0.999), (1, 0.7)]):
        X = make_tokens(1971 + call, B, dm, purpose=T_CALIB)
        q = torch.empty(B, dtype=torch.float64, device="cuda")
        cd.countdown_ffn_topk(plan, vid, dev_bf16(X), D["W_gate"], D["W_up"], D["W_down"], k,
                              A_t=D.get("A_t"), B_t=D.get("B_t"), thld_out=q)
        coef = cd.countdown_export_active(plan)[2].cpu().numpy().astype(np.float64)[:B]
        q = q.cpu().numpy()
        if dup == "all" and variant != "dual_ideal":
            assert (coef == coef[:, :1]).all()
        for t in range(B):
            v = coef[t] if signed else np.abs(coef[t])
            assert q[t] == exact_quantile(v, k), (variant, dup, call, B, k, t)
    plan.close()
