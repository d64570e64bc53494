"""GPU parity of the residual-stream entry point (countdown_ffn_residual):
h_out = h_in + y_prev, x = bf16(RMSNorm(h_out)), then the FFN on x. The
residual/normalisation step joins the layers of the stack workload; the FFN
part is checked against the oracle on the GPU's own x (teacher forcing), the
normalisation against the oracle's residual_rmsnorm."""
import numpy as np
import pytest

import oracle
from gpu_support import dev_bf16
from test_gpu_parity import Layer, calibrated, check_call, plan_for
from workloads import WORKLOADS, make_layer, make_predictor
from workloads.synth import bf16_to_f32, stream

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

EPS = 1e-5
X_SLACK = 1e-5  # relative: fp32 sum of squares and scaling against the fp64 oracle

VID = {"mono": 0, "dual_ideal": 1, "dual_pred": 2, "dense": 3}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def residual_inputs(seed, B, d_model, with_y=True):
    rng = stream(9000 + seed, B, d_model)
    h = rng.standard_normal((B, d_model)).astype(np.float32)
    y = (0.5 * rng.standard_normal((B, d_model))).astype(np.float32) if with_y else None
    return h, y


def run_residual(plan, variant, layer, h_in, y_prev, thld):
    from paper_2505_17701_amd import binding as cd

    B, dm = h_in.shape
    hd = torch.from_numpy(h_in).cuda()
    yp = None if y_prev is None else torch.from_numpy(y_prev).cuda()
    h_out = torch.empty_like(hd)
    x_out = torch.empty((B, dm), dtype=torch.bfloat16, device="cuda")
    D = layer.d
    y = cd.countdown_ffn_residual(plan, VID[variant], hd, yp, h_out, x_out, D["W_gate"],
                                  D["W_up"], D["W_down"], thld, A_t=D.get("A_t"),
                                  B_t=D.get("B_t"), eps=EPS)
    idx, s_c, coef = cd.countdown_export_active(plan)
    x_bits = x_out.view(torch.int16).cpu().numpy().view(np.uint16)
    return (h_out.cpu().numpy(), x_bits,
            (y.cpu().numpy().astype(np.float64), idx.cpu().numpy(), s_c.cpu().numpy(),
             None if coef is None else coef.cpu().numpy()))


def check_norm(h_in, y_prev, h_gpu, x_bits, label):
    # h_out: one fp32 addition of two fp32 values, correctly rounded
    ref_h = h_in if y_prev is None else (h_in.astype(np.float64) + y_prev).astype(np.float32)
    np.testing.assert_array_equal(h_gpu.view(np.uint32), ref_h.view(np.uint32), err_msg=label)
    # x: within half a bf16 ulp of the exact normalised value (plus the fp32 slack)
    x = bf16_to_f32(x_bits).astype(np.float64)
    for b in range(h_in.shape[0]):
        _, r = oracle.residual_rmsnorm(h_in[b], None if y_prev is None else y_prev[b], eps=EPS)
        mag = np.maximum(np.abs(r), np.abs(x[b]))
        ulp = np.exp2(np.floor(np.log2(np.maximum(mag, 1e-30))) - 7)
        err = np.abs(x[b] - r)
        bad = err > 0.5 * ulp + X_SLACK * np.abs(r)
        assert not bad.any(), f"{label}: token {b}, {bad.sum()} x values off, worst {err.max():.3e}"


@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "dual_pred", "dense"])
@pytest.mark.parametrize("shape", [(264, 520, 1), (1032, 1000, 3), (4096, 1376, 2), (2048, 776, 8)])
def test_residual_layer(variant, shape):
    dm, dff, B = shape
    L = make_layer(950 + dm, dm, dff, 0.03)
    P = make_predictor(950 + dm, dm, 64, dff, 0.05) if variant == "dual_pred" else None
    layer = Layer(L, P)
    h_in, y_prev = residual_inputs(dm + B, B, dm, with_y=(B != 2))
    # threshold: the variant's calibrated value on normalised inputs of the same recipe
    X = np.stack([oracle.residual_rmsnorm(h_in[b], None if y_prev is None else y_prev[b],
                                          eps=EPS)[1] for b in range(B)])
    Xb = np.array([np.float32(v) for v in X.ravel()], dtype=np.float32).reshape(X.shape)
    from workloads.synth import bf16_round
    thld = 0.0 if variant == "dense" else float(np.float32(oracle.calibrate(
        variant, bf16_round(Xb), 0.8, W_gate=L["W_gate"], W_up=L["W_up"],
        A_t=None if P is None else P["A_t"], B_t=None if P is None else P["B_t"])[0]))
    plan = plan_for(layer, max_batch=B)
    label = f"residual {variant} {shape}"
    h_gpu, x_bits, out = run_residual(plan, variant, layer, h_in, y_prev, thld)
    check_norm(h_in, y_prev, h_gpu, x_bits, label)
    check_call(variant, layer, x_bits, thld, out, label)


def test_residual_rejects_overlap():
    from paper_2505_17701_amd import binding as cd

    layer = Layer(make_layer(977, 264, 520, 0.03))
    plan = plan_for(layer, max_batch=2)
    D = layer.d
    h = torch.zeros((2, 264), dtype=torch.float32, device="cuda")
    x = torch.empty((2, 264), dtype=torch.bfloat16, device="cuda")
    y = torch.empty_like(h)
    with pytest.raises(cd.CountdownError):  # h_out aliasing h_in
        cd.countdown_ffn_residual(plan, 0, h, None, h, x, D["W_gate"], D["W_up"], D["W_down"],
                                  1.0, y=y)
    with pytest.raises(cd.CountdownError):  # eps NaN
        cd.countdown_ffn_residual(plan, 0, h, None, torch.empty_like(h), x, D["W_gate"],
                                  D["W_up"], D["W_down"], 1.0, eps=float("nan"), y=y)
    # y_prev may be y itself
    h2 = torch.empty_like(h)
    y.zero_()
    cd.countdown_ffn_residual(plan, 0, h, y, h2, x, D["W_gate"], D["W_up"], D["W_down"], 1.0,
                              y=y)
    torch.cuda.synchronize()


def test_stack_teacher_forced():
    """Three stacked 7B-shaped predictor layers run back to back on the GPU (the
    residual stream passed from layer to layer); every layer is checked against
    the oracle on the inputs the GPU layer received."""
    w = WORKLOADS["stack32_llama7b_pred"]
    B = 1
    rng = stream(9100, w.d_model)
    h = rng.standard_normal((B, w.d_model)).astype(np.float32)
    y_prev = None
    for l in range(3):
        L = w.layer(layer=l)
        P = w.predictor(layer=l)
        layer = Layer(L, P)
        X = np.stack([oracle.residual_rmsnorm(h[b], None if y_prev is None else y_prev[b],
                                              eps=EPS)[1] for b in range(B)]).astype(np.float32)
        from workloads.synth import bf16_round
        thld = float(np.float32(oracle.calibrate("dual_pred", bf16_round(X), 0.9, A_t=P["A_t"],
                                                 B_t=P["B_t"])[0]))
        plan = plan_for(layer, max_batch=B)
        label = f"stack layer {l}"
        h_gpu, x_bits, out = run_residual(plan, "dual_pred", layer, h, y_prev, thld)
        check_norm(h, y_prev, h_gpu, x_bits, label)
        n, flips, rel = check_call("dual_pred", layer, x_bits, thld, out, label)
        print(f"{label}: n={n} flips={flips} rel={rel:.2e}", flush=True)
        h, y_prev = h_gpu, out[0].astype(np.float32)
        del layer, plan
        torch.cuda.empty_cache()
