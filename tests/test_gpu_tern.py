"""GPU parity of the ternary predictor path (TernaryLinear, Sec. 6): the
packed theta through countdown_ffn_tern / _tern_topk / calibrate_tern
against the oracle's ternary functions on the unpacked int8 theta. Same
rules as the other parity tests: IDX exact outside the band around thld, y
on the GPU's index set, the score within an fp32 dot-product bound."""
import math

import numpy as np
import pytest

import oracle
from gpu_support import dev_bf16
from test_gpu_parity import Layer, check_call, run_gpu
from test_gpu_topk import check_topk
from workloads import WORKLOADS, make_layer, make_ternary, make_tokens
from workloads.synth import T_CALIB

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def tern_layer(dm, dff, seed):
    return Layer(make_layer(1700 + seed, dm, dff, 0.03), T=make_ternary(1700 + seed, dm, dff))


def thld_at(layer, x, q):
    """A threshold at quantile q of token 0's ternary score (the score is signed)."""
    s = oracle.ternary_predictor(x[:1], layer.h["theta_t"])[0]
    return float(np.float32(np.quantile(s, q)))


@pytest.mark.parametrize("shape", [(8, 16, 1), (256, 688, 1), (520, 776, 2), (1032, 1000, 3),
                                   (4096, 1376, 4), (1024, 520, 5), (2048, 776, 8),
                                   (8192, 264, 4),
                                   # 5-8 tokens at 3585-4096 columns: the score on MFMA,
                                   # ragged last chunk and ragged neuron count
                                   (3592, 1000, 5), (3848, 264, 7), (4088, 1032, 8),
                                   (4096, 776, 6)])
def test_tern_parity(shape):
    from paper_2505_17701_amd import binding as cd

    dm, dff, B = shape
    layer = tern_layer(dm, dff, dm + dff)
    x = make_tokens(1800 + dm, B, dm)
    plan = cd.Plan(dm, dff, max_batch=B, keep_coef=True)
    for q in (0.5, 0.9):
        th = thld_at(layer, x, q)
        n, flips, rel = check_call("dual_tern", layer, x, th, run_gpu(plan, "dual_tern", layer, x, th),
                                   f"tern {shape} q={q}")
        # at q 0.5 the union over 5-8 tokens (1 - 0.5^B of the neurons) may be all of them
        assert 0 < n <= dff and (q < 0.9 or n < dff), (n, dff)
    plan.close()


def test_tern_all_and_none():
    from paper_2505_17701_amd import binding as cd

    layer = tern_layer(512, 1000, 1)
    x = make_tokens(1900, 3, 512)
    plan = cd.Plan(512, 1000, max_batch=3, keep_coef=True)
    out = run_gpu(plan, "dual_tern", layer, x, -math.inf)
    assert len(out[1]) == 1000
    check_call("dual_tern", layer, x, -math.inf, out, "tern all")
    y, idx, _, _ = run_gpu(plan, "dual_tern", layer, x, math.inf)
    assert len(idx) == 0 and not y.any()
    plan.close()


@pytest.mark.parametrize("dm", [1024, 4096])
def test_tern_calibration_matches_oracle(dm):
    """Calibration runs the coefficient kernel on batches of 8 (at d_model 4096
    the MFMA score) and the exact select on the dense scores."""
    from paper_2505_17701_amd import binding as cd

    layer = tern_layer(dm, 1376, 2)
    X = make_tokens(1950, 40, dm, purpose=T_CALIB)
    for k in (0.5, 0.9):
        plan = cd.Plan(dm, 1376, max_batch=8)
        th, q = cd.countdown_calibrate_tern(plan, dev_bf16(X), layer.d["theta_p"], k)
        plan.close()
        tau, q_o = oracle.calibrate("dual_tern", X, k, theta_t=layer.h["theta_t"])
        c = oracle.ternary_predictor(X, layer.h["theta_t"])
        scale = np.maximum(np.abs(q_o), np.sqrt(np.mean(c * c, axis=1)))
        assert np.all(np.abs(q.cpu().numpy() - q_o) <= 1e-5 * scale)
        assert abs(float(th.item()) - tau) <= 1e-5 * float(scale.mean()) + abs(tau) * 2 ** -23


@pytest.mark.parametrize("shape", [(256, 688, 1, 0.9), (1032, 1000, 3, 0.75), (2048, 776, 8, 0.9),
                                   (4096, 1376, 2, 0.5), (4096, 1000, 6, 0.7), (3592, 520, 8, 0.9)])
def test_tern_topk(shape):
    dm, dff, B, k = shape
    layer = tern_layer(dm, dff, 3 + dm)
    x = make_tokens(2000 + dm, B, dm)
    n, flips, rel = check_topk("dual_tern", layer, x, k, f"tern topk {shape}")
    if B == 1 and flips == 0:
        assert n == dff - 1 - math.floor(k * (dff - 1))


def test_tern_llama3_8b_full_size():
    """The 8B-shaped layer (4096 x 14336) with a seeded ternary predictor at batch 1,
    4 and 8, thresholds calibrated on the GPU at k = 0.9, against the oracle."""
    from paper_2505_17701_amd import binding as cd

    w = WORKLOADS["llama3_8b_4096x14336_pred"]
    layer = Layer(w.layer(), T=w.ternary())
    cal = cd.Plan(w.d_model, w.d_ff, max_batch=8)
    th, _ = cd.countdown_calibrate_tern(cal, dev_bf16(w.tokens(64, purpose=T_CALIB)),
                                        layer.d["theta_p"], 0.9)
    cal.close()
    th = float(th.item())
    for B in (1, 4, 8):
        plan = cd.Plan(w.d_model, w.d_ff, max_batch=B, keep_coef=True)
        x = w.tokens(B)
        n, flips, rel = check_call("dual_tern", layer, x, th, run_gpu(plan, "dual_tern", layer, x, th),
                                   f"8b tern B={B}")
        print(f"8b tern B={B}: n={n} flips={flips} rel={rel:.2e}", flush=True)
        plan.close()


def test_tern_rejects():
    from paper_2505_17701_amd import binding as cd

    layer = tern_layer(256, 688, 4)
    plan = cd.Plan(256, 688, max_batch=1)
    x = dev_bf16(make_tokens(2100, 1, 256))
    D = layer.d
    with pytest.raises(cd.CountdownError):
        cd.countdown_ffn_tern(plan, x, D["W_gate"], D["W_up"], D["W_down"], D["theta_p"],
                              float("nan"))
    with pytest.raises(cd.CountdownError):  # the generic calibration does not take theta
        cd.countdown_calibrate(plan, cd.CD_VARIANT_DUAL_TERN, x, 0.9, W_gate=D["W_gate"],
                               W_up=D["W_up"])
    h = torch.zeros((1, 256), dtype=torch.float32, device="cuda")
    with pytest.raises(cd.CountdownError):  # no ternary variant in the residual stack
        cd.countdown_ffn_residual(plan, cd.CD_VARIANT_DUAL_TERN, h, None, torch.zeros_like(h),
                                  torch.zeros((1, 256), dtype=torch.bfloat16, device="cuda"),
                                  D["W_gate"], D["W_up"], D["W_down"])
    plan.close()
