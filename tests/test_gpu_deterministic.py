"""Deterministic mode (CD_PLAN_DETERMINISTIC): the down projection stores one
partial sum per neuron range and a second kernel adds them in ascending range
order, so y no longer depends on the order in which fp32 atomics arrive.
Checked through the C ABI for every variant and batch tile (the VALU down
kernel at 1-2 tokens, the MFMA one at 4-8), the per-token path and the
residual stack step: repeated calls give bit-identical y, y matches the oracle
to the parity bar, and it agrees with the atomic mode to fp32 rounding."""
import numpy as np
import pytest

import oracle
from gpu_support import dev_bf16
from test_gpu_parity import Layer, check_call, run_gpu
from workloads import make_layer, make_predictor, make_ternary, make_tokens
from workloads.synth import T_CALIB

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


DM, DFF, RANK = 1024, 4104, 64


@pytest.fixture(scope="module")
def layer():
    L = make_layer(2100, DM, DFF, 0.03)
    P = make_predictor(2100, DM, RANK, DFF, 0.05)
    T = make_ternary(2100, DM, DFF)
    return Layer(L, P, T)


def thld_for(variant, layer, k=0.8):
    if variant == "dense":
        return 0.0
    H = layer.h
    X = make_tokens(2100, 32, DM, purpose=T_CALIB)
    t, _ = oracle.calibrate(variant, X, k, W_gate=H["W_gate"], W_up=H["W_up"], A_t=H["A_t"],
                            B_t=H["B_t"], theta_t=H["theta_t"])
    return float(np.float32(t))


@pytest.mark.parametrize("B", [1, 2, 4, 8])
@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "dual_pred", "cats", "dense",
                                     "dual_tern"])
def test_deterministic_y_is_bit_identical(layer, variant, B):
    from paper_2505_17701_amd import binding as cd

    x = make_tokens(2101 + B, B, DM)
    thld = thld_for(variant, layer)
    rank = RANK if variant == "dual_pred" else 0
    det = cd.Plan(DM, DFF, max_batch=8, d_rank=rank, keep_coef=True, deterministic=True)
    outs = [run_gpu(det, variant, layer, x, thld) for _ in range(4)]
    for o in outs[1:]:
        assert np.array_equal(o[0], outs[0][0]), "deterministic y differs between calls"
        assert np.array_equal(o[1], outs[0][1])
    check_call(variant, layer, x, thld, outs[0], f"deterministic {variant} B={B}")
    atom = cd.Plan(DM, DFF, max_batch=8, d_rank=rank, keep_coef=True)
    ya = run_gpu(atom, variant, layer, x, thld)[0]
    yd = outs[0][0]
    assert np.max(np.abs(yd - ya)) <= 1e-5 * np.max(np.abs(ya)) + 1e-30
    det.close()
    atom.close()


@pytest.mark.parametrize("variant", ["mono", "cats"])
def test_deterministic_wide_rows_single_token(variant):
    """Rows of 8192 columns at batch 1 (16 loads per lane and row):
    coefficients, s and y are the same bits on every call."""
    from paper_2505_17701_amd import binding as cd

    dm, dff = 8192, 1048
    wide = Layer(make_layer(2130, dm, dff, 0.02))
    x = make_tokens(2131, 1, dm)
    u, g, _ = oracle.coefficients(x, wide.h["W_gate"], wide.h["W_up"])
    c = np.abs(u if variant == "mono" else g / (1.0 + np.exp(-g)))
    thld = float(np.float32(np.quantile(c, 0.8)))
    det = cd.Plan(dm, dff, max_batch=1, keep_coef=True, deterministic=True)
    outs = [run_gpu(det, variant, wide, x, thld) for _ in range(3)]
    for o in outs[1:]:
        for a, b in zip(o, outs[0]):
            assert np.array_equal(a, b), "deterministic output differs between calls"
    check_call(variant, wide, x, thld, outs[0], f"deterministic wide {variant}")
    det.close()


@pytest.mark.parametrize("B", [1, 3])
@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "dual_pred"])
def test_deterministic_per_token_path(layer, variant, B):
    from paper_2505_17701_amd import binding as cd

    vid = {"mono": cd.CD_VARIANT_MONO, "dual_ideal": cd.CD_VARIANT_DUAL_IDEAL,
           "dual_pred": cd.CD_VARIANT_DUAL_PRED}[variant]
    x = dev_bf16(make_tokens(2110, B, DM))
    D = layer.d
    det = cd.Plan(DM, DFF, max_batch=B, d_rank=RANK if variant == "dual_pred" else 0,
                  deterministic=True)
    ys = []
    for _ in range(3):
        y = cd.countdown_ffn_topk(det, vid, x, D["W_gate"], D["W_up"], D["W_down"], 0.85,
                                  A_t=D["A_t"] if variant == "dual_pred" else None,
                                  B_t=D["B_t"] if variant == "dual_pred" else None)
        ys.append(y.cpu().numpy())
    for y in ys[1:]:
        assert np.array_equal(y, ys[0])
    det.close()


def test_deterministic_residual_step(layer):
    from paper_2505_17701_amd import binding as cd

    D = layer.d
    h = torch.from_numpy(make_tokens(2120, 2, DM, as_fp32=True)).cuda()
    yp = torch.from_numpy(make_tokens(2121, 2, DM, as_fp32=True) * 0.1).cuda()
    det = cd.Plan(DM, DFF, max_batch=2, d_rank=RANK, deterministic=True)
    thld = thld_for("dual_pred", layer)
    outs = []
    for _ in range(3):
        h_out = torch.empty_like(h)
        x_out = torch.empty((2, DM), dtype=torch.bfloat16, device="cuda")
        y = torch.empty_like(h)
        cd.countdown_ffn_residual(det, cd.CD_VARIANT_DUAL_PRED, h, yp, h_out, x_out,
                                  D["W_gate"], D["W_up"], D["W_down"], thld, A_t=D["A_t"],
                                  B_t=D["B_t"], y=y)
        outs.append((h_out.cpu().numpy(), y.cpu().numpy()))
    for o in outs[1:]:
        assert np.array_equal(o[0], outs[0][0]) and np.array_equal(o[1], outs[0][1])
    det.close()
