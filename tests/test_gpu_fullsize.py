"""GPU parity at the full workload shapes, in the launch configuration the
bench times (one plan per shape, max_batch = the workload's largest batch)."""
import numpy as np
import pytest

from workloads import WORKLOADS

from test_gpu_parity import Layer, calibrated, compare, plan_for

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.fixture(scope="module")
def llama7b():
    w = WORKLOADS["llama7b_4096x11008"]
    return w, Layer(w.layer())


@pytest.mark.parametrize("variant", ["mono", "dual_ideal", "cats"])
@pytest.mark.parametrize("k", [0.9, 0.7, 0.5])
def test_llama7b_layer(llama7b, variant, k):
    w, layer = llama7b
    thld = calibrated(variant, layer, w.wid, k, T=32, outlier_frac=w.outlier_frac)
    plan = plan_for(layer)
    X = w.tokens(3)
    for t in range(3):
        n, flips, rel = compare(plan, variant, layer, X[t:t + 1], thld,
                                f"7b {variant} k={k} tok{t}")
        assert abs(n / w.d_ff - (1 - k)) < 0.15, n
        print(f"7b {variant} k={k} tok{t}: n={n} flips={flips} rel_err={rel:.2e}", flush=True)


@pytest.mark.parametrize("variant", ["mono", "cats"])
def test_llama7b_batch2(llama7b, variant):
    """Two tokens: the one-row kernel stages them in LDS (union over the batch)."""
    w, layer = llama7b
    thld = calibrated(variant, layer, w.wid, 0.9, T=32, outlier_frac=w.outlier_frac)
    plan = plan_for(layer, max_batch=2)
    n, flips, rel = compare(plan, variant, layer, w.tokens(2), thld, f"7b {variant} B=2")
    print(f"7b {variant} B=2: n={n} flips={flips} rel_err={rel:.2e}", flush=True)


@pytest.fixture(scope="module")
def llama3_pred():
    w = WORKLOADS["llama3_8b_4096x14336_pred"]
    return w, Layer(w.layer(), w.predictor())


@pytest.mark.parametrize("B", [1, 2, 4, 8])
def test_llama3_predictor_batch_union(llama3_pred, B):
    w, layer = llama3_pred
    thld = calibrated("dual_pred", layer, w.wid, 0.9, T=32)
    plan = plan_for(layer, max_batch=8)
    X = w.tokens(B)
    n, flips, rel = compare(plan, "dual_pred", layer, X, thld, f"8b pred B={B}")
    expect = 1 - 0.9 ** B
    assert abs(n / w.d_ff - expect) < 0.1, (n, expect)
    print(f"8b pred B={B}: n={n} flips={flips} rel_err={rel:.2e}", flush=True)


@pytest.mark.parametrize("variant", ["mono", "cats"])
def test_llama3_shape_mono_and_cats(llama3_pred, variant):
    """The kernel-speed sweep's M and CATS lines at the 8B shape (k 0.6)."""
    w, layer = llama3_pred
    thld = calibrated(variant, layer, w.wid, 0.6, T=16)
    plan = plan_for(layer, max_batch=8)
    n, flips, rel = compare(plan, variant, layer, w.tokens(1), thld, f"8b {variant} k=0.6")
    assert abs(n / w.d_ff - 0.4) < 0.15, n
    print(f"8b {variant} k=0.6: n={n} flips={flips} rel_err={rel:.2e}", flush=True)


@pytest.fixture(scope="module")
def llama70b():
    w = WORKLOADS["llama70b_8192x28672"]
    layer = Layer(w.layer())
    yield w, layer
    del layer
    torch.cuda.empty_cache()


@pytest.mark.parametrize("k", [0.9, 0.7])
def test_llama70b_layer(llama70b, k):
    w, layer = llama70b
    thld = calibrated("mono", layer, w.wid, k, T=8)
    plan = plan_for(layer)
    n, flips, rel = compare(plan, "mono", layer, w.tokens(1), thld, f"70b mono k={k}")
    print(f"70b mono k={k}: n={n} flips={flips} rel_err={rel:.2e}", flush=True)
    compare(plan, "dense", layer, w.tokens(1), 0.0, "70b dense", check_coef=False)


def test_llama70b_per_token_and_calibration(llama70b):
    """The 70B-shaped layer (d_ff 28672: the select with 32 keys per thread): the
    per-token path at batch 2 and the GPU calibration against the oracle."""
    import numpy as np

    import oracle
    from gpu_support import dev_bf16
    from paper_2505_17701_amd import binding as cd
    from test_gpu_topk import check_topk
    from workloads.synth import T_CALIB

    w, layer = llama70b
    n, flips, rel = check_topk("mono", layer, w.tokens(2), 0.9, "70b mono topk B=2")
    print(f"70b mono topk B=2: n={n} flips={flips} rel={rel:.2e}", flush=True)
    X = w.tokens(4, purpose=T_CALIB)
    plan = cd.Plan(w.d_model, w.d_ff, 4)
    th, q = cd.countdown_calibrate(plan, cd.CD_VARIANT_MONO, dev_bf16(X), 0.7,
                                   W_up=layer.d["W_up"])
    plan.close()
    t_o, q_o = oracle.calibrate("mono", X, 0.7, W_up=layer.h["W_up"])
    np.testing.assert_allclose(q.cpu().numpy(), q_o, rtol=2e-5)
    assert abs(float(th.item()) - t_o) <= 2e-5 * abs(t_o)
