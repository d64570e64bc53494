"""Predictor training (Sec. 4, Alg. 1) on synthetic activations: targets from
the HIP per-token ideal-D path, BCE + AdamW in PyTorch, inference through the
HIP predictor path. With random synthetic weights the masks carry no low-rank
structure, so only learning (against the untrained start) is asserted, and
the trained predictor's index sets are checked against the oracle."""
import numpy as np
import pytest

import oracle
from gpu_support import IDX_BAND, dev_bf16
from test_gpu_parity import Layer
from workloads import make_layer, make_tokens
from workloads.synth import T_CALIB

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def test_train_low_rank_predictor():
    from paper_2505_17701_amd.predictor import (calibrated_threshold, f1_score, ideal_masks,
                                                 predicted_masks, train_low_rank)

    dm, dff, k = 512, 1376, 0.7
    layer = Layer(make_layer(1600, dm, dff, 0.03))
    Xtr = dev_bf16(make_tokens(1600, 1024, dm, purpose=T_CALIB))
    Xte_h = make_tokens(1601, 64, dm)
    Xte = dev_bf16(Xte_h)
    Ytr = ideal_masks(layer.d, Xtr, k)
    Yte = ideal_masks(layer.d, Xte, k)
    assert abs(Ytr.float().mean().item() - (1 - k)) < 0.01
    A0, B0, _ = train_low_rank(Xtr, Ytr, 64, epochs=0)
    A, B, log = train_low_rank(Xtr, Ytr, 64, epochs=6)
    assert log["epoch_loss"][-1] < log["epoch_loss"][0]
    scores = {}
    for name, (At, Bt) in (("start", (A0, B0)), ("trained", (A, B))):
        th = calibrated_threshold(At, Bt, Xtr[:256], k)
        P = predicted_masks(layer.d, At, Bt, Xte, th)
        scores[name] = f1_score(P.cpu().numpy(), Yte.cpu().numpy())
    print(f"F1 on S^{k}: start {scores['start']:.3f} trained {scores['trained']:.3f}", flush=True)
    assert scores["trained"] > scores["start"] + 0.02
    # the HIP predictor path on the trained weights matches the oracle's index sets
    Ah = A.view(torch.int16).cpu().numpy().view(np.uint16)
    Bh = B.view(torch.int16).cpu().numpy().view(np.uint16)
    P0 = predicted_masks(layer.d, A, B, Xte[:4], 0.0).cpu().numpy()
    for t in range(4):
        idx_o, _, c = oracle.ffn_dual_pred(Xte_h[t:t + 1], layer.h["W_gate"], layer.h["W_up"],
                                           layer.h["W_down"], Ah, Bh, 0.0, want_coef=True)
        want = np.zeros(dff, dtype=bool)
        want[idx_o] = True
        diff = np.nonzero(P0[t] != want)[0]
        scale = np.sqrt(np.mean(c[0] ** 2))
        assert np.all(np.abs(c[0][diff]) <= IDX_BAND * scale), (t, len(diff))


def test_train_ternary_predictor():
    """The ternary predictor (Sec. 6) trained by Alg. 1 with the straight-through
    estimator; inference through the HIP ternary path."""
    from paper_2505_17701_amd.predictor import (calibrated_threshold_tern, f1_score, ideal_masks,
                                                 packed_ternary, predicted_masks_tern,
                                                 train_ternary)
    from workloads import make_ternary

    dm, dff, k = 512, 1376, 0.7
    layer = Layer(make_layer(1610, dm, dff, 0.03))
    Xtr = dev_bf16(make_tokens(1610, 1024, dm, purpose=T_CALIB))
    Xte_h = make_tokens(1611, 64, dm)
    Xte = dev_bf16(Xte_h)
    Ytr = ideal_masks(layer.d, Xtr, k)
    Yte = ideal_masks(layer.d, Xte, k)
    T, log = train_ternary(Xtr, Ytr, epochs=6)
    assert T.dtype == np.int8 and set(np.unique(T)) <= {-1, 0, 1}
    assert log["epoch_loss"][-1] < log["epoch_loss"][0]
    scores = {}
    for name, theta in (("random", make_ternary(1610, dm, dff)), ("trained", T)):
        tp = packed_ternary(theta)
        th = calibrated_threshold_tern(tp, Xtr[:256], k, dff)
        P = predicted_masks_tern(layer.d, tp, Xte, th)
        scores[name] = f1_score(P.cpu().numpy(), Yte.cpu().numpy())
    print(f"ternary F1 on S^{k}: random {scores['random']:.3f} trained {scores['trained']:.3f} "
          f"zeros {log['zero_frac']:.2f}", flush=True)
    assert scores["trained"] > scores["random"] + 0.02
    tp = packed_ternary(T)
    P0 = predicted_masks_tern(layer.d, tp, Xte[:4], 0.0).cpu().numpy()
    for t in range(4):
        idx_o, _, c = oracle.ffn_dual_tern(Xte_h[t:t + 1], layer.h["W_gate"], layer.h["W_up"],
                                           layer.h["W_down"], T, 0.0, want_coef=True)
        want = np.zeros(dff, dtype=bool)
        want[idx_o] = True
        diff = np.nonzero(P0[t] != want)[0]
        scale = np.sqrt(np.mean(c[0] ** 2))
        assert np.all(np.abs(c[0][diff]) <= IDX_BAND * scale), (t, len(diff))
