"""The seeded input generators: bf16 rounding, determinism, recipes."""
import numpy as np
import torch

from workloads import WORKLOADS, bf16_round, bf16_to_f32, make_tokens, outlier_channels
from workloads.synth import T_CALIB, T_EVAL


def test_bf16_round_matches_torch_rne():
    rng = np.random.default_rng(0)
    a = np.concatenate([
        rng.standard_normal(100000).astype(np.float32) * np.float32(3.0),
        np.array([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, 3.4e38, -3.4e38, 1e-40, -1e-40,
                  1.00390625, 1.01171875, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8], dtype=np.float32),
        # exact ties between two bf16 neighbours: lower mantissa bits 0x8000
        (np.arange(1000, dtype=np.uint32) << 16 | 0x8000).view(np.float32) + np.float32(0),
    ])
    ours = bf16_round(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)


def test_bf16_nan_stays_nan_and_widening_is_exact():
    a = np.array([np.nan, 1.5, -2.25], dtype=np.float32)
    r = bf16_round(a)
    back = bf16_to_f32(r)
    assert np.isnan(back[0])
    np.testing.assert_array_equal(back[1:], a[1:])


def test_streams_are_deterministic_and_distinct():
    w = WORKLOADS["tiny_256x688"]
    L1, L2 = w.layer(), w.layer()
    for k in L1:
        np.testing.assert_array_equal(L1[k], L2[k])
    assert not np.array_equal(L1["W_gate"], L1["W_up"])
    assert not np.array_equal(w.layer(copy=1)["W_up"], L1["W_up"])
    np.testing.assert_array_equal(w.tokens(4), w.tokens(4))
    assert not np.array_equal(w.tokens(4, purpose=T_CALIB), w.tokens(4, purpose=T_EVAL))


def test_weight_distribution_and_layout():
    w = WORKLOADS["tiny_256x688"]
    L = w.layer()
    for name in ("W_gate", "W_up", "W_down"):
        assert L[name].shape == (688, 256) and L[name].dtype == np.uint16
        v = bf16_to_f32(L[name]).astype(np.float64)
        assert abs(v.mean()) < 1e-3
        assert abs(v.std() - 0.02) < 5e-4


def test_outlier_channels_recipe():
    w = WORKLOADS["llama7b_4096x11008"]
    ch = outlier_channels(w.wid, w.d_model, w.outlier_frac)
    assert len(ch) == 41 and len(set(ch.tolist())) == 41
    x = bf16_to_f32(make_tokens(w.wid, 64, w.d_model, outlier_frac=w.outlier_frac))
    mask = np.zeros(w.d_model, bool)
    mask[ch] = True
    assert 15 < x[:, mask].std() < 25
    assert 0.9 < x[:, ~mask].std() < 1.1
