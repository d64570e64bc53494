"""Shared helpers of the GPU parity tests: upload, oracle comparison rules."""
import numpy as np

IDX_BAND = 1e-5       # relative band around thld inside which a membership flip is excused
Y_TOL = 2e-3          # max |y_gpu - y_oracle| <= Y_TOL * max |y_oracle|  (bf16 weights, fp32 sums)
S_TOL = 1e-5          # compact coefficients s: |ds| <= S_TOL * max |s_oracle|
COEF_TOL = 1e-5       # dense coefficient: |dc_i| <= COEF_TOL * sum_j |x_j w_ij| (fp32 dot bound)


def dev_bf16(a):
    """uint16 bf16 bit patterns (numpy) -> torch.bfloat16 on cuda:0."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    return t.to("cuda")


def coef_max(variant, c):
    """Per-neuron union coefficient: max over the batch of |c| (signed for the predictor)."""
    c = np.atleast_2d(c)
    return (c if variant in ("dual_pred", "dual_tern") else np.abs(c)).max(axis=0)


def check_idx(idx_gpu, idx_ref, cmax, thld, label=""):
    """IDX must equal the oracle's except for neurons whose coefficient lies within
    IDX_BAND (relative) of thld; it must be ascending and duplicate-free."""
    idx_gpu = np.asarray(idx_gpu, dtype=np.int64)
    assert np.all(np.diff(idx_gpu) > 0), f"{label}: IDX not strictly ascending"
    diff = np.setxor1d(idx_gpu, np.asarray(idx_ref, dtype=np.int64))
    if len(diff):
        band = IDX_BAND * max(abs(float(thld)), float(np.sqrt(np.mean(cmax ** 2))))
        gap = np.abs(cmax[diff] - float(thld))
        assert np.all(gap <= band), (f"{label}: {len(diff)} IDX flips, worst |c - thld| = "
                                     f"{gap.max():.3e} > band {band:.3e}")
    return len(diff)


def check_y(y_gpu, y_ref, label=""):
    y_gpu = np.asarray(y_gpu, dtype=np.float64)
    scale = float(np.abs(y_ref).max())
    if scale == 0.0:
        assert np.all(y_gpu == 0.0), f"{label}: expected y = 0"
        return 0.0
    err = float(np.abs(y_gpu - y_ref).max())
    assert err <= Y_TOL * scale, f"{label}: max|dy| = {err:.3e} > {Y_TOL} * {scale:.3e}"
    return err / scale


def check_s(s_gpu, s_ref, label=""):
    s_ref = np.atleast_2d(s_ref)
    if s_ref.size == 0:
        return 0.0
    scale = float(np.abs(s_ref).max()) or 1.0
    err = float(np.abs(np.asarray(s_gpu, np.float64) - s_ref).max())
    assert err <= S_TOL * scale, f"{label}: max|ds| = {err:.3e} > {S_TOL} * {scale:.3e}"
    return err / scale


def dot_bound(x_f64, W_f64):
    """sum_j |x_j| |w_ij| per token and neuron: the scale of an fp32 dot-product error."""
    return np.abs(np.atleast_2d(x_f64)) @ np.abs(W_f64).T
