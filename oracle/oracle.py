"""ctypes front end of the fp64 C oracle (``cd_oracle.c``).

TEST INFRASTRUCTURE ONLY (see the package docstring). Arrays of bf16 values
are passed as ``uint16`` bit patterns, neuron-major ``[d_ff, d_model]``;
results come back as float64 numpy arrays. Each function names the passage
of arXiv 2505.17701 it follows; the arithmetic itself is in the C file.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "cd_oracle.c")
# CD_ORACLE_LIB names another build of the oracle to load (the mutation test of
# the pins loads deliberately broken copies this way); build() leaves it alone
LIB = os.environ.get("CD_ORACLE_LIB") or os.path.join(HERE, "libcdoracle.so")

COEF_ABS_U, COEF_ABS_S, COEF_SHAT, COEF_ABS_H, COEF_TERN = 0, 1, 2, 3, 4
KIND = {"mono": COEF_ABS_U, "dual_ideal": COEF_ABS_S, "dual_pred": COEF_SHAT, "cats": COEF_ABS_H,
        "dual_tern": COEF_TERN}

_lib = None

__all__ = [
    "build", "load", "num_threads", "set_num_threads", "silu", "coefficients", "predictor", "select", "combine",
    "dense", "ffn_on_idx", "ffn_mono", "ffn_dual_ideal", "ffn_dual_pred", "quantile_linear",
    "calibrate", "ffn_topk", "ffn_cats", "residual_rmsnorm", "ternary_predictor",
    "ffn_dual_tern", "KIND",
]


def build(force: bool = True) -> str:
    """Compile ``cd_oracle.c`` with gcc (fp64, no fast-math, OpenMP over rows)."""
    if os.environ.get("CD_ORACLE_LIB"):
        return LIB
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-Wextra",
               "-o", tmp, SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB)
    return LIB


def load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        lib = C.CDLL(LIB)
        u16p = np.ctypeslib.ndpointer(np.uint16, flags="C_CONTIGUOUS")
        f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
        i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")
        i8p = np.ctypeslib.ndpointer(np.int8, flags="C_CONTIGUOUS")
        vp = C.c_void_p
        lib.cdo_num_threads.restype = C.c_int
        lib.cdo_set_num_threads.restype = None
        lib.cdo_set_num_threads.argtypes = [C.c_int]
        lib.cdo_silu.restype = C.c_double
        lib.cdo_silu.argtypes = [C.c_double]
        lib.cdo_coefficients.restype = C.c_int
        lib.cdo_coefficients.argtypes = [u16p, C.c_int, u16p, u16p, C.c_int, C.c_int, vp, vp, vp]
        lib.cdo_predictor.restype = C.c_int
        lib.cdo_predictor.argtypes = [u16p, C.c_int, u16p, u16p, C.c_int, C.c_int, C.c_int, vp,
                                      f64p]
        lib.cdo_select.restype = C.c_int64
        lib.cdo_select.argtypes = [f64p, C.c_int, C.c_int64, C.c_int, C.c_double, i32p]
        lib.cdo_combine.restype = C.c_int
        lib.cdo_combine.argtypes = [f64p, C.c_int, C.c_int64, u16p, C.c_int, vp, C.c_int64, f64p]
        lib.cdo_dense.restype = C.c_int
        lib.cdo_dense.argtypes = [u16p, C.c_int, u16p, u16p, u16p, C.c_int, C.c_int, f64p]
        lib.cdo_ffn_on_idx.restype = C.c_int
        lib.cdo_ffn_on_idx.argtypes = [u16p, C.c_int, u16p, u16p, u16p, C.c_int, C.c_int, vp,
                                       C.c_int64, f64p, vp]
        for name in ("cdo_ffn_mono", "cdo_ffn_dual_ideal", "cdo_ffn_cats"):
            f = getattr(lib, name)
            f.restype = C.c_int64
            f.argtypes = [u16p, C.c_int, u16p, u16p, u16p, C.c_int, C.c_int, C.c_double, i32p,
                          f64p, vp]
        lib.cdo_ffn_dual_pred.restype = C.c_int64
        lib.cdo_ffn_dual_pred.argtypes = [u16p, C.c_int, u16p, u16p, u16p, u16p, u16p, C.c_int,
                                          C.c_int, C.c_int, C.c_double, i32p, f64p, vp]
        lib.cdo_quantile_linear.restype = C.c_double
        lib.cdo_quantile_linear.argtypes = [C.c_double, f64p, C.c_int64]
        lib.cdo_calibrate.restype = C.c_double
        lib.cdo_ternary_predictor.restype = C.c_int
        lib.cdo_ternary_predictor.argtypes = [u16p, C.c_int, i8p, C.c_int, C.c_int, f64p]
        lib.cdo_ffn_dual_tern.restype = C.c_int64
        lib.cdo_ffn_dual_tern.argtypes = [u16p, C.c_int, u16p, u16p, u16p, i8p, C.c_int, C.c_int,
                                          C.c_double, i32p, f64p, vp]
        lib.cdo_calibrate.argtypes = [C.c_int, u16p, C.c_int, vp, vp, vp, vp, C.c_int, C.c_int,
                                      C.c_int, C.c_double, vp, vp]
        lib.cdo_ffn_topk.restype = C.c_int64
        lib.cdo_ffn_topk.argtypes = [C.c_int, u16p, C.c_int, u16p, u16p, u16p, vp, vp, C.c_int,
                                     C.c_int, C.c_int, C.c_double, i32p, f64p, f64p, vp]
        lib.cdo_residual_rmsnorm.restype = C.c_int
        lib.cdo_residual_rmsnorm.argtypes = [f64p, vp, C.c_int, C.c_double, f64p]
        _lib = lib
    return _lib


def _u16(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError(f"expected bf16 bit patterns (uint16), got {a.dtype}")
    return a


def _tok(x) -> np.ndarray:
    x = _u16(x)
    return x[None, :] if x.ndim == 1 else x


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _check(rc, what):
    if rc < 0:
        raise ValueError(f"oracle {what} failed with code {rc}")
    return rc


def num_threads() -> int:
    return load().cdo_num_threads()


def set_num_threads(n: int) -> None:
    """OpenMP threads of the following oracle calls (timing only)."""
    load().cdo_set_num_threads(int(n))


def silu(z: float) -> float:
    """SiLU(z) = z * sigmoid(z) (Sec. 3, sigma = SiLU)."""
    return load().cdo_silu(float(z))


def coefficients(x, W_gate, W_up):
    """Sec. 3: ``u = x.W_up``, ``g = x.W_gate``, ``s = u * SiLU(g)``; each ``[B, d_ff]``."""
    x = _tok(x)
    B, dm = x.shape
    dff = W_up.shape[0]
    u, g, s = (np.empty((B, dff)) for _ in range(3))
    _check(load().cdo_coefficients(x, B, _u16(W_gate), _u16(W_up), dm, dff, _ptr(u), _ptr(g),
                                   _ptr(s)), "coefficients")
    return u, g, s


def predictor(x, A_t, B_t):
    """Sec. 4 low-rank predictor: ``latent = x.theta_A``, ``shat = latent.theta_B``."""
    x = _tok(x)
    B, dm = x.shape
    dr, dff = A_t.shape[0], B_t.shape[0]
    lat, sh = np.empty((B, dr)), np.empty((B, dff))
    _check(load().cdo_predictor(x, B, _u16(A_t), _u16(B_t), dm, dr, dff, _ptr(lat), sh),
           "predictor")
    return lat, sh


def select(c, thld: float, use_abs: bool = True) -> np.ndarray:
    """Eq. (6) with a constant threshold (strict ``>``), union over the batch rows of ``c``."""
    c = np.ascontiguousarray(np.atleast_2d(c), dtype=np.float64)
    B, dff = c.shape
    idx = np.empty(dff, dtype=np.int32)
    n = _check(load().cdo_select(c, B, dff, int(bool(use_abs)), float(thld), idx), "select")
    return idx[:n].copy()


def combine(s, W_down, idx) -> np.ndarray:
    """Eq. (5) over ``idx``: ``y_b = sum_t s_b[idx[t]] W_down^T[idx[t]]``."""
    s = np.ascontiguousarray(np.atleast_2d(s), dtype=np.float64)
    B, dff = s.shape
    dm = W_down.shape[1]
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    y = np.empty((B, dm))
    _check(load().cdo_combine(s, B, dff, _u16(W_down), dm, _ptr(idx), len(idx), y), "combine")
    return y


def dense(x, W_gate, W_up, W_down) -> np.ndarray:
    """Eq. (1): the dense Gated-MLP output ``[B, d_model]``."""
    x = _tok(x)
    B, dm = x.shape
    y = np.empty((B, dm))
    _check(load().cdo_dense(x, B, _u16(W_gate), _u16(W_up), _u16(W_down), dm, W_up.shape[0], y),
           "dense")
    return y


def ffn_on_idx(x, W_gate, W_up, W_down, idx):
    """Eq. (2)-(3) and (5) on a given index set. Returns ``(y, s_c)`` with ``s_c [B, n]``."""
    x = _tok(x)
    B, dm = x.shape
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    y, sc = np.empty((B, dm)), np.empty((B, len(idx)))
    _check(load().cdo_ffn_on_idx(x, B, _u16(W_gate), _u16(W_up), _u16(W_down), dm,
                                 W_up.shape[0], _ptr(idx), len(idx), y, _ptr(sc)), "ffn_on_idx")
    return y, sc


def _variant(fn, x, W_gate, W_up, W_down, thld, want_coef):
    x = _tok(x)
    B, dm = x.shape
    dff = W_up.shape[0]
    idx = np.empty(dff, dtype=np.int32)
    y = np.empty((B, dm))
    coef = np.empty((B, dff)) if want_coef else None
    n = _check(fn(x, B, _u16(W_gate), _u16(W_up), _u16(W_down), dm, dff, float(thld), idx, y,
                  _ptr(coef)), fn.__name__)
    return idx[:n].copy(), y, coef


def ffn_mono(x, W_gate, W_up, W_down, thld, want_coef=False):
    """M-CountDown (Eq. 6b): returns ``(IDX, y, u or None)``."""
    return _variant(load().cdo_ffn_mono, x, W_gate, W_up, W_down, thld, want_coef)


def ffn_cats(x, W_gate, W_up, W_down, thld, want_coef=False):
    """CATS (Eq. 6a, the comparison method): returns ``(IDX, y, h or None)``."""
    return _variant(load().cdo_ffn_cats, x, W_gate, W_up, W_down, thld, want_coef)


def ffn_dual_ideal(x, W_gate, W_up, W_down, thld, want_coef=False):
    """D-CountDown ideal (Eq. 6c): returns ``(IDX, y, s or None)``."""
    return _variant(load().cdo_ffn_dual_ideal, x, W_gate, W_up, W_down, thld, want_coef)


def ffn_dual_pred(x, W_gate, W_up, W_down, A_t, B_t, thld, want_coef=False):
    """D-CountDown with the low-rank predictor (Sec. 4): returns ``(IDX, y, shat or None)``."""
    x = _tok(x)
    B, dm = x.shape
    dff, dr = B_t.shape
    idx = np.empty(dff, dtype=np.int32)
    y = np.empty((B, dm))
    coef = np.empty((B, dff)) if want_coef else None
    n = _check(load().cdo_ffn_dual_pred(x, B, _u16(W_gate), _u16(W_up), _u16(W_down), _u16(A_t),
                                        _u16(B_t), dm, dr, dff, float(thld), idx, y, _ptr(coef)),
               "ffn_dual_pred")
    return idx[:n].copy(), y, coef


def _tern(theta_t) -> np.ndarray:
    t = np.ascontiguousarray(theta_t)
    if t.dtype != np.int8:
        raise TypeError("theta_t must be int8 (-1, 0, +1)")
    return t


def ternary_predictor(x, theta_t):
    """The TernaryLinear score of Sec. 6: ``s_hat = x . theta`` (``theta_t`` = theta
    transposed, int8 ``[d_ff, d_model]``); returns ``[B, d_ff]`` float64."""
    x = _tok(x)
    t = _tern(theta_t)
    B, dm = x.shape
    out = np.empty((B, t.shape[0]))
    _check(load().cdo_ternary_predictor(x, B, t, dm, t.shape[0], out), "ternary_predictor")
    return out


def ffn_dual_tern(x, W_gate, W_up, W_down, theta_t, thld, want_coef=False):
    """D-CountDown with the ternary predictor (Sec. 6): returns ``(IDX, y, shat or None)``."""
    x = _tok(x)
    t = _tern(theta_t)
    B, dm = x.shape
    dff = t.shape[0]
    idx = np.empty(dff, dtype=np.int32)
    y = np.empty((B, dm))
    coef = np.empty((B, dff)) if want_coef else None
    n = _check(load().cdo_ffn_dual_tern(x, B, _u16(W_gate), _u16(W_up), _u16(W_down), t, dm, dff,
                                        float(thld), idx, y, _ptr(coef)), "ffn_dual_tern")
    return idx[:n].copy(), y, coef


def quantile_linear(k: float, v) -> float:
    """``Quantile(k, v)`` with linear interpolation between order statistics."""
    v = np.ascontiguousarray(np.ravel(v), dtype=np.float64)
    return load().cdo_quantile_linear(float(k), v, len(v))


def calibrate(variant: str, X, k: float, W_gate=None, W_up=None, A_t=None, B_t=None,
              theta_t=None):
    """Sec. 4 calibration: mean over tokens of ``Quantile(k, c^(t))``.

    Returns ``(tau_hat as float64, per-token quantiles)``. ``variant`` is one
    of ``mono`` (|u|), ``dual_ideal`` (|s|), ``dual_pred`` (signed s_hat),
    ``dual_tern`` (signed ternary score, ``theta_t``), ``cats`` (|h|).
    """
    X = _tok(X)
    T, dm = X.shape
    refs = [a for a in (W_up, W_gate, B_t, theta_t) if a is not None]
    dff = refs[0].shape[0]
    dr = A_t.shape[0] if A_t is not None else 0
    q = np.empty(T)
    keep = [None if a is None else _u16(a) for a in (W_gate, W_up, A_t, B_t)]
    tt = None if theta_t is None else _tern(theta_t)
    t = load().cdo_calibrate(KIND[variant], X, T, *(_ptr(a) for a in keep), dm, dr, dff,
                             float(k), _ptr(q), _ptr(tt))
    if np.isnan(t):
        raise ValueError("oracle calibrate failed")
    return t, q


def ffn_topk(variant: str, x, W_gate, W_up, W_down, k: float, A_t=None, B_t=None,
             theta_t=None):
    """Per-token threshold (Eq. 6 with thld_b = Quantile(k, c_b) of each token's own
    coefficients, union over the batch): returns ``(IDX, y, per-token thresholds)``."""
    x = _tok(x)
    B, dm = x.shape
    dff = W_up.shape[0]
    dr = 0 if A_t is None else A_t.shape[0]
    idx = np.empty(dff, dtype=np.int32)
    y = np.empty((B, dm))
    q = np.empty(B)
    tt = None if theta_t is None else _tern(theta_t)
    n = _check(load().cdo_ffn_topk(KIND[variant], x, B, _u16(W_gate), _u16(W_up), _u16(W_down),
                                   _ptr(None if A_t is None else _u16(A_t)),
                                   _ptr(None if B_t is None else _u16(B_t)), dm, dr, dff,
                                   float(k), idx, y, q, _ptr(tt)), "ffn_topk")
    return idx[:n].copy(), y, q


def residual_rmsnorm(h, y, eps: float = 1e-5):
    """Residual add then RMSNorm with unit gain (the layer-stack workload, not in the paper)."""
    h = np.array(h, dtype=np.float64, copy=True)
    r = np.empty_like(h)
    yy = None if y is None else np.ascontiguousarray(y, dtype=np.float64)
    _check(load().cdo_residual_rmsnorm(h, _ptr(yy), len(h), float(eps), r), "residual_rmsnorm")
    return h, r
