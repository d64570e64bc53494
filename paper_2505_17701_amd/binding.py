"""Thin ctypes binding of ``libcountdown.so`` (declared in ``include/countdown.h``).

The functions carry the C names and only marshal arguments: torch tensors
become device pointers, ``stream`` defaults to torch's current HIP stream,
and a non-OK status raises :class:`CountdownError`. All compute runs in the
library's HIP kernels; there is no fallback when the library or the GPU is
missing.
"""
from __future__ import annotations

import ctypes as C
import os

PKG = os.path.dirname(os.path.abspath(__file__))
# CD_LIBRARY names another build of the library to load (the sanitizer test of
# the host code loads an instrumented build this way)
LIB_PATH = os.environ.get("CD_LIBRARY") or os.path.join(PKG, "libcountdown.so")

CD_OK, CD_EINVAL, CD_EUNSUPPORTED, CD_EHIP, CD_ENOMEM = 0, -1, -2, -3, -4
CD_VARIANT_MONO, CD_VARIANT_DUAL_IDEAL, CD_VARIANT_DUAL_PRED, CD_VARIANT_DENSE = 0, 1, 2, 3
CD_VARIANT_CATS, CD_VARIANT_DUAL_TERN = 4, 5
CD_PLAN_KEEP_COEF, CD_PLAN_DETERMINISTIC = 1, 2
CD_PHASE_COEF, CD_PHASE_DOWN, CD_PHASE_ALL = 1, 2, 3

# every symbol include/countdown.h declares
EXPORTS = (
    "countdown_plan_create", "countdown_plan_destroy", "countdown_ffn_mono", "countdown_ffn_dual",
    "countdown_ffn_mono_noalloc",
    "countdown_ffn_dense", "countdown_ffn_cats", "countdown_ffn_topk", "countdown_ffn_residual",
    "countdown_calibrate", "countdown_ffn_tern", "countdown_ffn_tern_topk",
    "countdown_calibrate_tern", "countdown_ternary_words", "countdown_ternary_pack",
    "countdown_export_active",
    "countdown_plan_set_phases", "countdown_stream_read", "countdown_check_args",
    "countdown_check_shape", "countdown_status_string", "countdown_abi_version",
)

_lib = None


class CountdownError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)}")
        self.status = status


def load_library(path: str = LIB_PATH):
    """Load the built library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(python -m paper_2505_17701_amd.build)")
    lib = C.CDLL(path)
    vp, i, u, f, d = C.c_void_p, C.c_int, C.c_uint, C.c_float, C.c_double
    sig = {
        "countdown_plan_create": (i, [i, i, i, i, u, C.POINTER(vp)]),
        "countdown_plan_destroy": (i, [vp]),
        "countdown_ffn_mono": (i, [vp, vp, i, vp, vp, vp, f, vp, vp]),
        "countdown_ffn_dual": (i, [vp, vp, i, vp, vp, vp, vp, vp, f, vp, vp]),
        "countdown_ffn_mono_noalloc": (i, [vp, i, vp, vp, vp, i, i, f, vp, vp]),
        "countdown_ffn_dense": (i, [vp, vp, i, vp, vp, vp, vp, vp]),
        "countdown_ffn_cats": (i, [vp, vp, i, vp, vp, vp, f, vp, vp]),
        "countdown_ffn_residual": (i, [vp, i, vp, vp, vp, f, vp, i, vp, vp, vp, vp, vp, f, vp,
                                       vp]),
        "countdown_ffn_topk": (i, [vp, i, vp, i, vp, vp, vp, vp, vp, d, vp, vp, vp]),
        "countdown_calibrate": (i, [vp, i, vp, i, vp, vp, vp, vp, d, vp, vp, vp]),
        "countdown_ffn_tern": (i, [vp, vp, i, vp, vp, vp, vp, f, vp, vp]),
        "countdown_ffn_tern_topk": (i, [vp, vp, i, vp, vp, vp, vp, d, vp, vp, vp]),
        "countdown_calibrate_tern": (i, [vp, vp, i, vp, d, vp, vp, vp]),
        "countdown_ternary_words": (C.c_size_t, [i, i]),
        "countdown_ternary_pack": (i, [vp, i, i, vp]),
        "countdown_export_active": (i, [vp, vp, vp, vp, vp, vp]),
        "countdown_plan_set_phases": (i, [vp, u]),
        "countdown_stream_read": (i, [vp, C.c_size_t, vp, vp]),
        "countdown_check_args": (i, [i, i, i, i, i, vp, i, vp, vp, vp, vp, vp, f, vp]),
        "countdown_check_shape": (i, [i, i, i, i]),
        "countdown_status_string": (C.c_char_p, [i]),
        "countdown_abi_version": (i, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().countdown_status_string(int(status)).decode()


def _check(status: int, what: str) -> None:
    if status != CD_OK:
        raise CountdownError(status, what)


def _ptr(t) -> int | None:
    """Device pointer of a torch tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("countdown tensors must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("countdown tensors must be contiguous")
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        import torch

        return torch.cuda.current_stream().cuda_stream
    return int(stream) if not hasattr(stream, "cuda_stream") else stream.cuda_stream


def _bf16(t):
    import torch

    if t is not None and t.dtype != torch.bfloat16:
        raise TypeError(f"expected a bfloat16 tensor, got {t.dtype}")
    return t


def _f32(t):
    import torch

    if t.dtype != torch.float32:
        raise TypeError(f"expected a float32 tensor, got {t.dtype}")
    return t


class Plan:
    """Owns a ``cd_plan``: shape, workspace, and optional timing/coefficient capture."""

    def __init__(self, d_model: int, d_ff: int, max_batch: int = 1, d_rank: int = 0,
                 keep_coef: bool = False, deterministic: bool = False):
        self.d_model, self.d_ff, self.max_batch, self.d_rank = d_model, d_ff, max_batch, d_rank
        flags = (CD_PLAN_KEEP_COEF if keep_coef else 0) | (
            CD_PLAN_DETERMINISTIC if deterministic else 0)
        h = C.c_void_p()
        _check(load_library().countdown_plan_create(d_model, d_ff, max_batch, d_rank, flags,
                                                    C.byref(h)), "countdown_plan_create")
        self.handle = h.value
        self.keep_coef = keep_coef
        self.last_batch = 0

    def close(self):
        if getattr(self, "handle", None):
            _check(load_library().countdown_plan_destroy(self.handle), "countdown_plan_destroy")
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def countdown_plan_create(d_model, d_ff, max_batch=1, d_rank=0, keep_coef=False,
                          deterministic=False):
    return Plan(d_model, d_ff, max_batch, d_rank, keep_coef, deterministic)


def countdown_plan_destroy(plan: Plan) -> None:
    plan.close()


def _shape(t, shape, name):
    """ValueError unless ``t`` (None is skipped) has exactly ``shape``."""
    if t is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _layer_shapes(plan, x, W_gate=None, W_up=None, W_down=None, A_t=None, B_t=None,
                  theta_packed=None):
    """Check a call's tensors against the plan before any pointer is taken: the C ABI
    sees only pointers, and the kernels read exactly these extents."""
    if x.dim() != 2 or x.shape[1] != plan.d_model:
        raise ValueError(f"x must be [B, {plan.d_model}], got {tuple(x.shape)}")
    for t, name in ((W_gate, "W_gate"), (W_up, "W_up"), (W_down, "W_down")):
        _shape(t, (plan.d_ff, plan.d_model), name)
    _shape(A_t, (plan.d_rank, plan.d_model), "A_t")
    _shape(B_t, (plan.d_ff, plan.d_rank), "B_t")
    if theta_packed is not None:
        words = countdown_ternary_words(plan.d_model, plan.d_ff)
        if theta_packed.numel() * theta_packed.element_size() != 4 * words:
            raise ValueError(f"theta_packed must hold {words} 32-bit words "
                             f"(countdown_ternary_words), got {theta_packed.numel()} elements")


def _out(plan: Plan, x, y):
    import torch

    B = x.shape[0]
    if y is None:
        y = torch.empty((B, plan.d_model), dtype=torch.float32, device=x.device)
    _shape(y, (B, plan.d_model), "y")
    return B, _f32(y)


def countdown_ffn_mono(plan: Plan, x, W_gate, W_up, W_down, thld: float, y=None, stream=None):
    """M-CountDown FFN; returns y ``[B, d_model]`` fp32 (enqueued on ``stream``)."""
    _layer_shapes(plan, x, W_gate, W_up, W_down)
    B, y = _out(plan, x, y)
    _check(load_library().countdown_ffn_mono(
        plan.handle, _ptr(_bf16(x)), B, _ptr(_bf16(W_gate)), _ptr(_bf16(W_up)),
        _ptr(_bf16(W_down)), float(thld), _ptr(y), _stream(stream)), "countdown_ffn_mono")
    plan.last_batch = B
    return y


def countdown_ffn_mono_noalloc(x, W_gate, W_up, W_down, thld: float, y, stream=None):
    """M-CountDown without a plan (the library's static workspace); y [B, d_model] fp32
    must be given (nothing is allocated). Returns y."""
    for t, name in ((x, "x"), (W_gate, "W_gate"), (W_up, "W_up"), (W_down, "W_down")):
        if t is None or t.dim() != 2:
            raise ValueError(f"{name} must be a 2-D tensor")
    if y is None:
        raise ValueError("y must be given: countdown_ffn_mono_noalloc allocates nothing")
    B, dm = x.shape
    dff = W_up.shape[0]
    for t, name in ((W_gate, "W_gate"), (W_up, "W_up"), (W_down, "W_down")):
        _shape(t, (dff, dm), name)
    _shape(_f32(y), (B, dm), "y")
    _check(load_library().countdown_ffn_mono_noalloc(
        _ptr(_bf16(x)), B, _ptr(_bf16(W_gate)), _ptr(_bf16(W_up)), _ptr(_bf16(W_down)), dm, dff,
        float(thld), _ptr(y), _stream(stream)), "countdown_ffn_mono_noalloc")
    return y


def countdown_ffn_dual(plan: Plan, x, W_gate, W_up, W_down, thld: float, A_t=None, B_t=None,
                       y=None, stream=None):
    """D-CountDown FFN (ideal without a predictor, practical with ``A_t``/``B_t``)."""
    _layer_shapes(plan, x, W_gate, W_up, W_down, A_t, B_t)
    B, y = _out(plan, x, y)
    _check(load_library().countdown_ffn_dual(
        plan.handle, _ptr(_bf16(x)), B, _ptr(_bf16(W_gate)), _ptr(_bf16(W_up)),
        _ptr(_bf16(W_down)), _ptr(_bf16(A_t)), _ptr(_bf16(B_t)), float(thld), _ptr(y),
        _stream(stream)), "countdown_ffn_dual")
    plan.last_batch = B
    return y


def countdown_ffn_cats(plan: Plan, x, W_gate, W_up, W_down, thld: float, y=None, stream=None):
    """CATS (Eq. 6a): keep |SiLU(x.W_gate)| > thld, gather W_up on the kept neurons."""
    _layer_shapes(plan, x, W_gate, W_up, W_down)
    B, y = _out(plan, x, y)
    _check(load_library().countdown_ffn_cats(
        plan.handle, _ptr(_bf16(x)), B, _ptr(_bf16(W_gate)), _ptr(_bf16(W_up)),
        _ptr(_bf16(W_down)), float(thld), _ptr(y), _stream(stream)), "countdown_ffn_cats")
    plan.last_batch = B
    return y


def countdown_ffn_topk(plan: Plan, variant: int, x, W_gate, W_up, W_down, k: float, A_t=None,
                       B_t=None, y=None, thld_out=None, stream=None):
    """Per-token threshold: each token keeps the neurons above the k-quantile of its
    own coefficients (union over the batch). ``thld_out``: optional fp64 [B] device
    tensor for the thresholds. Returns y."""
    import torch

    _layer_shapes(plan, x, W_gate, W_up, W_down, A_t, B_t)
    B, y = _out(plan, x, y)
    if thld_out is not None and (thld_out.dtype != torch.float64 or thld_out.numel() < B):
        raise ValueError("thld_out must be a float64 device tensor with at least B entries")
    _check(load_library().countdown_ffn_topk(
        plan.handle, int(variant), _ptr(_bf16(x)), B, _ptr(_bf16(W_gate)), _ptr(_bf16(W_up)),
        _ptr(_bf16(W_down)), _ptr(_bf16(A_t)), _ptr(_bf16(B_t)), float(k), _ptr(thld_out),
        _ptr(y), _stream(stream)), "countdown_ffn_topk")
    plan.last_batch = B
    return y


def countdown_ffn_residual(plan: Plan, variant: int, h_in, y_prev, h_out, x_out, W_gate, W_up,
                           W_down, thld: float = 0.0, A_t=None, B_t=None, eps: float = 1e-5,
                           y=None, stream=None):
    """One layer of a residual stack: h_out = h_in + y_prev, x_out = bf16(RMSNorm(h_out)),
    then the ``variant`` FFN of x_out into ``y`` (returned). ``y_prev`` may be None or ``y``."""
    import torch

    B = h_in.shape[0]
    if y is None:
        y = torch.empty((B, plan.d_model), dtype=torch.float32, device=h_in.device)
    for t in (h_in, h_out, y) + (() if y_prev is None else (y_prev,)):
        if t.dtype != torch.float32 or not t.is_contiguous() or tuple(t.shape) != (B, plan.d_model):
            raise ValueError("h_in, y_prev, h_out and y must be contiguous fp32 [B, d_model]")
    if tuple(x_out.shape) != (B, plan.d_model) or not x_out.is_contiguous():
        raise ValueError("x_out must be a contiguous [B, d_model] bf16 tensor")
    _layer_shapes(plan, x_out, W_gate, W_up, W_down, A_t, B_t)
    _check(load_library().countdown_ffn_residual(
        plan.handle, int(variant), _ptr(h_in), _ptr(y_prev), _ptr(h_out), float(eps),
        _ptr(_bf16(x_out)), B, _ptr(_bf16(W_gate)), _ptr(_bf16(W_up)), _ptr(_bf16(W_down)),
        _ptr(_bf16(A_t)), _ptr(_bf16(B_t)), float(thld), _ptr(y), _stream(stream)),
        "countdown_ffn_residual")
    plan.last_batch = B
    return y


def countdown_ffn_dense(plan: Plan, x, W_gate, W_up, W_down, y=None, stream=None):
    """Dense Gated-MLP through the same kernels."""
    _layer_shapes(plan, x, W_gate, W_up, W_down)
    B, y = _out(plan, x, y)
    _check(load_library().countdown_ffn_dense(
        plan.handle, _ptr(_bf16(x)), B, _ptr(_bf16(W_gate)), _ptr(_bf16(W_up)),
        _ptr(_bf16(W_down)), _ptr(y), _stream(stream)), "countdown_ffn_dense")
    plan.last_batch = B
    return y


def countdown_calibrate(plan: Plan, variant: int, X, k: float, W_gate=None, W_up=None, A_t=None,
                        B_t=None, stream=None):
    """Layerwise threshold; returns ``(thld fp32 tensor [1], per-token quantiles fp64 [T])``."""
    import torch

    _layer_shapes(plan, X, W_gate, W_up, None, A_t, B_t)
    T = X.shape[0]
    thld = torch.empty(1, dtype=torch.float32, device=X.device)
    q = torch.empty(T, dtype=torch.float64, device=X.device)
    _check(load_library().countdown_calibrate(
        plan.handle, int(variant), _ptr(_bf16(X)), T, _ptr(_bf16(W_gate)), _ptr(_bf16(W_up)),
        _ptr(_bf16(A_t)), _ptr(_bf16(B_t)), float(k), _ptr(thld), _ptr(q), _stream(stream)),
        "countdown_calibrate")
    return thld, q


def _u32(t):
    import torch

    if t.dtype not in (torch.int32, torch.uint32):
        raise TypeError(f"expected a packed 32-bit tensor, got {t.dtype}")
    return t


def countdown_ternary_words(d_model: int, d_ff: int) -> int:
    """uint32 words of the packed ternary predictor of a shape (0 if rejected)."""
    return int(load_library().countdown_ternary_words(int(d_model), int(d_ff)))


def countdown_ternary_pack(theta_t):
    """Pack a host int8 ``theta_t [d_ff, d_model]`` (entries -1, 0, +1; theta transposed)
    into the kernels' layout; returns a host numpy uint32 array (move it to the GPU)."""
    import numpy as np

    t = np.ascontiguousarray(theta_t, dtype=np.int8)
    d_ff, d_model = t.shape
    n = countdown_ternary_words(d_model, d_ff)
    if n == 0:
        raise CountdownError(CD_EINVAL, "countdown_ternary_words")
    out = np.zeros(n, dtype=np.uint32)
    _check(load_library().countdown_ternary_pack(t.ctypes.data, d_model, d_ff, out.ctypes.data),
           "countdown_ternary_pack")
    return out


def countdown_ffn_tern(plan: Plan, x, W_gate, W_up, W_down, theta_packed, thld: float, y=None,
                       stream=None):
    """D-CountDown with the ternary predictor (``theta_packed``: device int32/uint32 tensor
    from :func:`countdown_ternary_pack`)."""
    _layer_shapes(plan, x, W_gate, W_up, W_down, theta_packed=theta_packed)
    B, y = _out(plan, x, y)
    _check(load_library().countdown_ffn_tern(
        plan.handle, _ptr(_bf16(x)), B, _ptr(_bf16(W_gate)), _ptr(_bf16(W_up)),
        _ptr(_bf16(W_down)), _ptr(_u32(theta_packed)), float(thld), _ptr(y), _stream(stream)),
        "countdown_ffn_tern")
    plan.last_batch = B
    return y


def countdown_ffn_tern_topk(plan: Plan, x, W_gate, W_up, W_down, theta_packed, k: float, y=None,
                            thld_out=None, stream=None):
    """Per-token threshold on the ternary predictor score; returns y."""
    import torch

    _layer_shapes(plan, x, W_gate, W_up, W_down, theta_packed=theta_packed)
    B, y = _out(plan, x, y)
    if thld_out is not None and (thld_out.dtype != torch.float64 or thld_out.numel() < B):
        raise ValueError("thld_out must be a float64 device tensor with at least B entries")
    _check(load_library().countdown_ffn_tern_topk(
        plan.handle, _ptr(_bf16(x)), B, _ptr(_bf16(W_gate)), _ptr(_bf16(W_up)),
        _ptr(_bf16(W_down)), _ptr(_u32(theta_packed)), float(k), _ptr(thld_out), _ptr(y),
        _stream(stream)), "countdown_ffn_tern_topk")
    plan.last_batch = B
    return y


def countdown_calibrate_tern(plan: Plan, X, theta_packed, k: float, stream=None):
    """Layerwise threshold of the ternary predictor score; returns ``(thld [1], q [T])``."""
    import torch

    _layer_shapes(plan, X, theta_packed=theta_packed)
    T = X.shape[0]
    thld = torch.empty(1, dtype=torch.float32, device=X.device)
    q = torch.empty(T, dtype=torch.float64, device=X.device)
    _check(load_library().countdown_calibrate_tern(
        plan.handle, _ptr(_bf16(X)), T, _ptr(_u32(theta_packed)), float(k), _ptr(thld), _ptr(q),
        _stream(stream)), "countdown_calibrate_tern")
    return thld, q


def countdown_export_active(plan: Plan, stream=None):
    """The last call's ``(IDX [n] int32, s_c [B, n] fp32, coef [B, d_ff] or None)`` as new
    device tensors. Synchronises the stream to read ``n``."""
    import torch

    dev = torch.device("cuda", torch.cuda.current_device())
    B = max(plan.last_batch, 1)
    idx = torch.empty(plan.d_ff, dtype=torch.int32, device=dev)
    n = torch.empty(1, dtype=torch.int32, device=dev)
    s = torch.empty((B, plan.d_ff), dtype=torch.float32, device=dev)
    coef = torch.empty((B, plan.d_ff), dtype=torch.float32, device=dev) if plan.keep_coef else None
    _check(load_library().countdown_export_active(plan.handle, _ptr(idx), _ptr(n), _ptr(s),
                                                  _ptr(coef), _stream(stream)),
           "countdown_export_active")
    m = int(n.item())  # .item() synchronises with the copy's stream
    return idx[:m], s[:, :m], coef


def countdown_plan_set_phases(plan: Plan, phases: int) -> None:
    """Launch only the kernels in ``phases`` (CD_PHASE_*) on later calls (measurement aid)."""
    _check(load_library().countdown_plan_set_phases(plan.handle, int(phases)),
           "countdown_plan_set_phases")


def countdown_stream_read(src, sink, stream=None) -> None:
    """Measurement aid: a plain streaming read of the whole of ``src`` (a contiguous
    device tensor) with the coefficient kernel's load pattern; ``sink`` is a one-word
    int32 / uint32 device tensor. Enqueued on ``stream``."""
    if sink.numel() * sink.element_size() < 4:
        raise ValueError("sink must hold at least one 32-bit word")
    _check(load_library().countdown_stream_read(
        _ptr(src), src.numel() * src.element_size(), _ptr(sink), _stream(stream)),
        "countdown_stream_read")


def countdown_check_args(variant, d_model, d_ff, max_batch, d_rank, x, B, W_gate, W_up, W_down,
                         A_t, B_t, thld, y) -> int:
    """Host-only argument validation (integer pointers); returns the status code."""
    return load_library().countdown_check_args(variant, d_model, d_ff, max_batch, d_rank, x, B,
                                               W_gate, W_up, W_down, A_t, B_t, float(thld), y)


def countdown_check_shape(d_model, d_ff, max_batch, d_rank) -> int:
    return load_library().countdown_check_shape(d_model, d_ff, max_batch, d_rank)


def max_batch_for(d_model: int, d_ff: int = 8, d_rank: int = 0) -> int:
    """Largest max_batch countdown_check_shape accepts for this shape (0 if none)."""
    for b in range(8, 0, -1):
        if countdown_check_shape(d_model, d_ff, b, d_rank) == CD_OK:
            return b
    return 0


def countdown_abi_version() -> int:
    return load_library().countdown_abi_version()
