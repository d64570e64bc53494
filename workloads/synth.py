"""Seeded synthetic inputs: weights, tokens and predictor matrices.

Layout convention (used by every consumer): each weight matrix is stored
neuron-major, ``[d_ff, d_model]`` row-major, so row ``i`` is the contiguous
``d_model``-long weight vector of intermediate neuron ``i``:

* ``W_gate[i, j]`` and ``W_up[i, j]`` are the paper's ``W_gate[j, i]`` and
  ``W_up[j, i]`` (its matrices are ``d_model x d_inter``, Sec. 3 "Problem
  Formulation"), i.e. the ``nn.Linear`` ``[out, in]`` layout;
* ``W_down[i, :]`` is the paper's ``W_down^T[i]``, the i-th vector of the
  linear combination of Eq. (5);
* the low-rank predictor ``theta_A`` (``d_model x d_rank``) is stored as
  ``A_t [d_rank, d_model]`` and ``theta_B`` (``d_rank x d_inter``) as
  ``B_t [d_ff, d_rank]`` (Sec. 4, "Constructing SP^Prac");
* the ternary predictor ``theta`` (``d_model x d_inter``, entries -1, 0, +1;
  Sec. 6, TernaryLinear) as int8 ``theta_t [d_ff, d_model]``.

bf16 tensors are carried as ``uint16`` bit patterns. Random streams come
from numpy ``PCG64`` seeded by ``SeedSequence(42, spawn_key=...)`` (the
paper's seed 42, Table 5), keyed by ``(workload, layer, tensor, copy)`` so
that every tensor can be regenerated on its own.

Nothing here computes any part of the FFN, a coefficient or a threshold.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

ROOT_SEED = 42

# tensor ids inside a spawn key
T_GATE, T_UP, T_DOWN, T_A, T_B, T_TERN = 0, 1, 2, 3, 4, 5
T_CALIB, T_EVAL, T_OUTLIER, T_RESID = 10, 11, 12, 13
# held-out calibration tokens of a trained predictor (neither its training nor its test set)
T_HELDOUT = 14
T_LOWRANK = 15


def stream(*key: int) -> np.random.Generator:
    """A PCG64 generator for the spawn key ``key`` under the root seed."""
    ss = np.random.SeedSequence(entropy=ROOT_SEED, spawn_key=tuple(int(k) for k in key))
    return np.random.Generator(np.random.PCG64(ss))


def bf16_round(a) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest, ties to even.

    NaN stays NaN (quietened); +-inf and overflow to inf follow IEEE rounding.
    Works in uint32 (no finite pattern overflows: the largest, -inf, is
    0xFF800000) over row chunks so that large matrices need little scratch.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    flat = a.reshape(-1).view(np.uint32)
    out = np.empty(flat.shape, dtype=np.uint16)
    step = 1 << 24
    for lo in range(0, flat.size, step):
        b = flat[lo:lo + step]
        nan = (b & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
        r = b + (np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1)))
        r >>= np.uint32(16)
        o = r.astype(np.uint16)
        if nan.any():
            o[nan] = ((b[nan] >> np.uint32(16)) | np.uint32(0x40)).astype(np.uint16)
        out[lo:lo + step] = o
    return out.reshape(a.shape)


def bf16_to_f32(u16) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact fp32 values."""
    u = np.ascontiguousarray(u16, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32)


def _normal_bf16(rng: np.random.Generator, shape, sigma: float) -> np.ndarray:
    a = rng.standard_normal(size=shape, dtype=np.float32)
    if sigma != 1.0:
        a *= np.float32(sigma)
    return bf16_round(a)


def make_layer(wid: int, d_model: int, d_ff: int, sigma: float, layer: int = 0, copy: int = 0):
    """Gated-MLP weights ``W_gate, W_up, W_down`` as bf16 ``[d_ff, d_model]``.

    Entries are i.i.d. N(0, sigma^2) in fp32, rounded once to bf16.
    """
    return {
        "W_gate": _normal_bf16(stream(wid, layer, T_GATE, copy), (d_ff, d_model), sigma),
        "W_up": _normal_bf16(stream(wid, layer, T_UP, copy), (d_ff, d_model), sigma),
        "W_down": _normal_bf16(stream(wid, layer, T_DOWN, copy), (d_ff, d_model), sigma),
    }


def make_predictor(wid: int, d_model: int, d_rank: int, d_ff: int, sigma: float,
                   layer: int = 0, copy: int = 0):
    """Seeded random low-rank predictor: ``A_t [d_rank, d_model]``, ``B_t [d_ff, d_rank]``."""
    return {
        "A_t": _normal_bf16(stream(wid, layer, T_A, copy), (d_rank, d_model), sigma),
        "B_t": _normal_bf16(stream(wid, layer, T_B, copy), (d_ff, d_rank), sigma),
    }


def make_low_rank(wid: int, rows: int, cols: int, rank: int, sigma: float, layer: int = 0,
                  tensor: int = T_GATE) -> np.ndarray:
    """A seeded ``[rows, cols]`` bf16 matrix of rank at most ``rank`` (before rounding):
    ``P @ Q`` with ``P [rows, rank]`` and ``Q [rank, cols]`` i.i.d. normal, scaled so that
    entries have standard deviation ``sigma``. A layer whose W_gate has low rank gives a
    predictor of matching rank something it can represent."""
    rng = stream(wid, layer, T_LOWRANK, tensor)
    P = rng.standard_normal(size=(rows, rank), dtype=np.float32)
    Q = rng.standard_normal(size=(rank, cols), dtype=np.float32)
    return bf16_round((P @ Q) * np.float32(sigma / np.sqrt(rank)))


def make_ternary(wid: int, d_model: int, d_ff: int, zero_frac: float = 1 / 3, layer: int = 0,
                 copy: int = 0) -> np.ndarray:
    """Seeded random ternary predictor ``theta_t [d_ff, d_model]`` int8: each entry is 0
    with probability ``zero_frac``, else -1 or +1 with equal probability (about what an
    absmean ternarisation of Gaussian weights gives at the default)."""
    rng = stream(wid, layer, T_TERN, copy)
    u = rng.random(size=(d_ff, d_model), dtype=np.float32)
    half = np.float32((1.0 - zero_frac) / 2.0)
    t = np.zeros((d_ff, d_model), dtype=np.int8)
    t[u < half] = -1
    t[u >= np.float32(1.0) - half] = 1
    return t


def outlier_channels(wid: int, d_model: int, frac: float) -> np.ndarray:
    """``round(frac * d_model)`` channel ids, drawn once per workload without replacement."""
    n = int(round(frac * d_model))
    if n == 0:
        return np.zeros(0, dtype=np.int64)
    return np.sort(stream(wid, 0, T_OUTLIER).choice(d_model, size=n, replace=False))


def make_tokens(wid: int, n: int, d_model: int, purpose: int = T_EVAL, layer: int = 0,
                outlier_frac: float = 0.0, outlier_scale: float = 20.0,
                as_fp32: bool = False) -> np.ndarray:
    """``n`` decode tokens ``[n, d_model]`` with x ~ N(0, 1) in fp32.

    With ``outlier_frac > 0`` a fixed set of channels (``outlier_channels``)
    is multiplied by ``outlier_scale`` in every token before rounding. The
    calibration and evaluation tokens use different streams
    (``purpose = T_CALIB`` / ``T_EVAL``). Returns bf16 bit patterns unless
    ``as_fp32`` (the fp32 residual stream of a layer stack).
    """
    x = stream(wid, layer, purpose).standard_normal(size=(n, d_model), dtype=np.float32)
    if outlier_frac > 0:
        x[:, outlier_channels(wid, d_model, outlier_frac)] *= np.float32(outlier_scale)
    return x if as_fp32 else bf16_round(x)


@dataclass(frozen=True)
class Workload:
    """One synthetic FFN workload (shapes and input recipe, no arithmetic)."""
    wid: int
    name: str
    d_model: int
    d_ff: int
    sigma: float
    batches: tuple = (1,)
    ks: tuple = (0.9,)
    variants: tuple = ("mono", "dual_ideal")
    calib_tokens: int = 256
    outlier_frac: float = 0.0
    d_rank: int = 0
    n_layers: int = 1
    eval_tokens: int = 128
    notes: str = ""
    extra: dict = field(default_factory=dict)

    def layer(self, layer: int = 0, copy: int = 0):
        return make_layer(self.wid, self.d_model, self.d_ff, self.sigma, layer, copy)

    def predictor(self, layer: int = 0, copy: int = 0):
        return make_predictor(self.wid, self.d_model, self.d_rank, self.d_ff, 0.02, layer, copy)

    def ternary(self, layer: int = 0, copy: int = 0):
        return make_ternary(self.wid, self.d_model, self.d_ff, layer=layer, copy=copy)

    def tokens(self, n: int, purpose: int = T_EVAL, layer: int = 0) -> np.ndarray:
        return make_tokens(self.wid, n, self.d_model, purpose, layer, self.outlier_frac)


WORKLOADS = {
    w.name: w
    for w in (
        Workload(0, "tiny_256x688", 256, 688, 0.02, calib_tokens=64, eval_tokens=64,
                 notes="single layer, d_model=256, d_ff=688, batch 1, k=0.9"),
        Workload(1, "llama7b_4096x11008", 4096, 11008, 0.02, ks=(0.5, 0.7, 0.9),
                 outlier_frac=0.01,
                 notes="Llama-7B-shaped layer, 1% outlier channels x20, batch 1"),
        Workload(2, "llama3_8b_4096x14336_pred", 4096, 14336, 0.02, batches=(1, 4, 8),
                 variants=("dual_pred",), d_rank=256,
                 notes="Llama-3-8B-shaped layer, seeded random low-rank predictor"),
        Workload(3, "llama70b_8192x28672", 8192, 28672, 0.015, ks=(0.7, 0.9),
                 variants=("mono", "dense"), eval_tokens=64,
                 notes="70B-shaped layer, ~1.4 GB of bf16 weights"),
        Workload(4, "stack32_llama7b_pred", 4096, 11008, 0.02, variants=("dual_pred",),
                 d_rank=256, n_layers=32,
                 notes="32 independent 7B-shaped layers, residual + RMSNorm between, "
                       "128 sequential decode tokens"),
    )
}
