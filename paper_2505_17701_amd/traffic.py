"""Algorithmic bytes and FLOPs of the sparse Gated-MLP FFN.

Two accountings:

* ``paper_flops`` / ``paper_mem_elements`` reproduce the closed forms of the
  paper's Appendix D (Table 9 FLOPs, Table 10 memory traffic, element
  counts, "MB" = elements / 2^20) and so Table 3. The active count there is
  ``s = int(d_inter * (1 - k))`` (the notation table prints ``int(d_inter * k)``,
  but only the active count reproduces the tabulated FLOPs). Table 3's
  D-CountDown memory entries equal the Table 10 sum with one ``d_inter`` term
  replaced by ``2 s``; ``tabulated=True`` gives that variant.
* ``algorithmic_bytes`` is what this implementation's kernels must move per
  call: the dense coefficient projection, the weight rows of the active
  neurons only, x and y (bf16 weights and x, fp32 y). Index lists and other
  bookkeeping are implementation overhead and are not counted.
"""
from __future__ import annotations

BF16 = 2
F32 = 4


def paper_active(d_inter: int, k: float) -> int:
    """Active neurons per token in the paper's accounting, int(d_inter (1 - k))."""
    return int(d_inter * (1.0 - k) + 1e-9)


def paper_flops(method: str, d_m: int, d_i: int, k: float, d_r: int = 512,
                c_act: int = 5) -> int:
    """FLOPs of one Gated-MLP evaluation (Table 9)."""
    if method == "dense":
        return 6 * d_m * d_i + c_act * d_i + d_i
    s = paper_active(d_i, k)
    if method == "cats":
        return 2 * d_m * d_i + c_act * d_i + 2 * d_i + 2 * d_m * s + s + 2 * d_m * s
    if method == "mono":
        return 2 * d_m * d_i + 2 * d_i + 2 * d_m * s + c_act * s + s + 2 * d_m * s
    if method == "dual_pred":
        return 2 * d_m * d_r + 2 * d_r * d_i + d_i + 4 * d_m * s + c_act * s + s + 2 * d_m * s
    raise ValueError(method)


def paper_mem_elements(method: str, d_m: int, d_i: int, k: float, d_r: int = 512,
                       tabulated: bool = True) -> int:
    """Memory reads + writes in elements (Table 10)."""
    if method == "dense":
        # W_up, W_gate; x twice; gate, up; gate; act_gate; act_gate, up; inter; W_down; inter; y
        return (2 * d_m * d_i + 2 * d_m + 2 * d_i + d_i + d_i + 2 * d_i + d_i + d_m * d_i + d_i
                + d_m)
    s = paper_active(d_i, k)
    if method == "cats":
        return (d_m * d_i + d_m + 7 * d_i + d_m * s + d_m + s + d_i + d_i + d_m * s + d_i + d_m)
    if method == "mono":
        return (d_m * d_i + d_m + 5 * d_i + d_m * s + d_m + s + d_i + d_i + d_m * s + d_i + d_m)
    if method == "dual_pred":
        total = (d_m * d_r + d_m + d_r + d_r * d_i + d_r + 3 * d_i + 2 * d_m * s + d_m + d_i + d_i
                 + d_m * s + d_i + d_m)
        return total - d_i + 2 * s if tabulated else total
    raise ValueError(method)


def algorithmic_bytes(variant: str, d_model: int, d_ff: int, n_active: int, B: int = 1,
                      d_rank: int = 0) -> dict:
    """Bytes the kernels must move for one call, per kernel and in total.

    ``coef`` is the coefficient kernel (dense projection + gathered gate /
    gate+up rows), ``down`` the gathered down projection, ``latent`` the
    predictor's first product. x and y are counted once, on the kernel that
    reads / writes them.
    """
    row = BF16 * d_model
    x = BF16 * B * d_model
    y = F32 * B * d_model
    if variant in ("mono", "cats"):  # one dense projection, the other gathered
        k = {"coef": d_ff * row + n_active * row + x, "down": n_active * row + y}
    elif variant == "dual_ideal":
        k = {"coef": 2 * d_ff * row + x, "down": n_active * row + y}
    elif variant == "dense":
        k = {"coef": 2 * d_ff * row + x, "down": d_ff * row + y}
    elif variant == "dual_pred":
        lat = F32 * B * d_rank
        k = {"latent": BF16 * d_rank * d_model + x + lat,
             "coef": BF16 * d_ff * d_rank + lat + 2 * n_active * row,
             "down": n_active * row + y}
    elif variant == "dual_tern":  # theta at 2 bits per weight, no latent
        k = {"coef": d_ff * d_model // 4 + x + 2 * n_active * row, "down": n_active * row + y}
    else:
        raise ValueError(variant)
    k["total"] = sum(k.values())
    return k


def algorithmic_flops(variant: str, d_model: int, d_ff: int, n_active: int, B: int = 1,
                      d_rank: int = 0) -> int:
    """Multiply-adds x 2 of one call (activation and threshold work not counted)."""
    mac = {
        "mono": d_ff * d_model + 2 * n_active * d_model,
        "cats": d_ff * d_model + 2 * n_active * d_model,
        "dual_ideal": 2 * d_ff * d_model + n_active * d_model,
        "dense": 3 * d_ff * d_model,
        "dual_pred": d_rank * d_model + d_ff * d_rank + 3 * n_active * d_model,
        "dual_tern": d_ff * d_model + 3 * n_active * d_model,
    }[variant]
    return 2 * B * mac
