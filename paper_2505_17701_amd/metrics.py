"""Mask agreement metrics of the paper's u-vs-h analysis (Sec. 6, "CIF and CAF").

For sparsity k the masks are S^k = {|s| > Quantile(k, |s|)}, U^k (from |u|) and
H^k (from |h|, h = SiLU(x.W_gate)), each with the token's own quantile. Then
  CIF^k(u, alive) = |S ^ ~H| / |S|         (u keeps alive what h would prune)
  CAF^k(u, alive) = |S ^ ~H ^ U| / |S|     (u agrees with s where h does not)
and the "dead" forms swap keeping and pruning:
  CIF^k(u, dead) = |~S ^ H| / |~S|,   CAF^k(u, dead) = |~S ^ H ^ ~U| / |~S|.
The h forms exchange U and H. Counts are pooled over the tokens (a ratio of
sums). The masks come from the GPU's per-token threshold path
(countdown_ffn_topk with the ideal D, M and CATS coefficients).
"""
from __future__ import annotations

import numpy as np


def cif_caf(S, U, H) -> dict:
    """CIF / CAF of u and of h against s from boolean masks [tokens, d_ff]."""
    S, U, H = (np.asarray(m, dtype=bool) for m in (S, U, H))
    alive, dead = S.sum(), (~S).sum()

    def ratio(num, den):
        return float(num) / float(den) if den else float("nan")

    out = {}
    for name, A, O in (("u", U, H), ("h", H, U)):  # A: the signal, O: the other factor
        out[f"CIF({name},alive)"] = ratio((S & ~O).sum(), alive)
        out[f"CAF({name},alive)"] = ratio((S & ~O & A).sum(), alive)
        out[f"CIF({name},dead)"] = ratio((~S & O).sum(), dead)
        out[f"CAF({name},dead)"] = ratio((~S & O & ~A).sum(), dead)
    return out


def masks_on_gpu(layer: dict, X, k: float):
    """Per-token masks (S, U, H) [T, d_ff] of the bf16 tokens X [T, d_model] on the GPU:
    one per-token threshold call per token and coefficient (|s|, |u|, |h|)."""
    import torch

    from . import binding as cd

    T, dm = X.shape
    dff = layer["W_up"].shape[0]
    plan = cd.Plan(dm, dff, max_batch=1)
    out = []
    for vid in (cd.CD_VARIANT_DUAL_IDEAL, cd.CD_VARIANT_MONO, cd.CD_VARIANT_CATS):
        m = torch.zeros((T, dff), dtype=torch.bool, device=X.device)
        for t in range(T):
            cd.countdown_ffn_topk(plan, vid, X[t:t + 1], layer["W_gate"], layer["W_up"],
                                  layer["W_down"], k)
            idx, _, _ = cd.countdown_export_active(plan)
            m[t, idx.long()] = True
        out.append(m.cpu().numpy())
    plan.close()
    return tuple(out)
