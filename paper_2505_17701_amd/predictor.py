"""Training the low-rank predictor of practical D-CountDown (Sec. 4, Alg. 1).

The target of token x is the ideal mask S^k = {i : |s[i]| > Quantile(k, |s|)}
(the per-token form of Eq. 6c), produced here by the HIP per-token threshold
path (countdown_ffn_topk with the ideal D coefficient). The predictor scores
s_hat = x . theta_A . theta_B (rank d_rank) and is trained with binary cross
entropy on the logits and AdamW, as in the paper's training table; at
inference a neuron is predicted alive when s_hat > thld (0 for the trained
logit). Training is plain PyTorch: only inference runs on the HIP kernels.

Layout: the returned predictor is in the kernels' layout, A_t [d_rank][d_model]
and B_t [d_ff][d_rank], bf16.

The ternary predictor of Sec. 6 (TernaryLinear, trained by the same Alg. 1)
keeps full-precision latent weights W and scores with their ternarisation
gamma * RoundClip(W / gamma, -1, 1), gamma = mean |W| (the absmean rule of
ternary "BitLinear" layers, whose name the paper's hyperparameter table
uses); the rounding passes gradients straight through. The result is the
int8 theta_t [d_ff][d_model] that countdown_ternary_pack takes (gamma > 0
only rescales the score, which the threshold absorbs).
"""
from __future__ import annotations

import time

import numpy as np


def ideal_masks(layer: dict, X, k: float):
    """S^k of every token of X [T, d_model] (bf16, on the GPU) as a bool tensor [T, d_ff]."""
    import torch

    from . import binding as cd

    T, dm = X.shape
    dff = layer["W_up"].shape[0]
    plan = cd.Plan(dm, dff, max_batch=1)
    masks = torch.zeros((T, dff), dtype=torch.bool, device=X.device)
    for t in range(T):
        cd.countdown_ffn_topk(plan, cd.CD_VARIANT_DUAL_IDEAL, X[t:t + 1], layer["W_gate"],
                              layer["W_up"], layer["W_down"], k)
        idx, _, _ = cd.countdown_export_active(plan)
        masks[t, idx.long()] = True
    plan.close()
    return masks


def random_mask_f1(true_frac: float, pred_frac: float) -> float:
    """Expected F1 of a predicted mask drawn independently of the true one, with the
    given alive fractions: precision is true_frac and recall is pred_frac, so
    F1 = 2 t p / (t + p). At a matched fraction (p = t) it equals t."""
    t, p = float(true_frac), float(pred_frac)
    return 2.0 * t * p / (t + p) if t + p > 0 else 0.0


def f1_score(pred, true) -> float:
    """F1 of predicted against true alive masks (bool arrays of one shape), pooled."""
    pred = np.asarray(pred, dtype=bool)
    true = np.asarray(true, dtype=bool)
    tp = np.count_nonzero(pred & true)
    fp = np.count_nonzero(pred & ~true)
    fn = np.count_nonzero(~pred & true)
    return 2.0 * tp / (2.0 * tp + fp + fn) if tp + fp + fn else 1.0


def train_low_rank(X, masks, d_rank: int, epochs: int = 10, lr: float = 1e-3, batch: int = 16,
                   seed: int = 42, weight_decay: float = 0.01):
    """Fit s_hat = x . theta_A . theta_B to the masks with BCE-with-logits and AdamW.

    X: [N, d_model] bf16 tokens on the GPU; masks: [N, d_ff] bool. Returns
    (A_t [d_rank, d_model] bf16, B_t [d_ff, d_rank] bf16, log dict)."""
    import torch

    g = torch.Generator(device=X.device).manual_seed(seed)
    N, dm = X.shape
    dff = masks.shape[1]
    xf = X.float()
    yf = masks.float()
    theta_a = (torch.randn(dm, d_rank, generator=g, device=X.device) / dm ** 0.5).requires_grad_()
    theta_b = (torch.randn(d_rank, dff, generator=g, device=X.device) / d_rank ** 0.5)
    theta_b.requires_grad_()
    opt = torch.optim.AdamW([theta_a, theta_b], lr=lr, weight_decay=weight_decay)
    loss_fn = torch.nn.BCEWithLogitsLoss()
    losses = []
    t0 = time.time()
    for _ in range(epochs):
        perm = torch.randperm(N, generator=g, device=X.device)
        tot, nb = 0.0, 0
        for i in range(0, N, batch):
            j = perm[i:i + batch]
            logits = (xf[j] @ theta_a) @ theta_b
            loss = loss_fn(logits, yf[j])
            opt.zero_grad(set_to_none=True)
            loss.backward()
            opt.step()
            tot += float(loss.detach())
            nb += 1
        losses.append(tot / nb)
    torch.cuda.synchronize()
    A_t = theta_a.detach().t().contiguous().to(torch.bfloat16)
    B_t = theta_b.detach().t().contiguous().to(torch.bfloat16)
    return A_t, B_t, {"epoch_loss": losses, "seconds": time.time() - t0}


def calibrated_threshold(A_t, B_t, X, k: float) -> float:
    """The Sec. 4 layerwise threshold of the predictor score s_hat at k over the
    calibration tokens X (mean of the per-token k-quantiles of s_hat). X must be
    held out from the predictor's training tokens: a trained predictor scores its
    own training tokens differently, and a threshold taken there misses the target
    alive fraction on new tokens."""
    from . import binding as cd

    dm = X.shape[1]
    plan = cd.Plan(dm, B_t.shape[0], max_batch=cd.max_batch_for(dm), d_rank=A_t.shape[0])
    th, _ = cd.countdown_calibrate(plan, cd.CD_VARIANT_DUAL_PRED, X, k, A_t=A_t, B_t=B_t)
    plan.close()
    return float(th.item())


def ternarize(W):
    """(RoundClip(W / gamma, -1, 1), gamma) with gamma = mean |W|."""
    import torch

    gamma = W.abs().mean().clamp_min(1e-8)
    return torch.clamp(torch.round(W / gamma), -1, 1), gamma


def train_ternary(X, masks, epochs: int = 10, lr: float = 1e-3, batch: int = 16, seed: int = 42,
                  weight_decay: float = 0.01):
    """Fit s_hat = x . (gamma * ternary(W)) to the masks (BCE-with-logits, AdamW, the
    straight-through estimator). X: [N, d_model] bf16 on the GPU; masks [N, d_ff] bool.
    Returns (theta_t int8 numpy [d_ff, d_model], log dict)."""
    import torch

    g = torch.Generator(device=X.device).manual_seed(seed)
    N, dm = X.shape
    dff = masks.shape[1]
    xf = X.float()
    yf = masks.float()
    W = (torch.randn(dff, dm, generator=g, device=X.device) / dm ** 0.5).requires_grad_()
    opt = torch.optim.AdamW([W], lr=lr, weight_decay=weight_decay)
    loss_fn = torch.nn.BCEWithLogitsLoss()
    losses = []
    t0 = time.time()
    for _ in range(epochs):
        perm = torch.randperm(N, generator=g, device=X.device)
        tot, nb = 0.0, 0
        for i in range(0, N, batch):
            j = perm[i:i + batch]
            q, gamma = ternarize(W)
            Wq = W + (q * gamma - W).detach()  # straight-through estimator
            loss = loss_fn(xf[j] @ Wq.t(), yf[j])
            opt.zero_grad(set_to_none=True)
            loss.backward()
            opt.step()
            tot += float(loss.detach())
            nb += 1
        losses.append(tot / nb)
    torch.cuda.synchronize()
    theta_t = ternarize(W.detach())[0].to(torch.int8).cpu().numpy()
    return theta_t, {"epoch_loss": losses, "seconds": time.time() - t0,
                     "zero_frac": float((theta_t == 0).mean())}


def calibrated_threshold_tern(theta_p, X, k: float, d_ff: int) -> float:
    """The Sec. 4 layerwise threshold of the ternary score at k over the tokens X
    (theta_p: the packed predictor on the device)."""
    from . import binding as cd

    dm = X.shape[1]
    plan = cd.Plan(dm, d_ff, max_batch=cd.max_batch_for(dm))
    th, _ = cd.countdown_calibrate_tern(plan, X, theta_p, k)
    plan.close()
    return float(th.item())


def packed_ternary(theta_t, device="cuda"):
    """countdown_ternary_pack of theta_t, moved to the device."""
    import torch

    from . import binding as cd

    return torch.from_numpy(cd.countdown_ternary_pack(theta_t).view(np.int32)).to(device)


def predicted_masks_tern(layer: dict, theta_p, X, thld: float = 0.0):
    """The ternary predictor's alive masks {s_hat > thld} of every token of X, from the
    HIP ternary path (countdown_ffn_tern) at batch 1."""
    import torch

    from . import binding as cd

    T, dm = X.shape
    dff = layer["W_up"].shape[0]
    plan = cd.Plan(dm, dff, max_batch=1)
    masks = torch.zeros((T, dff), dtype=torch.bool, device=X.device)
    for t in range(T):
        cd.countdown_ffn_tern(plan, X[t:t + 1], layer["W_gate"], layer["W_up"], layer["W_down"],
                              theta_p, thld)
        idx, _, _ = cd.countdown_export_active(plan)
        masks[t, idx.long()] = True
    plan.close()
    return masks


def predicted_masks(layer: dict, A_t, B_t, X, thld: float = 0.0):
    """The predictor's alive masks {s_hat > thld} of every token of X, from the HIP
    predictor path (countdown_ffn_dual with A_t / B_t) at batch 1."""
    import torch

    from . import binding as cd

    T, dm = X.shape
    dff = layer["W_up"].shape[0]
    plan = cd.Plan(dm, dff, max_batch=1, d_rank=A_t.shape[0])
    masks = torch.zeros((T, dff), dtype=torch.bool, device=X.device)
    for t in range(T):
        cd.countdown_ffn_dual(plan, X[t:t + 1], layer["W_gate"], layer["W_up"], layer["W_down"],
                              thld, A_t=A_t, B_t=B_t)
        idx, _, _ = cd.countdown_export_active(plan)
        masks[t, idx.long()] = True
    plan.close()
    return masks


def topk_masks(layer: dict, X, k: float, A_t=None, B_t=None, theta_p=None):
    """The predictor's alive masks at exactly the target fraction: each token keeps
    its neurons with s_hat above its own k-quantile of s_hat (the per-token form of
    the threshold, countdown_ffn_topk / countdown_ffn_tern_topk at batch 1), so the
    predicted and the true masks have the same alive count. Pass A_t and B_t for the
    low-rank predictor, theta_p (packed) for the ternary one."""
    import torch

    from . import binding as cd

    T, dm = X.shape
    dff = layer["W_up"].shape[0]
    plan = cd.Plan(dm, dff, max_batch=1, d_rank=A_t.shape[0] if A_t is not None else 0)
    masks = torch.zeros((T, dff), dtype=torch.bool, device=X.device)
    for t in range(T):
        if theta_p is not None:
            cd.countdown_ffn_tern_topk(plan, X[t:t + 1], layer["W_gate"], layer["W_up"],
                                       layer["W_down"], theta_p, k)
        else:
            cd.countdown_ffn_topk(plan, cd.CD_VARIANT_DUAL_PRED, X[t:t + 1], layer["W_gate"],
                                  layer["W_up"], layer["W_down"], k, A_t=A_t, B_t=B_t)
        idx, _, _ = cd.countdown_export_active(plan)
        masks[t, idx.long()] = True
    plan.close()
    return masks


def evaluate(layer: dict, X_cal, X_test, Y_test, k: float, A_t=None, B_t=None, theta_p=None):
    """A predictor's masks on the test tokens against their ideal masks Y_test:

    - at the Sec. 4 layerwise threshold calibrated on X_cal (held out from the
      training tokens): the threshold, the realised alive fraction and F1;
    - at the matched alive fraction (each token's own top 1 - k of s_hat): F1;
    - beside each, the F1 a random mask of the same alive fraction would score.

    Pass A_t and B_t for the low-rank predictor, theta_p for the packed ternary one."""
    ytrue = Y_test.cpu().numpy()
    t_frac = float(ytrue.mean())
    d_ff = layer["W_up"].shape[0]
    if theta_p is not None:
        th = calibrated_threshold_tern(theta_p, X_cal, k, d_ff)
        P = predicted_masks_tern(layer, theta_p, X_test, th).cpu().numpy()
    else:
        th = calibrated_threshold(A_t, B_t, X_cal, k)
        P = predicted_masks(layer, A_t, B_t, X_test, th).cpu().numpy()
    Pk = topk_masks(layer, X_test, k, A_t=A_t, B_t=B_t, theta_p=theta_p).cpu().numpy()
    alive = float(P.mean())
    return {"thld": round(th, 5), "alive_frac": round(alive, 4), "f1": round(f1_score(P, ytrue), 4),
            "f1_random_same_alive": round(random_mask_f1(t_frac, alive), 4),
            "matched_alive_frac": round(float(Pk.mean()), 4),
            "f1_matched": round(f1_score(Pk, ytrue), 4),
            "f1_random_matched": round(random_mask_f1(t_frac, float(Pk.mean())), 4)}
