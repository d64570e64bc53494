#!/usr/bin/env python3
"""Decode-step benchmark of the COUNTDOWN sparse Gated-MLP FFN on one MI355X.

A step is one decode token through one FFN layer on the HIP path: the
coefficient kernel (dense W_up projection, threshold, compaction, gathered
gate rows) and the gathered down projection. Default workload (the largest
single-GPU configuration): the 70B-shaped layer (d_model 8192, d_ff 28672,
bf16 weights N(0, 0.015^2), 1.41 GB, batch 1), M-CountDown at sparsity k = 0.9
with the layerwise threshold calibrated on the GPU from 256 seeded tokens.
Secondary lines: the Llama-7B-shaped layer (M, ideal D, CATS, per-token
thresholds, dense), the Llama-3-8B-shaped layer with the low-rank and ternary
predictors at batch 1/4/8, the 32-layer stack, predictor training. Weights
are rotated over enough independent copies (> 1 GB in total) that the 256 MB
Infinity Cache cannot serve them; inputs are resident in HBM before the timed
region starts.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E peak, GB/s
KERNEL_SRCS = [os.path.join(ROOT, "paper_2505_17701_amd", "csrc", f)
               for f in ("cd_kernels.hip", "cd_device.hpp", "cd_internal.hpp")]
# committed FETCH_SIZE / WRITE_SIZE summaries of a line's dominant kernel(s), by
# (workload, variant, k, batch)
TRAFFIC_SUMMARIES = {
    ("llama70b_8192x28672", "mono", 0.9, 1): "k_coef_mono_llama70b_8192x28672_k0.9_traffic.md",
    ("llama7b_4096x11008", "mono", 0.9, 1): "k_coef_mono_llama7b_4096x11008_k0.9_traffic.md",
    ("llama3_8b_4096x14336_pred", "dual_pred", 0.9, 1):
        "k_coef_pred_llama3_8b_4096x14336_k0.9_b1_traffic.md",
    ("llama3_8b_4096x14336_pred", "dual_pred", 0.9, 4):
        "k_coef_pred_llama3_8b_4096x14336_k0.9_b4_traffic.md",
    ("llama3_8b_4096x14336_pred", "dual_pred", 0.9, 8):
        "k_coef_pred_mfma_llama3_8b_4096x14336_k0.9_b8_traffic.md",
    ("llama3_8b_4096x14336_pred", "dual_tern", 0.9, 1):
        "k_coef_tern_llama3_8b_4096x14336_k0.9_b1_traffic.md",
    ("llama3_8b_4096x14336_pred", "dual_tern", 0.9, 8):
        "k_coef_tern_mfma_llama3_8b_4096x14336_k0.9_b8_traffic.md",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def dev_bf16(a):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to("cuda")


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=2000)
    p.add_argument("--warmup", type=int, default=200)
    p.add_argument("--workload", default="llama70b_8192x28672")
    p.add_argument("--variant", default="mono",
                   choices=["mono", "dual_ideal", "dual_pred", "dual_tern", "dense", "cats",
                            "mono_topk", "dual_ideal_topk", "dual_pred_topk", "dual_tern_topk",
                            "cats_topk"])
    p.add_argument("--batch", type=int, default=1, help="decode tokens per call (union IDX)")
    p.add_argument("--k", type=float, default=0.9)
    p.add_argument("--copies", type=int, default=0,
                   help="independent weight copies rotated (0: enough for more than 1 GB)")
    p.add_argument("--tokens", type=int, default=64, help="distinct eval tokens rotated")
    p.add_argument("--calib-tokens", type=int, default=256)
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="time budget of the oracle CPU baseline (0 disables it)")
    p.add_argument("--no-extra", action="store_true",
                   help="skip the secondary variants and the other workloads")
    p.add_argument("--no-other", action="store_true",
                   help="skip the other workloads (7B, 8B-predictor, 70B, stack, training)")
    p.add_argument("--no-7b", action="store_true", help="skip the 7B-shaped layer's lines")
    p.add_argument("--no-8b", action="store_true", help="skip the 8B predictor layer's lines")
    p.add_argument("--no-stack", action="store_true", help="skip the 32-layer stack")
    p.add_argument("--no-train", action="store_true", help="skip the predictor-training run")
    p.add_argument("--traffic-probe", action="store_true",
                   help="first copy a 256 MiB device buffer 3 times (the known-size reference "
                        "for FETCH_SIZE / WRITE_SIZE counters)")
    return p.parse_args()


def kernel_source_digest():
    """sha256 of the device sources with comments and whitespace removed: the
    identity of the kernels a traffic measurement belongs to."""
    import hashlib
    import re

    h = hashlib.sha256()
    for path in KERNEL_SRCS:
        src = open(path).read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()


def measured_traffic(key):
    """HBM bytes per launch of a line's dominant kernel(s) from the committed
    FETCH_SIZE / WRITE_SIZE summary, or None when there is none or the kernel
    source changed since it was taken."""
    name = TRAFFIC_SUMMARIES.get(key)
    path = os.path.join(ROOT, "profiles", name) if name else None
    if not path or not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and line.startswith("- "):
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    if fields.get("kernel_source_digest") != kernel_source_digest():
        return None
    try:
        return float(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def time_steps(fn, steps, warmup, stream):
    """Warm up, then time exactly `steps` eager calls between two synchronisations."""
    import torch

    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for i in range(steps):
        fn(i)
    t1.record(stream)
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps  # ms per step


def time_steps_graph(fn, steps, warmup, extra=None):
    """Warm up eagerly, capture exactly `steps` calls into one HIP graph, replay it once
    untimed and once timed between two synchronisations; returns ms per call of that
    replay. With a list `extra`, a few more timed replays append their ms per call to it
    (spread statistics only)."""
    import torch

    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(steps):
            fn(i)
    g.replay()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    g.replay()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    if extra is not None:
        for _ in range(5):
            t0.record()
            g.replay()
            t1.record()
            torch.cuda.synchronize()
            extra.append(t0.elapsed_time(t1) / steps)
    del g
    return ms


def pooled_thresholds(dm, dff, dr, L, X_cal, variants, ks):
    """The other reading of the calibration rule, reported beside the one used (the
    mean of per-token quantiles): one linear quantile of the coefficients of all
    calibration tokens pooled. The coefficients come from the HIP coefficient kernels
    (threshold +inf, coefficient phase only); the quantile is numpy's."""
    import torch

    from paper_2505_17701_amd import binding as cd

    mb = cd.max_batch_for(dm)
    plan = cd.Plan(dm, dff, max_batch=mb, d_rank=dr, keep_coef=True)
    cd.countdown_plan_set_phases(plan, cd.CD_PHASE_COEF)
    inf = float("inf")
    out = {}
    for variant in variants:
        chunks = []
        for t0 in range(0, X_cal.shape[0], mb):
            x = X_cal[t0:t0 + mb]
            y = torch.empty((x.shape[0], dm), dtype=torch.float32, device="cuda")
            if variant == "mono":
                cd.countdown_ffn_mono(plan, x, L["W_gate"], L["W_up"], L["W_down"], inf, y=y)
            elif variant == "dual_ideal":
                cd.countdown_ffn_dual(plan, x, L["W_gate"], L["W_up"], L["W_down"], inf, y=y)
            elif variant == "cats":
                cd.countdown_ffn_cats(plan, x, L["W_gate"], L["W_up"], L["W_down"], inf, y=y)
            elif variant == "dual_pred":
                cd.countdown_ffn_dual(plan, x, L["W_gate"], L["W_up"], L["W_down"], inf,
                                      A_t=L["A_t"], B_t=L["B_t"], y=y)
            elif variant == "dual_tern":
                cd.countdown_ffn_tern(plan, x, L["W_gate"], L["W_up"], L["W_down"],
                                      L["theta_p"], inf, y=y)
            else:
                continue
            chunks.append(cd.countdown_export_active(plan)[2].cpu().numpy().astype(np.float64))
        if not chunks:
            continue
        c = np.concatenate(chunks).ravel()
        if variant not in ("dual_pred", "dual_tern"):  # signed scores keep their sign
            c = np.abs(c)
        for k in ks:
            out[(variant, k)] = float(np.float32(np.quantile(c, k)))
    plan.close()
    return out


def stream_ceiling(ctx, nk):
    """Plain streaming reads (countdown_stream_read), timed like the kernels with one
    event pair around a graph-replayed loop: the W_up matrices of the rotated weight
    copies (the bytes the M coefficient kernel streams densely, one launch each), a
    1 GiB buffer (the asymptotic read rate), and a 32-byte read, whose time per
    launch is what one more dependent launch costs in a graph."""
    import torch

    from paper_2505_17701_amd import binding as cd

    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    ups = [L["W_up"] for L in ctx.layers]
    nb = ups[0].numel() * ups[0].element_size()
    ms = time_steps_graph(lambda i: cd.countdown_stream_read(ups[i % len(ups)], sink), nk, 20)
    out = {"W_up": {"bytes": nb, "us": ms * 1e3, "GBs": nb / (ms * 1e-3) / 1e9}}
    big = torch.zeros(1 << 29, dtype=torch.bfloat16, device="cuda")  # 1 GiB
    nb = big.numel() * 2
    ms = time_steps_graph(lambda i: cd.countdown_stream_read(big, sink), 40, 5)
    out["1GiB"] = {"bytes": nb, "us": ms * 1e3, "GBs": nb / (ms * 1e-3) / 1e9}
    del big
    tiny = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    ms = time_steps_graph(lambda i: cd.countdown_stream_read(tiny, sink), 400, 20)
    out["launch"] = {"bytes": 32, "us": ms * 1e3}
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def brief(r):
    return {kk: r[kk] for kk in ("us_per_layer", "us_per_layer_eager", "tokens_per_s",
                                 "achieved_GBs", "frac_hbm_peak", "n_active_mean",
                                 "realised_sparsity", "coef_kernel_us", "coef_kernel_GBs",
                                 "down_kernel_us", "latent_kernel_us")
            if kk in r}


class Context:
    """One workload on the device: rotated weight copies, eval tokens, thresholds
    calibrated on the GPU (mean of per-token quantiles over seeded tokens)."""

    def __init__(self, w, copies, ntok, ncal, ks, max_batch, variants=None):
        import torch

        from paper_2505_17701_amd import binding as cd
        from workloads.synth import T_CALIB

        self.w, self.copies, self.max_batch = w, copies, max_batch
        self.dm, self.dff, self.dr = w.d_model, w.d_ff, w.d_rank
        t = time.time()
        self.layers = []
        self.host0 = None
        variants = variants or [v for v in w.variants if v != "dense"]
        for c in range(copies):
            L = w.layer(copy=c)
            if w.d_rank:
                L.update(w.predictor(copy=c))
            D = {k: dev_bf16(v) for k, v in L.items()}
            if "dual_tern" in variants:  # the ternary predictor, packed for the kernels
                T = w.ternary(copy=c)
                packed = cd.countdown_ternary_pack(T)
                D["theta_p"] = torch.from_numpy(packed.view(np.int32)).to("cuda")
                L["theta_t"] = T
            if c == 0:
                self.host0 = L
            self.layers.append(D)
        self.X_eval_h = w.tokens(ntok)
        self.X_eval = dev_bf16(self.X_eval_h)
        X_cal = dev_bf16(w.tokens(ncal, purpose=T_CALIB))
        torch.cuda.synchronize()
        gb = sum(v.numel() * v.element_size() for v in self.layers[0].values()) * copies / 1e9
        log(f"[bench] {copies} weight copies of {w.name} on device ({gb:.2f} GB) in "
            f"{time.time() - t:.1f}s")
        vids = {"mono": cd.CD_VARIANT_MONO, "dual_ideal": cd.CD_VARIANT_DUAL_IDEAL,
                "dual_pred": cd.CD_VARIANT_DUAL_PRED, "cats": cd.CD_VARIANT_CATS}
        # tokens per calibration launch: the widest batch tile the shape allows
        cal_plan = cd.Plan(self.dm, self.dff, max_batch=cd.max_batch_for(self.dm), d_rank=self.dr)
        self.thld = {}
        L0 = self.layers[0]
        for variant in variants:
            for k in ks:
                if variant == "dual_tern":
                    th, _ = cd.countdown_calibrate_tern(cal_plan, X_cal, L0["theta_p"], k)
                else:
                    th, _ = cd.countdown_calibrate(cal_plan, vids[variant], X_cal, k,
                                                   W_gate=L0["W_gate"], W_up=L0["W_up"],
                                                   A_t=L0.get("A_t"), B_t=L0.get("B_t"))
                self.thld[(variant, k)] = float(th.item())
        cal_plan.close()
        self.thld_pooled = pooled_thresholds(self.dm, self.dff, self.dr, L0, X_cal, variants, ks)
        del X_cal
        log(f"[bench] thresholds: " + ", ".join(f"{v}@{k}={t:.4f}"
                                                 for (v, k), t in self.thld.items()))
        log(f"[bench] pooled-quantile thresholds (reported only): " + ", ".join(
            f"{v}@{k}={t:.4f}" for (v, k), t in self.thld_pooled.items()))

    def free(self):
        import torch

        self.layers = None
        self.X_eval = None
        torch.cuda.empty_cache()

    def make_step(self, plan, variant, k, B, y):
        from paper_2505_17701_amd import binding as cd

        th = self.thld.get((variant, k), 0.0)
        ntok = self.X_eval.shape[0] - B + 1
        X, layers, copies = self.X_eval, self.layers, self.copies

        topk = variant.endswith("_topk")
        base = variant[:-5] if topk else variant
        vid = {"mono": cd.CD_VARIANT_MONO, "dual_ideal": cd.CD_VARIANT_DUAL_IDEAL,
               "dual_pred": cd.CD_VARIANT_DUAL_PRED, "cats": cd.CD_VARIANT_CATS}.get(base)

        def step(i):
            L = layers[i % copies]
            x = X[i % ntok: i % ntok + B]
            if topk and base == "dual_tern":
                cd.countdown_ffn_tern_topk(plan, x, L["W_gate"], L["W_up"], L["W_down"],
                                           L["theta_p"], k, y=y)
            elif topk:  # per-token threshold: the k-quantile of each token's own coefficients
                cd.countdown_ffn_topk(plan, vid, x, L["W_gate"], L["W_up"], L["W_down"], k,
                                      A_t=L.get("A_t") if base == "dual_pred" else None,
                                      B_t=L.get("B_t") if base == "dual_pred" else None, y=y)
            elif variant == "mono":
                cd.countdown_ffn_mono(plan, x, L["W_gate"], L["W_up"], L["W_down"], th, y=y)
            elif variant == "dual_ideal":
                cd.countdown_ffn_dual(plan, x, L["W_gate"], L["W_up"], L["W_down"], th, y=y)
            elif variant == "cats":
                cd.countdown_ffn_cats(plan, x, L["W_gate"], L["W_up"], L["W_down"], th, y=y)
            elif variant == "dual_pred":
                cd.countdown_ffn_dual(plan, x, L["W_gate"], L["W_up"], L["W_down"], th,
                                      A_t=L["A_t"], B_t=L["B_t"], y=y)
            elif variant == "dual_tern":
                cd.countdown_ffn_tern(plan, x, L["W_gate"], L["W_up"], L["W_down"],
                                      L["theta_p"], th, y=y)
            else:
                cd.countdown_ffn_dense(plan, x, L["W_gate"], L["W_up"], L["W_down"], y=y)
        return step

    def measure(self, variant, k, B, steps, warmup, replays=False, deterministic=False):
        import torch

        from paper_2505_17701_amd import binding as cd
        from paper_2505_17701_amd import traffic

        dm, dff, dr = self.dm, self.dff, self.dr
        stream = torch.cuda.current_stream()
        y = torch.empty((B, dm), dtype=torch.float32, device="cuda")
        base = variant[:-5] if variant.endswith("_topk") else variant
        plan = cd.Plan(dm, dff, max_batch=max(B, self.max_batch),
                       d_rank=dr if base == "dual_pred" else 0, deterministic=deterministic)
        step = self.make_step(plan, variant, k, B, y)
        ms_eager = time_steps(step, steps, warmup, stream)
        rep = [] if replays else None
        ms = time_steps_graph(step, steps, warmup, rep)
        # per-kernel averages: graph-replayed loops of a single kernel (the plan's phase
        # selection), each bracketed by one HIP event pair on the launch stream
        nk = min(steps, 512)
        cd.countdown_plan_set_phases(plan, cd.CD_PHASE_COEF)
        ms_coef = time_steps_graph(step, nk, 20)
        lib = cd.load_library()
        n_down = torch.zeros(1, dtype=torch.int32, device="cuda")
        lib.countdown_export_active(plan.handle, None, n_down.data_ptr(), None, None,
                                    stream.cuda_stream)
        cd.countdown_plan_set_phases(plan, cd.CD_PHASE_DOWN)  # rows of the last coef call
        ms_down = time_steps_graph(step, nk, 20)
        cd.countdown_plan_set_phases(plan, cd.CD_PHASE_ALL)
        # |IDX| of every call of the loop, for the byte counts
        n_arr = torch.zeros(nk, dtype=torch.int32, device="cuda")
        for i in range(nk):
            step(i)
            lib.countdown_export_active(plan.handle, None, n_arr[i:i + 1].data_ptr(), None,
                                        None, stream.cuda_stream)
        torch.cuda.synchronize()
        plan.close()
        n = n_arr.cpu().numpy().astype(np.float64)
        dr_v = dr if base == "dual_pred" else 0
        per = [traffic.algorithmic_bytes(base, dm, dff, int(v), B=B, d_rank=dr_v) for v in n]
        res = {"batch": B, "ms_per_step": ms, "us_per_layer": ms * 1e3,
               **({"us_per_layer_5_more_replays": [r * 1e3 for r in rep],
                   "us_per_layer_median_of_6": float(np.median([ms] + rep)) * 1e3,
                   "us_per_layer_mean_of_6": float(np.mean([ms] + rep)) * 1e3} if rep else {}),
               "tokens_per_s": B * 1e3 / ms, "us_per_layer_eager": ms_eager * 1e3,
               "n_active_mean": float(n.mean()), "realised_sparsity": float(1 - n.mean() / dff)}
        # the coefficient loop includes the predictor's latent kernel (one launch each)
        coef_b = float(np.mean([p["coef"] + p.get("latent", 0) for p in per]))
        down_b = traffic.algorithmic_bytes(base, dm, dff, int(n_down.item()), B=B,
                                           d_rank=dr_v)["down"]
        for name, kms, kb in (("coef", ms_coef, coef_b), ("down", ms_down, down_b)):
            res[f"{name}_kernel_us"] = kms * 1e3
            res[f"{name}_kernel_bytes"] = kb
            res[f"{name}_kernel_GBs"] = kb / (kms * 1e-3) / 1e9
        tot_bytes = float(np.mean([p["total"] for p in per]))
        res["algorithmic_bytes"] = tot_bytes
        res["achieved_GBs"] = tot_bytes / (ms * 1e-3) / 1e9
        res["frac_hbm_peak"] = res["achieved_GBs"] / HBM_PEAK_GBS
        return res


def optimal_dense_us(ctx, k, steps):
    """The dense layer with only int(d_ff (1 - k)) neurons (rounded down to a multiple
    of 8): the first rows of the rotated weight copies, through the dense path."""
    import torch

    from paper_2505_17701_amd import binding as cd

    n = max(8, int(ctx.dff * (1 - k)) // 8 * 8)
    plan = cd.Plan(ctx.dm, n, max_batch=1)
    y = torch.empty((1, ctx.dm), dtype=torch.float32, device="cuda")
    views = [{m: L[m][:n] for m in ("W_gate", "W_up", "W_down")} for L in ctx.layers]
    X, nt = ctx.X_eval, ctx.X_eval.shape[0]

    def step(i):
        L = views[i % len(views)]
        cd.countdown_ffn_dense(plan, X[i % nt:i % nt + 1], L["W_gate"], L["W_up"], L["W_down"],
                               y=y)

    ms = time_steps_graph(step, steps, 30)
    plan.close()
    return ms * 1e3


def kernel_desc(variant, B=1):
    """The kernel(s) of a line's coefficient phase, the dominant part of every call."""
    pred = ("k_coef_pred_mfma" if B >= 5 else
            "k_coef_pred (8 waves per block)" if B >= 3 else "k_coef_pred")
    tern = ("k_coef_tern_mfma (score on MFMA at d_model 4096)" if B >= 5 else
            "k_coef_tern (8 waves per block)" if B >= 3 else "k_coef_tern")
    sel = "k_topk_gather1 (select, flags and gather in one launch)" if B == 1 else \
        "k_topk_select + k_gather_topk"
    return {"mono": "k_coef_mono (dense W_up GEMV, threshold, wave-local W_gate gather, s)",
            "dual_ideal": "k_coef_dual (dense W_gate + W_up GEMV, s, threshold)",
            "dual_pred": f"k_latent + {pred} (predictor latent, scores, threshold, block-local "
                         "W_gate / W_up gather, s)",
            "dense": "k_coef_dual (dense W_gate + W_up GEMV, s)",
            "mono_topk": f"k_coef_mono + {sel} (per-token threshold)",
            "dual_ideal_topk": "k_coef_dual + k_topk_select (per-token threshold; the select "
                               "sets the flags, s is the coefficient)"
                               + ("; the phase timed alone: a whole one-token call runs "
                                  "k_coef_dual, then k_topk_down1 (select, flags and down "
                                  "projection in one launch)" if B == 1 else ""),
            "dual_pred_topk": f"k_latent + {pred} + {sel} (per-token threshold)",
            "cats": "k_coef_mono<CATS> (dense W_gate GEMV, SiLU, threshold, W_up gather)",
            "cats_topk": f"k_coef_mono<CATS> + {sel} (per-token threshold)",
            "dual_tern": f"{tern} (ternary predictor scores, threshold, block-local W_gate / "
                         "W_up gather, s)",
            "dual_tern_topk": f"{tern} + {sel} (per-token threshold)"
            }[variant]


def roofline(res, variant, key, ceiling=None):
    """Roofline object of a line: the coefficient phase (its dominant kernel, with the
    predictor's latent launch where there is one): algorithmic bytes per launch over
    the launch's average duration, both measured in this run; traffic from the
    committed PMC summary of the same kernel source, or None."""
    kb, kus = res["coef_kernel_bytes"], res["coef_kernel_us"]
    ach = kb / (kus * 1e-6) / 1e9
    obj = {"bound": "hbm", "kernel": kernel_desc(variant, res["batch"]), "achieved": ach,
           "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBS,
           "traffic": measured_traffic(key), "bytes_per_launch": kb, "avg_launch_us": kus}
    if ceiling:
        # measured read ceilings: a plain read of one rotated W_up per launch, and of 1 GiB
        obj.update({"stream_W_up_GBs": ceiling["W_up"]["GBs"],
                    "stream_1GiB_GBs": ceiling["1GiB"]["GBs"],
                    "frac_of_stream_1GiB": ach / ceiling["1GiB"]["GBs"],
                    "dependent_launch_us": ceiling["launch"]["us"]})
    return obj


def auto_copies(w):
    """Weight copies to rotate: enough that they exceed 1 GB (the 256 MB Infinity Cache
    then serves none of a call's weight bytes)."""
    per = 3 * w.d_ff * w.d_model * 2 + (w.d_rank * (w.d_model + w.d_ff) * 2 if w.d_rank else 0)
    return max(1, -(-1_000_000_000 // per))


def workload_lines(ctx, args, skip):
    """The secondary lines of the 7B- and 70B-shaped layers (batch 1): the dense FFN and
    the other variants and sparsities of the workload, with speedups over dense beside
    the ideal byte ratio."""
    from paper_2505_17701_amd import traffic

    w = ctx.w
    if w.name == "llama7b_4096x11008":
        todo = (("mono", 0.9), ("dense", None), ("dual_ideal", 0.9), ("mono", 0.7), ("mono", 0.5),
                ("cats", 0.9), ("mono_topk", 0.9), ("dual_ideal_topk", 0.9), ("cats_topk", 0.9))
    elif w.name == "llama70b_8192x28672":
        todo = (("mono", 0.9), ("mono", 0.7), ("dense", None))
    else:
        return {}, {}
    n = max(100 if w.d_model > 4096 else 200, args.steps // 4)
    lines, res = {}, {}
    for variant, k in todo:
        name = variant + ("" if k is None else f"@k={k}")
        if (variant, k) == skip:
            continue
        res[name] = ctx.measure(variant, k, 1, n, 30)
        lines[name] = brief(res[name])
        log(f"[bench] {w.name} {name}: {json.dumps(lines[name])}")
    dense = res.get("dense")
    if dense:
        dense_b = traffic.algorithmic_bytes("dense", w.d_model, w.d_ff, w.d_ff)["total"]
        for name, r in res.items():
            if name != "dense":
                lines[name]["speedup_vs_dense"] = dense["us_per_layer"] / r["us_per_layer"]
                lines[name]["ideal_byte_ratio"] = dense_b / r["algorithmic_bytes"]
    if w.name == "llama7b_4096x11008":
        # mask agreement of u and h with s (CIF / CAF) on the layer's eval tokens
        from paper_2505_17701_amd.metrics import cif_caf, masks_on_gpu

        lines["cif_caf"] = {}
        for k in (0.5, 0.7, 0.9):
            m = cif_caf(*masks_on_gpu(ctx.layers[0], ctx.X_eval[:32], k))
            lines["cif_caf"][f"k={k}"] = {kk: round(v, 4) for kk, v in m.items()}
        log(f"[bench] CIF/CAF: {json.dumps(lines['cif_caf'])}")
    return lines, res


def layer_block(args, wname):
    """A single-layer workload that is not the headline: its M-CountDown k 0.9 line
    with a roofline object and the read ceilings, then its other lines."""
    from workloads import WORKLOADS

    w = WORKLOADS[wname]
    variants = ["mono", "dual_ideal", "cats"] if w.name == "llama7b_4096x11008" else ["mono"]
    ctx = Context(w, auto_copies(w), args.tokens, args.calib_tokens, list(w.ks),
                  max_batch=1, variants=variants)
    r = ctx.measure("mono", 0.9, 1, max(200 if w.d_model <= 4096 else 100, args.steps), 30,
                    replays=True)
    ceiling = stream_ceiling(ctx, min(max(args.steps, 64), 512))
    lines, res = workload_lines(ctx, args, ("mono", 0.9))
    # the same call with the fixed-order reduction of y (CD_PLAN_DETERMINISTIC)
    rd = ctx.measure("mono", 0.9, 1, max(200 if w.d_model <= 4096 else 100, args.steps // 4),
                     30, deterministic=True)
    lines["mono@k=0.9 deterministic"] = {**brief(rd), "cost_us": rd["us_per_layer"] -
                                         r["us_per_layer"]}
    log(f"[bench] {w.name} mono@k=0.9 deterministic: "
        f"{json.dumps(lines['mono@k=0.9 deterministic'])}")
    dense = res.get("dense")
    out = {"mono@k=0.9": {**brief(r), "us_per_layer_median_of_6": r["us_per_layer_median_of_6"],
                          "roofline": roofline(r, "mono", (w.name, "mono", 0.9, 1), ceiling)},
           **lines, "stream_ceiling": ceiling}
    if dense:
        from paper_2505_17701_amd import traffic

        out["mono@k=0.9"]["speedup_vs_dense"] = dense["us_per_layer"] / r["us_per_layer"]
        out["mono@k=0.9"]["ideal_byte_ratio"] = (traffic.algorithmic_bytes(
            "dense", w.d_model, w.d_ff, w.d_ff)["total"] / r["algorithmic_bytes"])
    log(f"[bench] {w.name} mono@k=0.9: {json.dumps(out['mono@k=0.9'])}")
    ctx.free()
    return out


def eight_b_block(args):
    """The Llama-3-8B-shaped layer with the low-rank predictor at batch 1/4/8 (each with
    a roofline object), the per-token form, the ternary predictor, dense, and the
    paper's kernel-speed comparison across sparsity at this shape."""
    from workloads import WORKLOADS

    w = WORKLOADS["llama3_8b_4096x14336_pred"]
    sweep_ks = (0.5, 0.6, 0.7, 0.8, 0.9)
    ctx = Context(w, auto_copies(w), 64, args.calib_tokens, list(sweep_ks), max_batch=8,
                  variants=["dual_pred", "dual_tern", "mono", "cats"])
    r8 = {}
    n = max(200, args.steps // 4)
    for B in w.batches:
        r = ctx.measure("dual_pred", 0.9, B, n, 50)
        r8[f"B={B}"] = {**brief(r), "roofline": roofline(r, "dual_pred",
                                                         (w.name, "dual_pred", 0.9, B))}
        log(f"[bench] {w.name} dual_pred B={B}: {json.dumps(r8[f'B={B}'])}")
    for B in (1, 8):  # the fixed-order reduction of y (CD_PLAN_DETERMINISTIC)
        r = ctx.measure("dual_pred", 0.9, B, n, 50, deterministic=True)
        r8[f"B={B} deterministic"] = {**brief(r), "cost_us": r["us_per_layer"] -
                                      r8[f"B={B}"]["us_per_layer"]}
        log(f"[bench] {w.name} dual_pred B={B} deterministic: "
            f"{json.dumps(r8[f'B={B} deterministic'])}")
    r = ctx.measure("dual_pred_topk", 0.9, 1, n, 50)
    r8["per-token k=0.9 B=1"] = brief(r)
    log(f"[bench] {w.name} dual_pred per-token B=1: {json.dumps(r8['per-token k=0.9 B=1'])}")
    for B in w.batches:  # the ternary predictor (Sec. 6) in the low-rank one's place
        r = ctx.measure("dual_tern", 0.9, B, n, 50)
        r8[f"ternary B={B}"] = {**brief(r), "roofline": roofline(r, "dual_tern",
                                                                 (w.name, "dual_tern", 0.9, B))}
        log(f"[bench] {w.name} dual_tern B={B}: {json.dumps(r8[f'ternary B={B}'])}")
    r = ctx.measure("dense", None, 1, n, 50)
    r8["dense B=1"] = brief(r)
    for B in w.batches:
        r8[f"B={B}"]["speedup_vs_dense_B1"] = r["us_per_layer"] / r8[f"B={B}"]["us_per_layer"]
    # the paper's kernel-speed comparison at this shape (its Llama-3.1-8B figure): CATS,
    # M-CountDown and practical D-CountDown at calibrated thresholds across sparsity,
    # beside the dense layer ("Full") and a dense layer of the active count ("Optimal")
    sweep = {"dense_us": r["us_per_layer"]}
    for k in sweep_ks:
        row = {v: ctx.measure(v, k, 1, max(200, args.steps // 8), 30)["us_per_layer"]
               for v in ("cats", "mono", "dual_pred")}
        row["optimal_us"] = optimal_dense_us(ctx, k, max(200, args.steps // 8))
        sweep[f"k={k}"] = row
        log(f"[bench] {w.name} kernel speed k={k} (us per layer): {json.dumps(row)}")
    r8["kernel_speed_sweep"] = sweep
    ctx.free()
    return r8


def predictor_training_bench(args, n_train=8192, n_cal=256, n_test=256, epochs=4):
    """Alg. 1 on the Llama-3-8B-shaped layer (d_rank 256): targets S^k from the HIP
    per-token ideal-D path, BCE + AdamW (lr 1e-3, batch 16) in PyTorch, then each
    predictor through the HIP predictor path on held-out test tokens:

    - at its Sec. 4 threshold, calibrated at k on held-out tokens (neither training
      nor test): the realised alive fraction and F1, beside the F1 of a random
      mask with that alive fraction;
    - at exactly the target alive fraction (each token's own top 1 - k of the
      score), where a random mask scores F1 = 1 - k;
    - at the paper's inference rule s_hat > 0 (low-rank only).

    Weights and tokens are seeded random. A linear predictor of rank 256 follows a
    random full-rank W_gate only within a 256-dimensional subspace, so the low-rank
    predictor stays near the random baseline here; the full-rank ternary one does
    not. The paper's F1 values need its trained models."""
    import torch

    from paper_2505_17701_amd.predictor import (evaluate, f1_score, ideal_masks, packed_ternary,
                                                 predicted_masks, train_low_rank, train_ternary)
    from workloads import WORKLOADS
    from workloads.synth import T_CALIB, T_HELDOUT

    w = WORKLOADS["llama3_8b_4096x14336_pred"]
    L = {kk: dev_bf16(v) for kk, v in w.layer().items()}
    Xtr = dev_bf16(w.tokens(n_train, purpose=T_CALIB))
    Xcal = dev_bf16(w.tokens(n_cal, purpose=T_HELDOUT))
    Xte = dev_bf16(w.tokens(n_test))
    out = {"d_rank": w.d_rank, "train_tokens": n_train, "calibration_tokens": n_cal,
           "test_tokens": n_test, "epochs": epochs,
           "calibration": "held-out tokens (a stream of their own), not the training set"}
    for k in (0.7, 0.9):
        t = time.time()
        Ytr = ideal_masks(L, Xtr, k)
        Yte = ideal_masks(L, Xte, k)
        t_mask = time.time() - t
        A0, B0, _ = train_low_rank(Xtr, Ytr, w.d_rank, epochs=0)
        A, B, tl = train_low_rank(Xtr, Ytr, w.d_rank, epochs=epochs)
        ytrue = Yte.cpu().numpy()
        r = {"target_alive_frac": round(float(ytrue.mean()), 4)}
        for name, (At, Bt) in (("untrained", (A0, B0)), ("trained", (A, B))):
            r[name] = evaluate(L, Xcal, Xte, Yte, k, A_t=At, B_t=Bt)
            P_0 = predicted_masks(L, At, Bt, Xte, 0.0).cpu().numpy()
            r[name].update({"f1_thld0": round(f1_score(P_0, ytrue), 4),
                            "alive_frac_thld0": round(float(P_0.mean()), 4)})
        r.update({"epoch_loss": [round(v, 5) for v in tl["epoch_loss"]],
                  "train_seconds": round(tl["seconds"], 2), "mask_seconds": round(t_mask, 2)})
        # the ternary predictor (Sec. 6) by the same procedure, straight-through estimator
        T, tt = train_ternary(Xtr, Ytr, epochs=epochs)
        tern = {}
        for name, theta in (("random", w.ternary()), ("trained", T)):
            tp = packed_ternary(theta)
            tern[name] = evaluate(L, Xcal, Xte, Yte, k, theta_p=tp)
            del tp
        tern.update({"epoch_loss": [round(v, 5) for v in tt["epoch_loss"]],
                     "train_seconds": round(tt["seconds"], 2),
                     "zero_frac": round(tt["zero_frac"], 4)})
        r["ternary"] = tern
        out[f"k={k}"] = r
        log(f"[bench] predictor training k={k}: {json.dumps(out[f'k={k}'])}")
        del A0, B0, A, B, Ytr, Yte
    del L, Xtr, Xcal, Xte
    torch.cuda.empty_cache()
    return out


def stack_bench(args, steps_tokens=128, warmup_tokens=8, dense_layer_us=None):
    """The 32-layer stack of 7B-shaped predictor layers joined by the residual stream
    (h += y, x = bf16(RMSNorm(h))): per-layer thresholds calibrated at k on 256 seeded
    tokens propagated through the dense stack, then 128 independent decode tokens at
    batch 1, each through all layers. One HIP graph holds the whole timed run."""
    import torch

    from paper_2505_17701_amd import binding as cd
    from workloads import WORKLOADS
    from workloads.synth import T_CALIB, T_EVAL, stream

    w = WORKLOADS["stack32_llama7b_pred"]
    dm, dff, dr, nl = w.d_model, w.d_ff, w.d_rank, w.n_layers
    k = 0.9
    t = time.time()
    layers = []
    for l in range(nl):
        L = dict(w.layer(layer=l))
        L.update(w.predictor(layer=l))
        layers.append({kk: dev_bf16(v) for kk, v in L.items()})
    torch.cuda.synchronize()
    gb = sum(v.numel() * 2 for v in layers[0].values()) * nl / 1e9
    log(f"[bench] stack: {nl} layers of {dm}x{dff} (+ predictor rank {dr}) on device "
        f"({gb:.2f} GB) in {time.time() - t:.1f}s")

    def h0(n, purpose):
        return torch.from_numpy(stream(w.wid, 0, purpose, 77).standard_normal(
            (n, dm)).astype(np.float32)).cuda()

    # calibration on inputs propagated through the dense stack
    ncal, cb = args.calib_tokens, 8
    hc = [h0(ncal, T_CALIB), torch.empty((ncal, dm), dtype=torch.float32, device="cuda")]
    yc = torch.zeros((ncal, dm), dtype=torch.float32, device="cuda")
    xc = torch.empty((ncal, dm), dtype=torch.bfloat16, device="cuda")
    dplan = cd.Plan(dm, dff, max_batch=cb, d_rank=dr)
    thld = []
    for l, L in enumerate(layers):
        src, dst = hc[l % 2], hc[(l + 1) % 2]
        for i in range(0, ncal, cb):
            cd.countdown_ffn_residual(dplan, cd.CD_VARIANT_DENSE, src[i:i + cb],
                                      None if l == 0 else yc[i:i + cb], dst[i:i + cb],
                                      xc[i:i + cb], L["W_gate"], L["W_up"], L["W_down"],
                                      y=yc[i:i + cb])
        th, _ = cd.countdown_calibrate(dplan, cd.CD_VARIANT_DUAL_PRED, xc, k, A_t=L["A_t"],
                                       B_t=L["B_t"])
        thld.append(float(th.item()))
    dplan.close()
    del hc, yc, xc
    log(f"[bench] stack thresholds (k={k}): first {thld[:3]}, last {thld[-1]:.4f}")

    H = h0(steps_tokens + warmup_tokens, T_EVAL)
    hb = [torch.empty((1, dm), dtype=torch.float32, device="cuda") for _ in range(2)]
    xb = torch.empty((1, dm), dtype=torch.bfloat16, device="cuda")
    yb = torch.empty((1, dm), dtype=torch.float32, device="cuda")
    plan = cd.Plan(dm, dff, max_batch=1, d_rank=dr)
    n_arr = torch.zeros(nl, dtype=torch.int32, device="cuda")
    lib = cd.load_library()

    def token(i, variant, record=False):
        for l, L in enumerate(layers):
            src = H[i:i + 1] if l == 0 else hb[(l + 1) % 2]
            cd.countdown_ffn_residual(plan, variant, src, None if l == 0 else yb, hb[l % 2], xb,
                                      L["W_gate"], L["W_up"], L["W_down"], thld[l],
                                      A_t=L["A_t"] if variant == cd.CD_VARIANT_DUAL_PRED else None,
                                      B_t=L["B_t"] if variant == cd.CD_VARIANT_DUAL_PRED else None,
                                      y=yb)
            if record:
                lib.countdown_export_active(plan.handle, None, n_arr[l:l + 1].data_ptr(), None,
                                            None, torch.cuda.current_stream().cuda_stream)

    res = {}
    for name, variant in (("dual_pred", cd.CD_VARIANT_DUAL_PRED), ("dense", cd.CD_VARIANT_DENSE)):
        ntok = steps_tokens if name == "dual_pred" else max(16, steps_tokens // 8)
        for i in range(warmup_tokens):
            token(steps_tokens + i, variant)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(ntok):
                token(i, variant)
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        del g
        res[name] = {"tokens": ntok, "ms_total": ms, "tokens_per_s": ntok / (ms * 1e-3),
                     "us_per_token": ms * 1e3 / ntok, "us_per_layer": ms * 1e3 / (ntok * nl)}
    # |IDX| per layer for one token, and the algorithmic bytes of a token
    token(0, cd.CD_VARIANT_DUAL_PRED, record=True)
    torch.cuda.synchronize()
    n = n_arr.cpu().numpy()
    from paper_2505_17701_amd import traffic

    per = [traffic.algorithmic_bytes("dual_pred", dm, dff, int(v), d_rank=dr) for v in n]
    tok_bytes = sum(p["total"] for p in per)
    dense_bytes = nl * traffic.algorithmic_bytes("dense", dm, dff, dff)["total"]
    r = res["dual_pred"]
    r["algorithmic_bytes_per_token"] = tok_bytes
    r["achieved_GBs"] = tok_bytes / (r["us_per_token"] * 1e-6) / 1e9
    r["frac_hbm_peak"] = r["achieved_GBs"] / HBM_PEAK_GBS
    r["n_active_mean"] = float(n.mean())
    r["realised_sparsity"] = float(1 - n.mean() / dff)
    r["speedup_vs_dense"] = res["dense"]["us_per_token"] / r["us_per_token"]
    r["ideal_byte_ratio"] = dense_bytes / tok_bytes
    # the dense stack runs its residual RMSNorm as a kernel of its own, while the
    # predictor path folds it into the latent kernel: the speedup is also given against
    # 32 single dense layers (no residual stream) timed in this run
    if dense_layer_us:
        r["dense_layer_us"] = dense_layer_us
        r["speedup_vs_32_dense_layers"] = nl * dense_layer_us / r["us_per_token"]

    # the coefficient phase alone (k_latent_norm + k_coef_pred of every layer) and the
    # down kernel alone (on the last coefficient call's rows), each as one graph of
    # tokens x layers with the plan's phase selection and one event pair
    def phase_us(phases, ntok):
        cd.countdown_plan_set_phases(plan, phases)
        for i in range(2):
            token(i, cd.CD_VARIANT_DUAL_PRED)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(ntok):
                token(i, cd.CD_VARIANT_DUAL_PRED)
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        del g
        cd.countdown_plan_set_phases(plan, cd.CD_PHASE_ALL)
        return e0.elapsed_time(e1) * 1e3 / (ntok * nl)

    coef_us = phase_us(cd.CD_PHASE_COEF, 32)
    down_us = phase_us(cd.CD_PHASE_DOWN, 32)
    coef_b = float(np.mean([p["coef"] + p["latent"] for p in per]))
    ach = coef_b / (coef_us * 1e-6) / 1e9
    r["coef_phase_us_per_layer"] = coef_us
    r["down_kernel_us_per_layer"] = down_us
    r["roofline"] = {"bound": "hbm", "kernel": "k_latent_norm + k_coef_pred (residual + "
                     "RMSNorm, predictor latent, scores, threshold, W_gate / W_up gather, s)",
                     "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": ach / HBM_PEAK_GBS, "traffic": None, "bytes_per_launch": coef_b,
                     "avg_launch_us": coef_us}
    plan.close()
    del layers
    torch.cuda.empty_cache()
    log(f"[bench] stack: {json.dumps(res)}")
    return {"workload": w.name, "layers": nl, "k": k, "batch": 1,
            "thld_first_last": [thld[0], thld[-1]], **res}


def cpu_baseline(args, w, host0, X_eval_h, thld):
    """The fp64 oracle on the host cores, timed on a bounded sample of the headline
    workload (same weights, thresholds and eval tokens), with its dense path on the
    same threads and the same sparse path on one thread beside it."""
    import oracle

    th = np.float32(thld.get((args.variant, args.k), 0.0))
    H = host0
    fns = {"mono": lambda x: oracle.ffn_mono(x, H["W_gate"], H["W_up"], H["W_down"], th),
           "dual_ideal": lambda x: oracle.ffn_dual_ideal(x, H["W_gate"], H["W_up"],
                                                         H["W_down"], th),
           "dual_pred": lambda x: oracle.ffn_dual_pred(x, H["W_gate"], H["W_up"], H["W_down"],
                                                       H.get("A_t"), H.get("B_t"), th),
           "dense": lambda x: oracle.dense(x, H["W_gate"], H["W_up"], H["W_down"]),
           "cats": lambda x: oracle.ffn_cats(x, H["W_gate"], H["W_up"], H["W_down"], th),
           "dual_tern": lambda x: oracle.ffn_dual_tern(x, H["W_gate"], H["W_up"],
                                                       H["W_down"], H.get("theta_t"), th)}
    for vb in ("mono", "dual_ideal", "dual_pred", "cats", "dual_tern"):
        fns[vb + "_topk"] = (lambda b: lambda x: oracle.ffn_topk(
            b, x, H["W_gate"], H["W_up"], H["W_down"], args.k, A_t=H.get("A_t"),
            B_t=H.get("B_t"), theta_t=H.get("theta_t")))(vb)
    fn = fns[args.variant]
    nt = len(X_eval_h) - args.batch + 1

    def rate(f, secs):
        n, t = 0, time.perf_counter()
        while n < 2 or time.perf_counter() - t < secs:
            f(X_eval_h[n % nt:n % nt + args.batch])
            n += 1
        return n, time.perf_counter() - t

    n_done, el = rate(fn, args.cpu_seconds)
    cpu = {"value": n_done * args.batch / el, "unit": "tokens/s",
           "cores": oracle.num_threads(), "kind": "oracle",
           "sample": f"{n_done} calls of {w.name} {args.variant} k={args.k}, "
                     f"batch {args.batch}, one weight copy, fp64 C oracle ({el:.1f} s)"}
    secs = max(1.0, args.cpu_seconds / 4)
    n, el = rate(fns["dense"], secs)
    cpu["detail"] = {"dense_tokens_per_s": n * args.batch / el}
    nthreads = oracle.num_threads()
    oracle.set_num_threads(1)
    n, el = rate(fn, secs)
    cpu["detail"]["one_thread_tokens_per_s"] = n * args.batch / el
    oracle.set_num_threads(nthreads)
    log(f"[bench] cpu baseline: {json.dumps(cpu)}")
    return cpu


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the sparse FFN layer "
              "runs and is timed on a single MI355X; sharding it across GPUs is not "
              "implemented.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2505_17701_amd import binding as cd
    from workloads import WORKLOADS

    cd.load_library()
    if not torch.cuda.is_available():
        sys.exit("bench.py needs a GPU")
    torch.cuda.set_device(0)
    w = WORKLOADS[args.workload]
    dm, dff = w.d_model, w.d_ff
    copies = args.copies or auto_copies(w)
    if args.traffic_probe:
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")  # 256 MiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    base = args.variant[:-5] if args.variant.endswith("_topk") else args.variant
    main_variants = (["mono", "dual_ideal", "cats"] if "mono" in w.variants
                     else [v for v in w.variants if v != "dense"])
    if w.name == "llama70b_8192x28672":
        main_variants = ["mono"]
    if base == "dual_tern":
        main_variants.append("dual_tern")
    main_ctx = Context(w, copies, args.tokens, args.calib_tokens,
                       sorted(set((args.k,) + tuple(w.ks))), max_batch=args.batch,
                       variants=main_variants)
    main_res = main_ctx.measure(args.variant, args.k, args.batch, args.steps, args.warmup,
                                replays=True)
    log(f"[bench] {w.name} {args.variant} k={args.k}: {json.dumps(main_res)}")
    ceiling = stream_ceiling(main_ctx, min(max(args.steps, 64), 512))
    log(f"[bench] plain streaming read: {json.dumps(ceiling)}")

    extra = {}
    if not args.no_extra:
        extra, _ = workload_lines(main_ctx, args, (args.variant, args.k))
        if "dense" in extra:
            from paper_2505_17701_amd import traffic

            extra["speedup_vs_dense"] = extra["dense"]["us_per_layer"] / main_res["us_per_layer"]
            extra["ideal_byte_ratio"] = (traffic.algorithmic_bytes("dense", dm, dff, dff)["total"]
                                         / main_res["algorithmic_bytes"])
    host0, X_eval_h = main_ctx.host0, main_ctx.X_eval_h
    thld, thld_pooled = main_ctx.thld, main_ctx.thld_pooled
    main_ctx.free()

    others = {}
    if not args.no_extra and not args.no_other:
        seven_dense_us = None
        for name in ("llama7b_4096x11008", "llama70b_8192x28672"):
            if name != w.name and not (args.no_7b and name == "llama7b_4096x11008"):
                others[name] = layer_block(args, name)
        if "llama7b_4096x11008" in others:
            seven_dense_us = others["llama7b_4096x11008"].get("dense", {}).get("us_per_layer")
        elif w.name == "llama7b_4096x11008":
            seven_dense_us = extra.get("dense", {}).get("us_per_layer")
        if not args.no_8b:
            others["llama3_8b_4096x14336_pred"] = eight_b_block(args)
        if not args.no_stack:
            others["stack32_llama7b_pred"] = stack_bench(args, dense_layer_us=seven_dense_us)
        if not args.no_train:
            others["predictor_training_llama3_8b"] = predictor_training_bench(args)

    cpu = cpu_baseline(args, w, host0, X_eval_h, thld) if args.cpu_seconds > 0 else None
    roof = roofline(main_res, args.variant, (w.name, args.variant, args.k, args.batch), ceiling)

    out = {
        "metric": "sparse-FFN decode tokens/s and \u00b5s/layer; achieved HBM GB/s vs peak at 90% "
                  "sparsity",
        "metric_detail": f"one FFN layer, batch {args.batch}, k={args.k}",
        "value": main_res["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_res["ms_per_step"],
        "us_per_layer": main_res["us_per_layer"],
        "us_per_layer_eager": main_res["us_per_layer_eager"],
        "us_per_layer_median_of_6": main_res["us_per_layer_median_of_6"],
        "us_per_layer_mean_of_6": main_res["us_per_layer_mean_of_6"],
        "launch": "one HIP graph of exactly `steps` layer calls, replayed once (timed)",
        "achieved_GBs": main_res["achieved_GBs"],
        "frac_hbm_peak": main_res["frac_hbm_peak"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "accumulate": "fp32",
        "data": f"synthetic (seeded N(0, {w.sigma}^2) bf16 weights, N(0,1) tokens"
                + (f" with {w.outlier_frac:.0%} outlier channels x20)" if w.outlier_frac else ")"),
        "config": {"workload": w.name, "d_model": dm, "d_ff": dff, "batch": args.batch,
                   "variant": args.variant, "k": args.k,
                   "thld": thld.get((args.variant, args.k)),
                   "thld_pooled_reading": thld_pooled.get((base, args.k)),
                   "weight_copies": copies,
                   "n_active_mean": main_res["n_active_mean"],
                   "realised_sparsity": main_res["realised_sparsity"],
                   "algorithmic_bytes_per_step": main_res["algorithmic_bytes"],
                   "parallelism": "single GPU"},
        "kernels": {**{k: main_res.get(k) for k in ("coef_kernel_us", "coef_kernel_GBs",
                                                     "down_kernel_us", "down_kernel_GBs")
                       if main_res.get(k) is not None},
                    **({"phases_note": "each phase timed alone (coefficient phase with its "
                                       "select, then k_down); a whole one-token call fuses "
                                       "the select into the down launch (k_topk_down1)"}
                       if args.variant == "dual_ideal_topk" and args.batch == 1 else {})},
        "roofline_traffic_source": "profiles/ PMC summary of the same kernel source (FETCH_SIZE "
                                   "+ WRITE_SIZE scaled by a 256 MiB copy), null when absent "
                                   "or stale; not read in this run",
        "variants": extra,
        "other_workloads": others,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
