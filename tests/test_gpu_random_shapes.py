"""Seeded random configurations of the FFN calls through the C ABI against the
oracle: variant, constant or per-token threshold, ragged d_model and d_ff,
batch 1-8 and k, all drawn from one fixed generator, so every run checks the
same cases. They complement the hand-picked shapes of the other parity tests
with combinations nobody chose (the one-launch per-token kernel at odd slice
sizes, ragged token tiles, batch tiles of every width)."""
import numpy as np
import pytest

import oracle
from test_gpu_parity import Layer, compare, plan_for
from test_gpu_topk import check_topk
from workloads import make_layer, make_predictor, make_ternary, make_tokens

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

VARIANTS = ["mono", "dual_ideal", "dual_pred", "cats", "dual_tern"]


def cases(n=30, n_wide=18, seed=2405):
    """n cases with d_model <= 2048 at 1-8 tokens, then n_wide with rows of
    4104-8192 columns (16 loads per lane and row) at 1-4 tokens, the most a
    plan takes at that width."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n + n_wide):
        wide = i >= n
        dm = 8 * int(rng.integers(513, 1025) if wide else rng.integers(1, 257))
        dff = 8 * int(rng.integers(1, 1025) if wide else rng.integers(1, 513))
        B = int(rng.integers(1, 5 if wide else 9))
        out.append((i, VARIANTS[i % len(VARIANTS)], bool(rng.integers(2)), dm, dff, B,
                    round(float(rng.uniform(0.3, 0.95)), 3)))
    return out


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("case", cases(),
                         ids=lambda c: f"{c[0]}-{c[1]}-{'topk' if c[2] else 'thld'}-"
                                       f"{c[3]}x{c[4]}-B{c[5]}")
def test_random_configuration(case):
    i, variant, topk, dm, dff, B, k = case
    wid = 3000 + i
    L = make_layer(wid, dm, dff, 0.05)
    P = make_predictor(wid, dm, 16, dff, 0.05) if variant == "dual_pred" else None
    T = make_ternary(wid, dm, dff) if variant == "dual_tern" else None
    layer = Layer(L, P, T)
    x = make_tokens(wid, B, dm)
    label = f"random {case}"
    if topk:
        n, flips, rel = check_topk(variant, layer, x, k, label)
    else:
        if variant == "dual_pred":
            c = oracle.predictor(x, P["A_t"], P["B_t"])[1]
        elif variant == "dual_tern":
            c = oracle.ternary_predictor(x, T)
        else:
            u, g, s = oracle.coefficients(x, L["W_gate"], L["W_up"])
            c = np.abs({"mono": u, "dual_ideal": s, "cats": g / (1.0 + np.exp(-g))}[variant])
        thld = float(np.float32(np.quantile(c, k)))
        plan = plan_for(layer, max_batch=B)
        n, flips, rel = compare(plan, variant, layer, x, thld, label)
        plan.close()
    print(f"{label}: n={n} flips={flips} rel={rel:.2e}", flush=True)
