"""The FLOP / byte counters against the paper's Table 3 and against hand counts."""
import json
import os

import numpy as np
import pytest

from paper_2505_17701_amd import traffic

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_table3.json")))


@pytest.mark.parametrize("row", GOLD["rows"], ids=lambda r: f"{r['method']}-k{r['k']}")
def test_paper_table3_reproduced(row):
    dm, di, dr, ca = GOLD["d_model"], GOLD["d_inter"], GOLD["d_rank"], GOLD["c_act"]
    f = traffic.paper_flops(row["method"], dm, di, row["k"], dr, ca) / 1e6
    m = traffic.paper_mem_elements(row["method"], dm, di, row["k"], dr) / 2 ** 20
    assert round(f, 2) == pytest.approx(row["flops_m"], abs=1e-9)
    assert round(m, 3) == pytest.approx(row["mem"], abs=1e-9)


def test_dual_pred_memory_slip_is_one_term():
    """The Table 10 sum exceeds Table 3's D-CountDown entries by exactly d_inter - 2 s."""
    dm, di, dr = GOLD["d_model"], GOLD["d_inter"], GOLD["d_rank"]
    for k in (0.7, 0.8, 0.9):
        s = traffic.paper_active(di, k)
        full = traffic.paper_mem_elements("dual_pred", dm, di, k, dr, tabulated=False)
        tab = traffic.paper_mem_elements("dual_pred", dm, di, k, dr, tabulated=True)
        assert full - tab == di - 2 * s


def test_active_count_reading():
    assert traffic.paper_active(14336, 0.7) == 4300
    assert traffic.paper_active(14336, 0.9) == 1433
    assert traffic.paper_active(11008, 0.9) == 1100


def test_algorithmic_bytes_hand_counts():
    dm, dff, n = 4096, 11008, 1101
    b = traffic.algorithmic_bytes("mono", dm, dff, n)
    assert b["coef"] == 2 * dm * dff + 2 * dm * n + 2 * dm
    assert b["down"] == 2 * dm * n + 4 * dm
    assert b["total"] == b["coef"] + b["down"]
    assert abs(b["total"] / 1e6 - 108.2) < 0.1          # 7B-shaped layer, k = 0.9
    d = traffic.algorithmic_bytes("dense", dm, dff, dff)
    assert d["total"] == 6 * dm * dff + 6 * dm
    p = traffic.algorithmic_bytes("dual_pred", 4096, 14336, 1434, B=1, d_rank=256)
    assert abs(p["total"] / 1e6 - 44.7) < 0.2
    assert traffic.algorithmic_flops("dense", dm, dff, dff) == 6 * dm * dff


def test_cif_caf_closed_form():
    """Masks small enough to count by hand (sparsity-analysis metrics of Sec. 6)."""
    from paper_2505_17701_amd.metrics import cif_caf

    S = [[1, 1, 1, 0, 0, 0]]
    U = [[1, 0, 1, 1, 0, 0]]
    H = [[0, 1, 0, 1, 1, 0]]
    m = cif_caf(S, U, H)
    # alive: S = {0,1,2}; ~H there = {0,2}; of those U keeps {0,2}
    assert m["CIF(u,alive)"] == 2 / 3 and m["CAF(u,alive)"] == 2 / 3
    # h: ~U on S = {1}; H keeps 1
    assert m["CIF(h,alive)"] == 1 / 3 and m["CAF(h,alive)"] == 1 / 3
    # dead: ~S = {3,4,5}; H there = {3,4}; ~U of those = {4}
    assert m["CIF(u,dead)"] == 2 / 3 and m["CAF(u,dead)"] == 1 / 3
    # h dead: U on ~S = {3}; ~H of those = {} -> 0
    assert m["CIF(h,dead)"] == 1 / 3 and m["CAF(h,dead)"] == 0.0


def test_cif_caf_pools_tokens():
    from paper_2505_17701_amd.metrics import cif_caf

    rng = np.random.default_rng(0)
    S, U, H = (rng.random((5, 40)) < 0.3 for _ in range(3))
    pooled = cif_caf(S, U, H)
    assert pooled["CIF(u,alive)"] == (S & ~H).sum() / S.sum()
    # u and h exchange roles exactly
    swapped = cif_caf(S, H, U)
    assert swapped["CIF(u,alive)"] == pooled["CIF(h,alive)"]
    assert swapped["CAF(h,dead)"] == pooled["CAF(u,dead)"]


def test_f1_score_by_hand():
    from paper_2505_17701_amd.predictor import f1_score

    # tp 1, fp 1, fn 1 -> 2/(2+1+1)
    assert f1_score([1, 1, 0, 0], [1, 0, 1, 0]) == 0.5
    assert f1_score([1, 1, 0], [1, 1, 0]) == 1.0
    assert f1_score([0, 0, 1], [1, 1, 0]) == 0.0
    # pooled over tokens, not averaged per token
    assert f1_score([[1, 0], [1, 1]], [[1, 0], [0, 0]]) == 2 * 1 / (2 * 1 + 2 + 0)
    assert f1_score([[0, 0]], [[0, 0]]) == 1.0
