"""Memory model (Section 3.3) and cost model (Appendix B) against the paper's
own numbers: the worked example of Appendix B.4 (tests/golden) and the rank
r = 204 the paper uses for eta = 0.2 at D' = 1024."""

import json
import os

import numpy as np
import pytest

from oracle import cost, decode

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "appB4_worked_example.json")))


def test_appendix_b4_coefficients():
    g = GOLD
    r, rho, Dp, W = g["inputs"]["r"], g["inputs"]["rho"], g["inputs"]["Dp"], g["inputs"]["W"]
    assert cost.full_rec_coeff(r, Dp, 0) == g["full_rec_base"]
    assert cost.s4r_coeff(r, Dp, 1, W, 0.0) - cost.s4r_coeff(r, Dp, 0, W, 0.0) == g["latent_scoring_per_G"]
    assert cost.s4r_coeff(r, Dp, 0, W, rho) == pytest.approx(g["sparse_reconstruction"])
    per_G = cost.s4r_coeff(r, Dp, 1, W, rho) - cost.s4r_coeff(r, Dp, 0, W, rho)
    assert per_G == pytest.approx(g["latent_scoring_per_G"] + g["sparse_attention_per_G"])
    assert round(per_G) == g["s4r_per_G_rounded"]


@pytest.mark.parametrize("G,key", [(1, "G1"), (4, "G4")])
def test_appendix_b4_ratios(G, key):
    r, rho, Dp, W = (GOLD["inputs"][k] for k in ("r", "rho", "Dp", "W"))
    s4r = cost.s4r_coeff(r, Dp, G, W, rho)
    full = cost.full_rec_coeff(r, Dp, G)
    assert round(s4r) == GOLD[key]["s4r"]
    assert full == GOLD[key]["full"]
    assert round(s4r / full, 3) == GOLD[key]["ratio"]
    lo, hi = GOLD["speedup_range"]
    assert lo <= full / s4r <= hi + 0.01
    assert cost.s4r_beneficial(r, Dp, G, W, rho)


def test_rank_for_eta_matches_paper_rank():
    # r solves Eq. memory_ratio for eta; as L grows it tends to eta * D'
    Dp, eta = 1024, 0.2
    r_inf = cost.rank_for_ratio(eta, 10 ** 12, 4, Dp, 4, 4)
    assert r_inf == pytest.approx(eta * Dp, rel=1e-6)
    assert int(np.floor(eta * Dp)) == GOLD["inputs"]["r"]
    r120k = cost.rank_for_ratio(eta, 120_000, 4, Dp, 4, 4)
    assert 203 <= r120k <= 205
    # plugging the solution back gives the target ratio
    assert cost.mem_ratio(120_000, 4, Dp, r120k, 4, 4) == pytest.approx(eta, rel=1e-12)


def test_memory_model_consistency():
    for L, s, Dp, r, G, W in [(1000, 4, 1024, 160, 4, 32), (131068, 4, 512, 96, 7, 64), (10, 0, 64, 8, 1, 1)]:
        assert cost.mem_s4r(L, s, Dp, r, G, W) / cost.mem_full(L, s, Dp) == pytest.approx(
            cost.mem_ratio(L, s, Dp, r, G, W), rel=1e-12)
    # long-context limit: ratio -> r / D'
    assert cost.mem_ratio(10 ** 9, 4, 1024, 160, 4, 32) == pytest.approx(160 / 1024, rel=1e-5)


def test_budget_formulas():
    for L in (1, 10, 100, 4092, 131068):
        for W in (0, 4, 32, 128):
            for rho in (0.0, 0.05, 0.2, 1.0):
                k = cost.k_from_rho(L, W, rho)
                assert k == max(int(np.floor(rho * L)) - W, 0)
                assert cost.m_from_rho(L, W, rho) == max(W, int(np.floor(rho * L)))
                if L >= W:
                    assert decode.num_selected(L, W, k) == cost.m_from_rho(L, W, rho)
