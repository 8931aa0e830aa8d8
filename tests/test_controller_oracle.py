"""Pins of the depth-controller oracle (Sec. 5.1, App. D Algorithm 1) against
facts it does not compute itself: a hand-derived worked example, closed
forms, a library quantile, and planted mistakes."""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import depth_controller as D

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "depth_controller_example.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def test_worked_example_matches_hand_derivation():
    g = _golden()
    cfg = D.Config()
    pb = g["probe_batch"]
    centroid = D.efficiency_centroid(cfg, pb["kl_mean"], pb["n_traj"])
    num, den = g["centroid_fraction"]
    assert abs(centroid - num / den) < 1e-12
    assert D.round_half_even(centroid) == g["h_eff"]
    assert D.coverage_floor(cfg, pb["success_lengths"]) == g["h_cov"]
    st = D.update(cfg, D.init(cfg), pb["kl_mean"], pb["n_traj"], pb["success_lengths"])
    assert (st.h_eff, st.h_cov, st.h_ctrl) == (g["h_eff"], g["h_cov"], g["h_ctrl"])
    out = D.run(cfg, lambda k: (pb["kl_mean"], pb["n_traj"], pb["success_lengths"]),
                len(g["steps"]))
    for (k, h_cap, probe, h_roll, s), ref in zip(out, g["steps"]):
        assert (k, h_cap, probe, h_roll) == (ref["k"], ref["cap"], ref["probe"], ref["roll"])
        assert abs(s.h_bar - ref["h_bar"]) < 1e-9, (k, s.h_bar, ref["h_bar"])


def test_all_mass_on_one_turn_puts_the_centroid_there():
    cfg = D.Config()
    for t_star in (0, 1, 7, 29):
        K = [0.0] * 30
        K[t_star] = 0.37
        n = list(range(40, 10, -1))
        c = D.efficiency_centroid(cfg, K, n)
        assert abs(c - t_star) < 1e-9
        assert D.round_half_even(c) == t_star


def test_uniform_mass_centroid_is_the_mean_index():
    cfg = D.Config()
    for T in (1, 2, 5, 12):
        c = D.efficiency_centroid(cfg, [0.25] * T, [9] * T)
        assert abs(c - (T - 1) / 2.0) < 1e-9


def test_negative_kl_carries_no_mass_and_survivors_weight_it():
    cfg = D.Config()
    # a negative K_t counts as zero
    a = D.efficiency_centroid(cfg, [0.5, -0.3, 0.5], [4, 4, 4])
    b = D.efficiency_centroid(cfg, [0.5, 0.0, 0.5], [4, 4, 4])
    assert a == b == pytest.approx(1.0)
    # survivors thin out -> the centroid moves shallower, by the exact ratio
    c = D.efficiency_centroid(cfg, [1.0, 1.0], [4, 1])
    assert abs(c - Fraction(1, 4) / Fraction(5, 4)) < 1e-12
    # no trajectory supervised at turn 0
    assert D.efficiency_centroid(cfg, [1.0, 1.0], [0, 3]) == 0.0


@pytest.mark.parametrize("p", [0.4, 0.6, 0.8, 1.0])
def test_coverage_floor_is_the_inverted_cdf_quantile_minus_one(p):
    cfg = D.Config(coverage_quantile=p)
    rng = np.random.default_rng(5)
    for _ in range(50):
        L = rng.integers(1, 40, size=int(rng.integers(1, 60)))
        want = int(np.quantile(L, p, method="inverted_cdf")) - 1
        assert D.coverage_floor(cfg, list(L)) == want


def test_ema_closed_form_and_cap_clipping():
    cfg = D.Config()
    st = D.init(cfg)
    c = 6
    K = [0.0] * 10
    K[c] = 1.0
    for n in range(1, 30):
        st = D.update(cfg, st, K, [5] * 10, [])
        want = c + (cfg.h_max - c) * (1.0 - cfg.ema_alpha) ** n
        assert abs(st.h_bar - want) < 1e-9
    assert D.cap(cfg, st) == c + 1
    assert D.cap(cfg, D.State(h_bar=0.0)) == cfg.h_min
    assert D.cap(cfg, D.State(h_bar=400.0)) == cfg.h_max
    assert D.cap(cfg, D.State(h_bar=-3.0)) == cfg.h_min


def test_probe_schedule():
    cfg = D.Config()
    probes = [k for k in range(1, 101) if D.is_probe(cfg, k)]
    assert probes == [1, 2, 3] + list(range(8, 101, 8))
    st = D.init(cfg)
    for k in range(1, 20):
        h_cap, probe, h_roll = D.plan(cfg, st, k)
        assert h_roll == (cfg.h_max if probe else h_cap)


def test_coverage_needs_enough_successes():
    cfg = D.Config()
    st = D.init(cfg)
    st = D.update(cfg, st, [1.0, 0.0], [3, 3], [5] * 7)  # 7 < 8: H_cov stays 0
    assert st.h_cov == 0 and st.h_ctrl == 0
    st = D.update(cfg, st, [1.0, 0.0], [3, 3], [5] * 8)
    assert st.h_cov == 4 and st.h_ctrl == 4
    st = D.update(cfg, st, [1.0, 0.0], [3, 3], [2] * 3)  # too few again: keep 4
    assert st.h_cov == 4


def test_round_half_even_reading():
    assert [D.round_half_even(x) for x in (0.5, 1.5, 2.5, 2.49999, 2.50001, 3.5, -0.5)] == \
        [0, 2, 2, 2, 3, 4, 0]
    for x in np.linspace(-5, 5, 101):
        assert D.round_half_even(float(x)) == round(float(x))


def test_pins_catch_planted_mistakes():
    g = _golden()
    pb = g["probe_batch"]
    cfg = D.Config()
    n = pb["n_traj"]
    K = pb["kl_mean"]
    # (1) 1-based turn index in the centroid
    m = [max(k, 0) * nt / n[0] for k, nt in zip(K, n)]
    one_based = sum((t + 1) * mt for t, mt in enumerate(m)) / sum(m)
    assert round(one_based) != g["h_eff"]
    # (2) survivors ignored (m_t = [K_t]_+)
    m2 = [max(k, 0) for k in K]
    no_surv = sum(t * mt for t, mt in enumerate(m2)) / sum(m2)
    assert abs(no_surv - Fraction(*g["centroid_fraction"])) > 1e-3
    # (3) coverage on lengths rather than last indices (off by one)
    L = np.array(pb["success_lengths"])
    assert int(np.quantile(L, 0.8, method="inverted_cdf")) != g["h_cov"]
    # (4) EMA weights swapped
    swapped = cfg.ema_alpha * cfg.h_max + (1 - cfg.ema_alpha) * g["h_ctrl"]
    assert abs(swapped - g["steps"][0]["h_bar"]) > 1
    # (5) no +1 in the cap
    assert D.round_half_even(g["steps"][1]["h_bar"]) != g["steps"][2]["cap"]
