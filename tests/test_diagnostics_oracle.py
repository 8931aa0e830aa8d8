"""Pins of the loss-allocation diagnostics oracle (Sec. 4.4 s_t and Table 1;
Sec. 7.2 Table 3; Sec. 4.2 G_t) against hand-derived values, closed forms of
the trajectory- and turn-level objectives, and brute-force group-bys."""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pandas as pd
import pytest

from oracle import diagnostics as D
from oracle import turnkl_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _stats(n_traj, kl_mean, loss_mass, n_tokens=None):
    st = np.zeros(len(n_traj), O.STAT_DTYPE)
    st["n_traj"] = n_traj
    st["kl_mean"] = kl_mean
    st["loss_mass"] = loss_mass
    st["n_tokens"] = n_tokens if n_tokens is not None else np.asarray(n_traj) * 3
    return st


def test_worked_example():
    g = _load("budget_diagnostics_example.json")
    st = _stats(**g["stats"])
    np.testing.assert_allclose(D.loss_share(st), [float(Fraction(x)) for x in g["loss_share"]],
                               rtol=1e-15)
    for c in g["cases"]:
        r = D.budget_report(st, g["n_traj_batch"], c["floor"], c["frac"])
        assert (r.n_min, r.prefix, r.third) == (c["n_min"], c["prefix"], c["third"])
        for k in ("shallow_budget", "deep_budget", "deep_support"):
            assert abs(getattr(r, k) - float(Fraction(c[k]))) < 1e-15, k
        if c["deep_shallow_kl"] is None:
            assert math.isnan(r.deep_shallow_kl)
        else:
            assert abs(r.deep_shallow_kl - float(Fraction(c["deep_shallow_kl"]))) < 1e-15


def _full_depth_batch(B, T, rng, const_kl=0.7):
    """B trajectories that all reach turns 0..T-1, random supervised counts,
    every supervised token with the same KL."""
    traj, turn, mask = [], [], []
    for b in range(B):
        for t in range(T):
            n = int(rng.integers(1, 9))
            traj += [b] * (n + 1)
            turn += [t] * (n + 1)
            mask += [0] + [1] * n
    traj, turn, mask = (np.array(traj, np.int32), np.array(turn, np.int32),
                        np.array(mask, np.uint8))
    kl = np.where(mask == 1, const_kl, 0.0)
    return traj, turn, mask, kl


@pytest.mark.parametrize("T", [3, 7, 9, 12])
def test_hard_turn_level_spends_a_third_on_the_deep_third(T):
    """alpha = 1 with every trajectory at full depth and constant KL: s_t = 1/T,
    so the deep third gets ceil(T/3)/T (about a third, as the hard switch of
    Table 3 does); alpha = 0: s_t = mean over trajectories of n_bt / N_b."""
    rng = np.random.default_rng(T)
    B = 11
    traj, turn, mask, kl = _full_depth_batch(B, T, rng)
    seg = O.segments(traj, turn, mask, T)
    w1 = O.token_weights(seg, len(traj), mask, 1.0)
    st1 = O.turn_stats([(seg, mask, kl, w1)], T)
    np.testing.assert_allclose(D.loss_share(st1), np.full(T, 1.0 / T), rtol=1e-12)
    r = D.budget_report(st1, B, 8, 0.15)
    k = -(-T // 3)
    assert r.prefix == T and r.third == k
    assert abs(r.deep_budget - k / T) < 1e-12 and abs(r.shallow_budget - k / T) < 1e-12
    assert r.deep_support == 1.0 and abs(r.deep_shallow_kl - 1.0) < 1e-15
    w0 = O.token_weights(seg, len(traj), mask, 0.0)
    st0 = O.turn_stats([(seg, mask, kl, w0)], T)
    df = pd.DataFrame({"traj": traj, "turn": turn})[mask == 1]
    n_bt = df.groupby(["traj", "turn"]).size().unstack(fill_value=0).to_numpy(np.float64)
    want = (n_bt / n_bt.sum(axis=1, keepdims=True)).mean(axis=0)
    np.testing.assert_allclose(D.loss_share(st0), want, rtol=1e-12)


@pytest.mark.parametrize("seed", range(5))
def test_loss_share_matches_group_by_of_the_weighted_kl(seed):
    rng = np.random.default_rng(1000 + seed)
    traj, turn, mask = [], [], []
    for b in range(9):
        for t in range(int(rng.integers(1, 8))):
            n = int(rng.integers(1, 6))
            traj += [b] * n
            turn += [t] * n
            mask += [int(v) for v in rng.integers(0, 2, n)]
    traj, turn, mask = np.array(traj, np.int32), np.array(turn, np.int32), np.array(mask, np.uint8)
    seg = O.segments(traj, turn, mask, 8)
    kl = rng.gamma(2.0, 0.4, len(traj))
    w = O.token_weights(seg, len(traj), mask, 0.3, 2, 0.2)
    st = O.turn_stats([(seg, mask, kl, w)], 8)
    s = D.loss_share(st)
    df = pd.DataFrame({"turn": turn, "m": w * kl})[mask == 1]
    want = df.groupby("turn")["m"].sum().reindex(range(8), fill_value=0.0).to_numpy()
    np.testing.assert_allclose(s, want / want.sum(), rtol=1e-12, atol=1e-16)
    assert abs(s.sum() - 1.0) < 1e-12


def test_prefix_stops_at_the_first_unsupported_turn():
    st = _stats([20, 5, 12, 12], [1, 1, 1, 1], [1, 1, 1, 1])
    r = D.budget_report(st, 20, 8, 0.0)
    assert r.prefix == 1 and r.third == 1
    assert r.shallow_budget == r.deep_budget == 0.25
    # an empty turn ends the prefix even when n_min is 0
    st = _stats([4, 0, 3], [1, 0, 1], [1, 0, 1])
    assert D.budget_report(st, 4, 0, 0.0).prefix == 1
    # no loss mass: every share is 0
    assert not D.loss_share(_stats([3, 2], [0, 0], [0, 0])).any()


def test_outcome_gap_of_the_worked_example():
    ex = _load("support_floor_outcome_example.json")
    tok = ex["tokens"]
    traj = np.array(tok["traj_id"], np.int32)
    turn = np.array(tok["turn_id"], np.int32)
    mask = np.array(tok["loss_mask"], np.uint8)
    succ = np.array(tok["success"], np.uint8)
    seg = O.segments(traj, turn, mask, ex["max_turns"], succ)
    kl = np.arange(len(traj)) / 10.0
    w = O.token_weights(seg, len(traj), mask, 0.5)
    gap = D.outcome_gap(O.outcome_split(seg, mask, kl, w, ex["max_turns"]))
    for t, want in enumerate(ex["outcome"]["gap_fail_minus_succ"]):
        if want is None:
            assert math.isnan(gap[t])
        else:
            assert abs(gap[t] - float(Fraction(want))) < 1e-14


def test_pins_catch_planted_mistakes():
    g = _load("budget_diagnostics_example.json")
    st = _stats(**g["stats"])
    c = g["cases"][0]
    s = D.loss_share(st)
    # (1) floor(P / 3) instead of the ceiling: a deep third of one turn
    assert abs(s[4] - float(Fraction(c["deep_budget"]))) > 1e-3
    # (2) valid turns instead of the prefix: the [20, 5, 12, 12] case has 3 valid turns, P = 1
    assert sum(n >= 8 for n in [20, 5, 12, 12]) != 1
    # (3) pooled-token KL means instead of per-turn means change the ratio
    n_tok = np.array([60, 54, 45, 33, 27])
    kl = np.array(g["stats"]["kl_mean"][:5])
    pooled = (n_tok[3:] * kl[3:]).sum() / n_tok[3:].sum() / ((n_tok[:2] * kl[:2]).sum() / n_tok[:2].sum())
    assert abs(pooled - float(Fraction(c["deep_shallow_kl"]))) > 1e-3
    # (4) support relative to the batch size instead of n_0 differs when n_0 < n_traj
    r = D.budget_report(st, 40, 8, 0.15)
    assert abs(r.deep_support - (11 / 40 + 9 / 40) / 2) > 1e-3
