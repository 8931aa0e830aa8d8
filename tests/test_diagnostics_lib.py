"""The library's host diagnostics (turnkl_loss_share, turnkl_budget_report,
turnkl_outcome_gap) against the diagnostics oracle: the hand-derived example
and random per-turn statistics, plus argument errors.  Host code: no GPU."""
import ctypes
import json
import math
import os

import numpy as np
import pytest

from oracle import diagnostics as D
from oracle import turnkl_oracle as O
from paper_2607_05804_amd import turnkl as T

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _random_stats(rng, n_turns):
    st = np.zeros(n_turns, O.STAT_DTYPE)
    surv = np.sort(rng.integers(0, 40, n_turns))[::-1]
    st["n_traj"] = surv
    st["n_tokens"] = surv * rng.integers(1, 30, n_turns)
    st["kl_mean"] = np.where(surv > 0, rng.gamma(2.0, 0.3, n_turns), 0.0)
    st["loss_mass"] = np.where(surv > 0, rng.uniform(0, 0.1, n_turns), 0.0)
    return st


def _same(a, b):
    return (math.isnan(a) and math.isnan(b)) or a == b


def test_worked_example_matches_the_oracle():
    g = json.load(open(os.path.join(GOLDEN, "budget_diagnostics_example.json")))
    st = np.zeros(len(g["stats"]["n_traj"]), O.STAT_DTYPE)
    for k, v in g["stats"].items():
        st[k] = v
    np.testing.assert_array_equal(T.loss_share(st), D.loss_share(st))
    for c in g["cases"]:
        got = T.budget_report(st, g["n_traj_batch"], c["floor"], c["frac"])
        want = D.budget_report(st, g["n_traj_batch"], c["floor"], c["frac"])
        for k in ("n_min", "prefix", "third", "shallow_budget", "deep_budget", "deep_support",
                  "deep_shallow_kl"):
            assert _same(got[k], getattr(want, k)), (c, k, got[k], getattr(want, k))


@pytest.mark.parametrize("seed", range(20))
def test_random_statistics_bit_identical_to_the_oracle(seed):
    rng = np.random.default_rng(1100 + seed)
    n_turns = int(rng.integers(1, 80))
    st = _random_stats(rng, n_turns)
    np.testing.assert_array_equal(T.loss_share(st), D.loss_share(st))
    n_traj = int(st["n_traj"][0]) + int(rng.integers(0, 5))
    for floor, frac in ((8, 0.15), (8, 0.10), (0, 0.0), (3, 0.5), (1, 1.0)):
        got = T.budget_report(st, n_traj, floor, frac)
        want = D.budget_report(st, n_traj, floor, frac)
        for k, v in dataclasses_items(want):
            assert _same(float(got[k]), float(v)), (seed, floor, frac, k)
    ost = np.concatenate([_random_stats(rng, n_turns), _random_stats(rng, n_turns)])
    ost["n_tokens"][rng.integers(0, 2 * n_turns, 3)] = 0
    g = T.outcome_gap(ost)
    np.testing.assert_array_equal(np.isnan(g), np.isnan(D.outcome_gap(ost.reshape(2, n_turns))))
    np.testing.assert_array_equal(np.nan_to_num(g), np.nan_to_num(
        D.outcome_gap(ost.reshape(2, n_turns))))


def dataclasses_items(b):
    return [(k, getattr(b, k)) for k in ("n_min", "prefix", "third", "shallow_budget",
                                         "deep_budget", "deep_support", "deep_shallow_kl")]


def test_argument_errors():
    st = np.zeros(3, O.STAT_DTYPE)
    l = T.lib()
    out = np.zeros(3)
    b = T.Budget()
    assert l.turnkl_loss_share(None, 3, out.ctypes.data) == T.ERR_INVALID_ARG
    assert l.turnkl_loss_share(st.ctypes.data, 0, out.ctypes.data) == T.ERR_INVALID_ARG
    assert l.turnkl_budget_report(st.ctypes.data, 3, -1, 8, 0.1, ctypes.byref(b)) == \
        T.ERR_INVALID_ARG
    assert l.turnkl_budget_report(st.ctypes.data, 3, 5, -1, 0.1, ctypes.byref(b)) == \
        T.ERR_INVALID_ARG
    assert l.turnkl_budget_report(st.ctypes.data, 3, 5, 8, float("nan"), ctypes.byref(b)) == \
        T.ERR_INVALID_ARG
    assert l.turnkl_budget_report(st.ctypes.data, 3, 5, 8, 0.1, None) == T.ERR_INVALID_ARG
    assert l.turnkl_outcome_gap(st.ctypes.data, 0, out.ctypes.data) == T.ERR_INVALID_ARG
    with pytest.raises(ValueError):
        T.outcome_gap(st)  # odd number of entries
    # an all-zero batch: no prefix, no mass
    r = T.budget_report(st, 0, 8, 0.15)
    assert r["prefix"] == 0 and r["third"] == 0 and math.isnan(r["deep_shallow_kl"])
    assert not T.loss_share(st).any()
