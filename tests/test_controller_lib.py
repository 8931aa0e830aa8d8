"""The library's depth controller (turnkl_depth_*, host code) against the
oracle: the worked example, long random runs, and argument errors."""
import json
import os

import numpy as np
import pytest

from oracle import depth_controller as D
from paper_2607_05804_amd import turnkl as T

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "depth_controller_example.json")


def _stats(kl_mean, n_traj):
    st = np.zeros(len(kl_mean), T.STAT_DTYPE)
    st["kl_mean"] = kl_mean
    st["n_traj"] = n_traj
    return st


def _oracle_cfg(lib_ctl):
    c = lib_ctl.config
    return D.Config(h_min=c.h_min, h_max=c.h_max, warmup_steps=c.warmup_steps,
                    probe_interval=c.probe_interval, min_cov_traj=c.min_cov_traj,
                    coverage_quantile=c.coverage_quantile, ema_alpha=c.ema_alpha, eps=c.eps)


def test_default_config_is_the_papers_table():
    c = T.DepthController().config
    assert (c.h_min, c.h_max, c.warmup_steps, c.probe_interval, c.min_cov_traj) == (2, 50, 3, 8, 8)
    assert (c.coverage_quantile, c.ema_alpha) == (0.8, 0.3)
    assert _oracle_cfg(T.DepthController()) == D.Config()


def test_worked_example():
    with open(GOLDEN) as f:
        g = json.load(f)
    pb = g["probe_batch"]
    ctl = T.DepthController()
    for ref in g["steps"]:
        cap, probe, roll = ctl.plan(ref["k"])
        assert (cap, probe, roll) == (ref["cap"], ref["probe"], ref["roll"])
        if probe:
            ctl.update(_stats(pb["kl_mean"], pb["n_traj"]), pb["success_lengths"])
        assert abs(ctl.state.h_bar - ref["h_bar"]) < 1e-9
    assert (ctl.state.h_eff, ctl.state.h_cov, ctl.state.h_ctrl) == (g["h_eff"], g["h_cov"], g["h_ctrl"])


@pytest.mark.parametrize("seed", range(6))
def test_random_runs_match_the_oracle(seed):
    rng = np.random.default_rng(1000 + seed)
    kw = dict(h_min=int(rng.integers(1, 4)), h_max=int(rng.integers(8, 80)),
              warmup_steps=int(rng.integers(0, 5)), probe_interval=int(rng.integers(1, 10)),
              min_cov_traj=int(rng.integers(0, 12)),
              coverage_quantile=float(rng.choice([0.4, 0.6, 0.8, 1.0, rng.uniform(0.05, 1.0)])),
              ema_alpha=float(rng.uniform(0.0, 1.0)))
    ctl = T.DepthController(**kw)
    cfg = _oracle_cfg(ctl)
    st = D.init(cfg)
    for k in range(1, 150):
        want = D.plan(cfg, st, k)
        assert ctl.plan(k) == want, k
        if want[1]:
            T_ = int(rng.integers(1, 60))
            n = np.sort(rng.integers(0, 64, size=T_))[::-1].astype(np.int64)
            if rng.uniform() < 0.1:
                n[0] = 0
            K = rng.normal(0.2, 0.3, size=T_) * np.exp(-0.1 * np.arange(T_))
            L = rng.integers(1, 60, size=int(rng.integers(0, 40)))
            ctl.update(_stats(K, n), L)
            st = D.update(cfg, st, list(K), list(n), list(L))
            s = ctl.state
            assert (s.h_eff, s.h_cov, s.h_ctrl, s.n_probes) == (st.h_eff, st.h_cov, st.h_ctrl,
                                                                st.n_probes)
            assert abs(s.h_eff_bar - st.h_eff_bar) <= 1e-12 * max(1.0, abs(st.h_eff_bar))
            assert abs(s.h_bar - st.h_bar) <= 1e-12 * max(1.0, abs(st.h_bar))


def test_argument_errors():
    with pytest.raises(T.TurnKLError):
        T.DepthController(h_min=0)
    with pytest.raises(T.TurnKLError):
        T.DepthController(h_min=10, h_max=5)
    with pytest.raises(T.TurnKLError):
        T.DepthController(coverage_quantile=0.0)
    with pytest.raises(T.TurnKLError):
        T.DepthController(coverage_quantile=1.5)
    with pytest.raises(T.TurnKLError):
        T.DepthController(ema_alpha=-0.1)
    with pytest.raises(T.TurnKLError):
        T.DepthController(probe_interval=0)
    with pytest.raises(T.TurnKLError):
        T.DepthController(eps=float("nan"))
    ctl = T.DepthController()
    with pytest.raises(T.TurnKLError):
        ctl.plan(0)
    before = (ctl.state.h_bar, ctl.state.n_probes)
    with pytest.raises(T.TurnKLError):
        ctl.update(_stats([0.1], [3]), [2, 0, 3])  # a length < 1
    with pytest.raises(T.TurnKLError):
        ctl.update(np.zeros(0, T.STAT_DTYPE), [])  # no turns
    assert (ctl.state.h_bar, ctl.state.n_probes) == before
