"""CPU oracle for TurnOPD's adaptive rollout-depth controller (arXiv 2607.05804).

TEST INFRASTRUCTURE.  Only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may import this module.  It shares no code with the
library (paper_2607_05804_amd/) and imports nothing from it.

What it states, in the paper's order:
  Sec. 5.1 (External Mismatch: Adaptive Rollout-Depth Budgeting) and App. D,
  Algorithm 1:
    efficiency arm   m_t = [K_t]_+ * n_t / n_0,  q_t = m_t / (sum_j m_j + eps),
                     H_eff = round(sum_t t q_t)        (t is the 0-based turn index)
    coverage arm     H_cov = min{H : F_succ(H) >= p} over the completion lengths
                     of successful probe trajectories, refreshed only when at
                     least n_min^cov of them are available (else kept; 0 at start)
    controller       H_ctrl = max(H_eff, H_cov)
    smoothing        Hbar_k = (1 - alpha_ema) Hbar_{k-1} + alpha_ema H_ctrl on probe
                     steps, Hbar_k = Hbar_{k-1} otherwise; Hbar_0 = H_max
    applied cap      Hhat_k = clip(round(Hbar_{k-1}) + 1, H_min, H_max)
    probe schedule   probe_k = (k <= K_warm) or (k mod r_probe == 0), k = 1, 2, ...
                     probe steps roll out to H_max, others to Hhat_k
  App. D, full-configuration table: p = 0.80, n_min^cov = 8, H_min/H_max = 2/50,
  alpha_ema = 0.30, r_probe = 8, K_warm = 3.

Readings where the paper is silent or ambiguous:
  * turn indices are 0-based throughout (the rollout-depth figure states the
    convention; the +1 of the applied cap converts an index to a depth), so a
    successful trajectory of L turns completes at index L - 1 and
    H_cov = min{H >= 0 : #{L_i - 1 <= H} / n >= p}, the inverted-CDF p-quantile
    of L minus one;
  * round() is round-half-to-even;
  * eps = 1e-12 (the paper only says a small constant);
  * n_0 = 0 (no trajectory supervised at turn 0) gives m_t = 0 for every t;
  * K_t and n_t are the pooled per-turn KL mean and the survivor count of the
    probe batch's per-turn statistics.
"""
from __future__ import annotations

import dataclasses
import math

DEFAULT_EPS = 1e-12


@dataclasses.dataclass(frozen=True)
class Config:
    """App. D, full-configuration table."""
    h_min: int = 2
    h_max: int = 50
    warmup_steps: int = 3
    probe_interval: int = 8
    min_cov_traj: int = 8
    coverage_quantile: float = 0.80
    ema_alpha: float = 0.30
    eps: float = DEFAULT_EPS


@dataclasses.dataclass
class State:
    h_bar: float             # EMA of H_ctrl; starts at H_max
    h_cov: int = 0           # coverage floor (0-based index); 0 until refreshed
    h_eff: int = -1          # last efficiency centroid, rounded; -1 before any probe
    h_eff_bar: float = -1.0  # last centroid before rounding
    h_ctrl: int = -1         # last max(H_eff, H_cov)
    n_probes: int = 0


def round_half_even(x: float) -> int:
    """round() with ties to the even integer (Python's own rule, written out)."""
    f = math.floor(x)
    d = x - f
    if d > 0.5:
        return f + 1
    if d < 0.5:
        return f
    return f if f % 2 == 0 else f + 1


def init(cfg: Config) -> State:
    """Algorithm 1: Hbar_0 = H_max, H_cov = 0."""
    return State(h_bar=float(cfg.h_max))


def is_probe(cfg: Config, k: int) -> bool:
    """Algorithm 1: a probe step during warm-up and every r_probe-th step."""
    return k <= cfg.warmup_steps or k % cfg.probe_interval == 0


def cap(cfg: Config, st: State) -> int:
    """Hhat_k = clip(round(Hbar_{k-1}) + 1, H_min, H_max) (Sec. 5.1)."""
    h = round_half_even(st.h_bar) + 1
    return min(max(h, cfg.h_min), cfg.h_max)


def plan(cfg: Config, st: State, k: int):
    """(Hhat_k, probe_k, rollout depth) for step k."""
    h_cap = cap(cfg, st)
    probe = is_probe(cfg, k)
    return h_cap, probe, (cfg.h_max if probe else h_cap)


def efficiency_centroid(cfg: Config, kl_mean, n_traj):
    """m_t = [K_t]_+ n_t / n_0, q_t = m_t / (sum m + eps), centroid sum t q_t."""
    n0 = n_traj[0] if len(n_traj) else 0
    m = []
    for t in range(len(kl_mean)):
        k_pos = kl_mean[t] if kl_mean[t] > 0.0 else 0.0
        m.append(k_pos * n_traj[t] / n0 if n0 > 0 else 0.0)
    total = sum(m) + cfg.eps
    centroid = 0.0
    for t, mt in enumerate(m):
        centroid += t * (mt / total)
    return centroid


def coverage_floor(cfg: Config, success_lengths):
    """min{H >= 0 : F_succ(H) >= p}, F_succ(H) = share of successful
    trajectories whose last turn index L - 1 is <= H."""
    n = len(success_lengths)
    h = 0
    while True:
        done = sum(1 for L in success_lengths if L - 1 <= h)
        if done / n >= cfg.coverage_quantile:
            return h
        h += 1


def update(cfg: Config, st: State, kl_mean, n_traj, success_lengths) -> State:
    """One probe step of Algorithm 1, given the probe batch's per-turn KL
    means K_t, survivor counts n_t and the completion lengths (turns) of its
    successful trajectories."""
    st = dataclasses.replace(st)
    st.h_eff_bar = efficiency_centroid(cfg, kl_mean, n_traj)
    st.h_eff = round_half_even(st.h_eff_bar)
    if len(success_lengths) >= max(cfg.min_cov_traj, 1):
        st.h_cov = coverage_floor(cfg, success_lengths)
    st.h_ctrl = max(st.h_eff, st.h_cov)
    st.h_bar = (1.0 - cfg.ema_alpha) * st.h_bar + cfg.ema_alpha * st.h_ctrl
    st.n_probes += 1
    return st


def run(cfg: Config, probes, n_steps: int):
    """Drive the controller for steps 1..n_steps.  probes(k) -> (kl_mean,
    n_traj, success_lengths) is called on probe steps only.  Returns the list
    of (k, Hhat_k, probe_k, rollout depth, state after step k)."""
    st = init(cfg)
    out = []
    for k in range(1, n_steps + 1):
        h_cap, probe, h_roll = plan(cfg, st, k)
        if probe:
            st = update(cfg, st, *probes(k))
        out.append((k, h_cap, probe, h_roll, dataclasses.replace(st)))
    return out
