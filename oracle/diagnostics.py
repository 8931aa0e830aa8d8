"""CPU oracle for TurnOPD's turn-level loss-allocation diagnostics
(arXiv 2607.05804).

TEST INFRASTRUCTURE.  Only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may import this module.  It shares no code with the HIP
path (paper_2607_05804_amd/) and imports nothing from it.

Inputs are the per-turn statistics of one batch (STAT_DTYPE rows: n_tokens,
n_traj, kl_mean, kl_m2, kl_var, loss_mass), as the fused call returns them.

  loss_share     Sec. 4.4: s_t, the share of the batch's loss mass that turn
                 t carries; with statistics taken at alpha = 0 it is
                 s_t^traj of the trajectory-level objective, otherwise the
                 budget the blended objective actually spends (Sec. 7.2).
  budget_report  Sec. 4.4, Table 1 (deep/shallow raw KL, deep support, deep
                 loss budget) and Sec. 7.2, Table 3 (deep budget) over the
                 reliable turn prefix.
  outcome_gap    Sec. 4.2: G_t = K_t^fail - K_t^succ.

Readings where the paper is silent:
  * the reliable prefix is the run of leading turns whose survivor count is
    at least n_min = max(floor, ceil(frac * n_traj)); with (8, 0.15) and the
    batch's trajectory count it is the training floor of App. D, with (8,
    0.10) and n_traj = n_0 the per-step part of Sec. 4.1's plotting rule
    (its persistence over 60% of the training steps spans steps and is left
    to the caller);
  * the shallow and the deep third are the first and the last ceil(P / 3)
    turns of a prefix of P turns;
  * deep support is the mean over the deep third of n_t / n_0; the
    deep/shallow raw-KL ratio is the mean of K_t over the deep third divided
    by its mean over the shallow third (NaN when that is 0 or P = 0);
  * s_t is 0 for every turn when the batch has no loss mass; G_t is NaN where
    either outcome has no supervised token at turn t.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np


def loss_share(stats: np.ndarray) -> np.ndarray:
    """s_t = loss_mass[t] / sum_u loss_mass[u]."""
    mass = np.asarray(stats["loss_mass"], np.float64)
    total = float(sum(float(m) for m in mass))
    if total == 0.0:
        return np.zeros(mass.shape[0])
    return mass / total


def reliable_prefix(stats: np.ndarray, n_min: int) -> int:
    """P: the number of leading turns t = 0, 1, ... with n_t >= n_min."""
    p = 0
    for n_t in np.asarray(stats["n_traj"]):
        if int(n_t) < n_min or int(n_t) == 0:
            break
        p += 1
    return p


@dataclasses.dataclass
class Budget:
    n_min: int
    prefix: int
    third: int
    shallow_budget: float
    deep_budget: float
    deep_support: float
    deep_shallow_kl: float


def budget_report(stats: np.ndarray, n_traj: int, floor: int, frac: float) -> Budget:
    n_min = max(int(floor), math.ceil(float(frac) * float(n_traj)))
    P = reliable_prefix(stats, n_min)
    if P == 0:
        return Budget(n_min, 0, 0, 0.0, 0.0, 0.0, math.nan)
    k = -(-P // 3)
    s = loss_share(stats)
    shallow = list(range(0, k))
    deep = list(range(P - k, P))
    n0 = float(stats["n_traj"][0])
    kl = np.asarray(stats["kl_mean"], np.float64)
    kl_sh = sum(kl[t] for t in shallow) / k
    kl_dp = sum(kl[t] for t in deep) / k
    return Budget(
        n_min=n_min, prefix=P, third=k,
        shallow_budget=float(sum(s[t] for t in shallow)),
        deep_budget=float(sum(s[t] for t in deep)),
        deep_support=float(sum(float(stats["n_traj"][t]) / n0 for t in deep) / k),
        deep_shallow_kl=float(kl_dp / kl_sh) if kl_sh != 0.0 else math.nan)


def outcome_gap(outcome_stats: np.ndarray) -> np.ndarray:
    """G_t = K_t^fail - K_t^succ from the [2, T] per-outcome statistics
    (row 0 failed, row 1 successful); NaN where either side is empty."""
    fail, succ = outcome_stats[0], outcome_stats[1]
    g = np.full(fail.shape[0], np.nan)
    for t in range(fail.shape[0]):
        if fail["n_tokens"][t] > 0 and succ["n_tokens"][t] > 0:
            g[t] = float(fail["kl_mean"][t]) - float(succ["kl_mean"][t])
    return g
