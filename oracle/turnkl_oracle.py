"""CPU oracle for TurnOPD's fused turn-KL loss (arXiv 2607.05804).

TEST INFRASTRUCTURE.  Only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may import this module.  It shares no code with the HIP
path (paper_2607_05804_amd/) and imports nothing from it.

It is a plain, slow, float64 statement of what the hot path computes:

  segments     Sec. 3 (Preliminaries): a trace is x, o_1, r_1, ..., o_T, r_T;
               turn t = observation o_t then response r_t; only response
               tokens carry the mask m_i.  Sec. 4.4 (Loss Aggregation): a
               trajectory has T supervised turns, turn t has n_t supervised
               tokens, N = sum_t n_t.
  row_kl       Sec. 3, Eq. (opd-rkl): per-token reverse KL over the full
               vocabulary, and its student-logit gradient (oracle/rows.c).
  weights      Sec. 5.2 (Progressive Turn-Normalized Loss Budgeting):
               q_traj_t = n_t / sum_j n_j, q_turn_t = 1 / T,
               q_blend_t = (1 - alpha) q_traj_t + alpha q_turn_t; App. D,
               Algorithm 1: w_blend = (1 - alpha) w_traj + alpha w_turn and
               L = sum_i w_blend,i l_i; base aggregation seq-mean-token-mean
               (App. D, full-configuration table), i.e. a mean over
               trajectories of per-trajectory token means (Eq. (opd-rkl)).
  turn_stats   Sec. 4.3, Eq. (observed-turn-kl): K_t is the mean raw KL over
               the supervised token contexts collected at turn t; Sec. 5.1 and
               App. D: survivors n_t (trajectories that reach turn t) and
               K_t drive the depth controller; Sec. 4.4: s_t, the turn's share
               of the loss mass.
  alpha_schedule  Sec. 5.2 / Algorithm 1: alpha = clip((k/K - s)/(e - s), 0, 1).
  support floor   App. D (full-configuration table, internal blend): the
               turn-level floor n_min = max(floor, ceil(frac * n_traj)), with
               floor 8 and frac 0.15 in the paper; Sec. 7.2 calls the turns it
               admits "valid turns" (turns reached by enough trajectories).
  outcome split   Sec. 4.2: K_t^fail and K_t^succ, the per-turn KL means over
               failed and successful rollouts, whose difference is G_t.

Readings where the paper is silent:
  * the loss is over the full vocabulary (the paper trains a top-50 variant);
  * T counts only turns with at least one supervised token; trajectories with
    no supervised token are left out of the mean over trajectories;
  * a segment is a maximal run of consecutive tokens with equal
    (trajectory id, turn id); negative trajectory ids mark padding, which
    belongs to no segment and must carry mask 0; trajectory ids increase from
    one segment to the next, turn ids increase within a trajectory, and
    0 <= turn id < max_turns; the first violation in token order is reported;
  * per-turn variance is the population variance (ddof = 0);
  * no clamp is applied to per-token KL;
  * support floor (the paper does not say how n_min enters the turn term):
    n_traj is B, the trajectories of the call with a supervised token; turn t
    is valid when its survivor count n_t (trajectories with a supervised token
    at t) is at least n_min, with frac * B rounded once in float64 before the
    ceiling; a trajectory's turn term gives each of its valid supervised turns
    1 / T_v (T_v of them) and its other turns 0; a trajectory with no valid
    supervised turn takes its trajectory term for the turn term.  floor = 0
    and frac = 0 admit every supervised turn (the plain blend);
  * outcome flags are per token, equal across every non-padding token of a
    trajectory (padding tokens' flags are ignored); nonzero means success.
    The first token in token order where a flag differs from the one before
    it in its segment, or a segment start whose flag differs from its
    trajectory's first segment, is an error (after the other checks at the
    same token).
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle_rows.so")

OK = 0
ERR_UNSORTED = -4
ERR_TURN_RANGE = -5
ERR_PAD_MASK = -6
ERR_OUTCOME = -10

DTYPE_BF16 = 0
DTYPE_F32 = 1
DTYPE_F64 = 2

STAT_DTYPE = np.dtype([("n_tokens", "<i8"), ("n_traj", "<i8"), ("kl_mean", "<f8"),
                       ("kl_m2", "<f8"), ("kl_var", "<f8"), ("loss_mass", "<f8")])

_lib = None


def _rows_lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python oracle/build.py`")
        lib = ctypes.CDLL(LIB_PATH)
        lib.oracle_rows.restype = ctypes.c_int
        lib.oracle_rows.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                    ctypes.c_int64, ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
                                    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                    ctypes.c_void_p, ctypes.c_int]
        lib.oracle_max_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def max_threads() -> int:
    return int(_rows_lib().oracle_max_threads())


# ----------------------------------------------------------------------------
# segments


@dataclasses.dataclass
class Segments:
    status: int
    start: np.ndarray   # first token of the segment
    length: np.ndarray  # tokens in the segment (consecutive)
    traj: np.ndarray    # trajectory id
    turn: np.ndarray    # turn id
    n_sup: np.ndarray   # supervised tokens, n_t for (traj, turn)
    success: np.ndarray = None  # outcome flag (0/1) of the segment's trajectory, if given

    @property
    def count(self) -> int:
        return int(self.start.shape[0])


def segments(traj_id, turn_id, loss_mask, max_turns: int, success=None) -> Segments:
    """Walk the packed tokens in order and cut them into (trajectory, turn) runs.

    success: optional per-token outcome flags (nonzero = the trajectory
    succeeded), checked to be constant over each trajectory's tokens."""
    traj_id = np.asarray(traj_id)
    turn_id = np.asarray(turn_id)
    loss_mask = np.asarray(loss_mask)
    flags = None if success is None else np.asarray(success)
    start, length, traj, turn, n_sup, seg_flag = [], [], [], [], [], []
    traj_flag = {}  # trajectory id -> flag of its first segment
    prev = None  # (traj, turn) of the previous token, None after padding
    for i in range(traj_id.shape[0]):
        b, t, m = int(traj_id[i]), int(turn_id[i]), int(loss_mask[i])
        if b < 0:
            if m != 0:
                return _failed(ERR_PAD_MASK)
            prev = None
            continue
        if not 0 <= t < max_turns:
            return _failed(ERR_TURN_RANGE)
        f = None if flags is None else int(flags[i] != 0)
        if prev != (b, t):
            if traj:
                pb, pt = traj[-1], turn[-1]
                if b < pb or (b == pb and t <= pt):
                    return _failed(ERR_UNSORTED)
            if f is not None:
                if traj_flag.setdefault(b, f) != f:
                    return _failed(ERR_OUTCOME)
                seg_flag.append(f)
            start.append(i)
            length.append(0)
            traj.append(b)
            turn.append(t)
            n_sup.append(0)
        elif f is not None and f != seg_flag[-1]:
            return _failed(ERR_OUTCOME)
        length[-1] += 1
        n_sup[-1] += 1 if m else 0
        prev = (b, t)
    a = lambda x: np.asarray(x, dtype=np.int64)
    return Segments(OK, a(start), a(length), a(traj), a(turn), a(n_sup),
                    None if flags is None else a(seg_flag))


def _failed(code: int) -> Segments:
    e = np.zeros(0, np.int64)
    return Segments(code, e, e, e, e, e)


# ----------------------------------------------------------------------------
# token weights (Sec. 5.2; App. D, Algorithm 1)


def n_min_of(n_traj: int, floor: int, frac: float) -> int:
    """n_min = max(floor, ceil(frac * n_traj)) (App. D, full-configuration
    table: min_floor and min_frac of the internal blend)."""
    return max(int(floor), math.ceil(float(frac) * float(n_traj)))


def turn_survivors(seg: Segments, max_turns: int) -> np.ndarray:
    """n_t: trajectories with at least one supervised token at turn t."""
    n = np.zeros(max_turns, np.int64)
    for s in range(seg.count):
        if seg.n_sup[s] > 0:
            n[int(seg.turn[s])] += 1
    return n


def token_weights(seg: Segments, n_tokens: int, loss_mask, alpha: float,
                  floor: int = 0, frac: float = 0.0) -> np.ndarray:
    """w_i such that the batch loss is sum_i w_i * l_i.

    Per trajectory: q_traj_t = n_t / sum_j n_j, q_turn_t = 1 / T,
    q_blend_t = (1 - alpha) q_traj_t + alpha q_turn_t; the turn's weight is
    shared equally by its n_t supervised tokens, and trajectories are
    averaged (seq-mean-token-mean).  With a support floor, the turn term
    covers only the valid turns (survivors >= n_min): 1 / T_v on each, 0 on
    the others, and the trajectory term when the trajectory has none.
    """
    loss_mask = np.asarray(loss_mask)
    w = np.zeros(n_tokens, np.float64)
    by_traj: dict[int, list[int]] = {}
    for s in range(seg.count):
        by_traj.setdefault(int(seg.traj[s]), []).append(s)
    live = [b for b, ss in by_traj.items() if sum(int(seg.n_sup[s]) for s in ss) > 0]
    if not live:
        return w
    n_live = len(live)
    max_turn = int(seg.turn.max()) + 1
    surv = turn_survivors(seg, max_turn)
    n_min = n_min_of(n_live, floor, frac)
    for b in live:
        ss = [s for s in by_traj[b] if seg.n_sup[s] > 0]
        n_t = {s: int(seg.n_sup[s]) for s in ss}
        total = sum(n_t.values())          # N = sum_t n_t
        valid = {s: surv[int(seg.turn[s])] >= n_min for s in ss}
        n_valid = sum(valid.values())      # T_v; T when every turn is valid
        for s in ss:
            q_traj = n_t[s] / total
            if n_valid:
                q_turn = (1.0 / n_valid) if valid[s] else 0.0
            else:
                q_turn = q_traj
            q_blend = (1.0 - alpha) * q_traj + alpha * q_turn
            per_token = q_blend / n_t[s] / n_live
            lo, hi = int(seg.start[s]), int(seg.start[s] + seg.length[s])
            for i in range(lo, hi):
                if loss_mask[i]:
                    w[i] = per_token
    return w


# ----------------------------------------------------------------------------
# per-row KL and gradient (oracle/rows.c)


def row_kl(zs: np.ndarray, zt: np.ndarray, dtype: int, want_grad: bool = True,
           n_threads: int = 0, lse_out: np.ndarray | None = None):
    """KL and dKL/dz_s for each row of [R, V] host arrays.

    dtype DTYPE_BF16 takes uint16 bf16 bit patterns, DTYPE_F32 float32 and
    DTYPE_F64 float64 logits.  Returns (kl [R], g [R, V] or None); lse_out, a
    float64 [R, 2] array, receives each row pair's log-partition functions
    (lse_s, lse_t).
    """
    want = {DTYPE_BF16: np.uint16, DTYPE_F32: np.float32, DTYPE_F64: np.float64}[dtype]
    zs = np.ascontiguousarray(zs, dtype=want) if dtype == DTYPE_F64 else np.ascontiguousarray(zs)
    zt = np.ascontiguousarray(zt, dtype=want) if dtype == DTYPE_F64 else np.ascontiguousarray(zt)
    assert zs.shape == zt.shape and zs.ndim == 2
    assert zs.dtype == want and zt.dtype == want, (zs.dtype, want)
    r, v = zs.shape
    kl = np.empty(r, np.float64)
    g = np.empty((r, v), np.float64) if want_grad else None
    if lse_out is not None:
        assert lse_out.dtype == np.float64 and lse_out.shape == (r, 2)
        assert lse_out.flags.c_contiguous
    rc = _rows_lib().oracle_rows(zs.ctypes.data, v, zt.ctypes.data, v, dtype, r, v,
                                 kl.ctypes.data, None if g is None else g.ctypes.data, v,
                                 None if lse_out is None else lse_out.ctypes.data, n_threads)
    if rc != 0:
        raise RuntimeError("oracle_rows failed")
    return kl, g


# ----------------------------------------------------------------------------
# loss and per-turn statistics


def losses(w_blend: np.ndarray, w_traj: np.ndarray, w_turn: np.ndarray, kl: np.ndarray):
    """(L_blend, L_traj, L_turn) = sum_i w_i * KL_i for the three weightings."""
    return (float(np.sum(w_blend * kl)), float(np.sum(w_traj * kl)), float(np.sum(w_turn * kl)))


def turn_stats(parts, max_turns: int, outcome=None) -> np.ndarray:
    """Per-turn-index statistics over one or more micro-batches.

    parts: iterable of (seg, loss_mask, kl, w) per micro-batch; outcome 0 or 1
    keeps only the segments of failed or successful trajectories (their
    flags in seg.success).  Everything is
    recomputed from the pooled per-token values (no merge formula):
      n_tokens[t]  supervised tokens at turn t
      n_traj[t]    trajectories with a supervised token at turn t (survivors)
      kl_mean[t]   pooled mean KL,  kl_m2[t] = sum (KL - mean)^2,
      kl_var[t]    kl_m2 / n_tokens (population variance)
      loss_mass[t] sum_i w_i KL_i over turn-t tokens
    """
    vals = [[] for _ in range(max_turns)]
    mass = np.zeros(max_turns, np.float64)
    surv = np.zeros(max_turns, np.int64)
    for seg, loss_mask, kl, w in parts:
        loss_mask = np.asarray(loss_mask)
        for s in range(seg.count):
            if outcome is not None and int(seg.success[s]) != int(outcome):
                continue
            t = int(seg.turn[s])
            if seg.n_sup[s] > 0:
                surv[t] += 1
            lo, hi = int(seg.start[s]), int(seg.start[s] + seg.length[s])
            for i in range(lo, hi):
                if loss_mask[i]:
                    vals[t].append(float(kl[i]))
                    mass[t] += float(w[i]) * float(kl[i])
    out = np.zeros(max_turns, STAT_DTYPE)
    for t in range(max_turns):
        x = np.asarray(vals[t], np.float64)
        n = x.shape[0]
        out["n_tokens"][t] = n
        out["n_traj"][t] = surv[t]
        out["loss_mass"][t] = mass[t]
        if n:
            mean = x.sum() / n
            m2 = float(np.sum((x - mean) ** 2))
            out["kl_mean"][t] = mean
            out["kl_m2"][t] = m2
            out["kl_var"][t] = m2 / n
    return out


def alpha_schedule(k: int, K: int, s: float = 0.0, e: float = 1.0) -> float:
    """alpha_k = clip((k/K - s) / (e - s), 0, 1); for e <= s a step at s."""
    prog = k / K
    if e <= s:
        return 1.0 if prog >= s else 0.0
    return min(1.0, max(0.0, (prog - s) / (e - s)))


# ----------------------------------------------------------------------------
# whole pass


@dataclasses.dataclass
class Result:
    status: int
    seg: Segments
    w: np.ndarray            # blended weights (float64, per token)
    kl: np.ndarray           # per-token KL (float64; 0 where unsupervised)
    loss: tuple              # (L_blend, L_traj, L_turn)
    stats: np.ndarray        # STAT_DTYPE [max_turns]
    grads: dict              # row -> unweighted dKL/dz_s float64 [V]; G = grad_scale * w[row] * g
    outcome_stats: np.ndarray = None  # STAT_DTYPE [2, max_turns]: failed, successful
    lse: np.ndarray = None   # [N, 2] (lse_s, lse_t) of supervised rows, NaN elsewhere


def fwd_bwd(traj_id, turn_id, loss_mask, alpha: float, max_turns: int, row_source,
            dtype: int, grad_scale: float = 1.0, grad_rows=(), chunk_rows: int = 512,
            n_threads: int = 0, support_floor: int = 0, support_frac: float = 0.0,
            success=None) -> Result:
    """Reference for one call of the fused path.

    row_source(rows) -> (zs, zt): host arrays [len(rows), V] holding the
    listed rows (uint16 bf16 patterns or float32).  Only supervised rows are
    evaluated; rows listed in grad_rows also return their gradient.
    support_floor, support_frac: the turn-support floor of the turn term;
    success: per-token outcome flags (adds the per-outcome statistics).
    """
    traj_id = np.asarray(traj_id)
    loss_mask = np.asarray(loss_mask)
    n = int(traj_id.shape[0])
    seg = segments(traj_id, turn_id, loss_mask, max_turns, success)
    if seg.status != OK:
        return Result(seg.status, seg, np.zeros(n), np.zeros(n), (np.nan,) * 3,
                      np.zeros(max_turns, STAT_DTYPE), {})
    w = token_weights(seg, n, loss_mask, alpha, support_floor, support_frac)
    w0 = token_weights(seg, n, loss_mask, 0.0, support_floor, support_frac)
    w1 = token_weights(seg, n, loss_mask, 1.0, support_floor, support_frac)
    kl = np.zeros(n, np.float64)
    lse = np.full((n, 2), np.nan)
    sup = np.nonzero(loss_mask)[0]
    for k0 in range(0, sup.shape[0], chunk_rows):
        rows = sup[k0:k0 + chunk_rows]
        zs, zt = row_source(rows)
        part = np.empty((rows.shape[0], 2))
        kl[rows], _ = row_kl(zs, zt, dtype, want_grad=False, n_threads=n_threads, lse_out=part)
        lse[rows] = part
    grads = {}
    want = np.asarray(sorted(set(int(r) for r in grad_rows)), np.int64)
    for k0 in range(0, want.shape[0], chunk_rows):
        rows = want[k0:k0 + chunk_rows]
        zs, zt = row_source(rows)
        _, g = row_kl(zs, zt, dtype, want_grad=True, n_threads=n_threads)
        for k, r in enumerate(rows.tolist()):
            grads[r] = g[k]
    stats = turn_stats([(seg, loss_mask, kl, w)], max_turns)
    return Result(OK, seg, w, kl, losses(w, w0, w1, kl), stats, grads,
                  outcome_split(seg, loss_mask, kl, w, max_turns), lse)


def outcome_split(seg: Segments, loss_mask, kl, w, max_turns: int):
    """Per-turn statistics of the failed (row 0) and successful (row 1)
    trajectories (Sec. 4.2), or None without outcome flags."""
    if seg.success is None:
        return None
    out = np.zeros((2, max_turns), STAT_DTYPE)
    for f in (0, 1):
        out[f] = turn_stats([(seg, loss_mask, kl, w)], max_turns, outcome=f)
    return out
