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

Readings where the paper is silent (each is listed in the design doc):
  * the loss is over the full vocabulary (the paper trains a top-50 variant);
  * T counts only turns with at least one supervised token; trajectories with
    no supervised token are left out of the mean over trajectories;
  * a segment is a maximal run of consecutive tokens with equal
    (trajectory id, turn id); negative trajectory ids mark padding, which
    belongs to no segment and must carry mask 0; trajectory ids increase from
    one segment to the next, turn ids increase within a trajectory, and
    0 <= turn id < max_turns; the first violation in token order is reported;
  * per-turn variance is the population variance (ddof = 0);
  * no clamp is applied to per-token KL.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle_rows.so")

OK = 0
ERR_UNSORTED = -4
ERR_TURN_RANGE = -5
ERR_PAD_MASK = -6

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
                                    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int]
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

    @property
    def count(self) -> int:
        return int(self.start.shape[0])


def segments(traj_id, turn_id, loss_mask, max_turns: int) -> Segments:
    """Walk the packed tokens in order and cut them into (trajectory, turn) runs."""
    traj_id = np.asarray(traj_id)
    turn_id = np.asarray(turn_id)
    loss_mask = np.asarray(loss_mask)
    start, length, traj, turn, n_sup = [], [], [], [], []
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
        if prev != (b, t):
            if traj:
                pb, pt = traj[-1], turn[-1]
                if b < pb or (b == pb and t <= pt):
                    return _failed(ERR_UNSORTED)
            start.append(i)
            length.append(0)
            traj.append(b)
            turn.append(t)
            n_sup.append(0)
        length[-1] += 1
        n_sup[-1] += 1 if m else 0
        prev = (b, t)
    a = lambda x: np.asarray(x, dtype=np.int64)
    return Segments(OK, a(start), a(length), a(traj), a(turn), a(n_sup))


def _failed(code: int) -> Segments:
    e = np.zeros(0, np.int64)
    return Segments(code, e, e, e, e, e)


# ----------------------------------------------------------------------------
# token weights (Sec. 5.2; App. D, Algorithm 1)


def token_weights(seg: Segments, n_tokens: int, loss_mask, alpha: float) -> np.ndarray:
    """w_i such that the batch loss is sum_i w_i * l_i.

    Per trajectory: q_traj_t = n_t / sum_j n_j, q_turn_t = 1 / T,
    q_blend_t = (1 - alpha) q_traj_t + alpha q_turn_t; the turn's weight is
    shared equally by its n_t supervised tokens, and trajectories are
    averaged (seq-mean-token-mean).
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
    for b in live:
        ss = [s for s in by_traj[b] if seg.n_sup[s] > 0]
        n_t = {s: int(seg.n_sup[s]) for s in ss}
        total = sum(n_t.values())          # N = sum_t n_t
        n_turns = len(ss)                  # T, turns with supervision
        for s in ss:
            q_traj = n_t[s] / total
            q_turn = 1.0 / n_turns
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
           n_threads: int = 0):
    """KL and dKL/dz_s for each row of [R, V] host arrays.

    dtype DTYPE_BF16 takes uint16 bf16 bit patterns, DTYPE_F32 float32 and
    DTYPE_F64 float64 logits.  Returns (kl [R], g [R, V] or None).
    """
    want = {DTYPE_BF16: np.uint16, DTYPE_F32: np.float32, DTYPE_F64: np.float64}[dtype]
    zs = np.ascontiguousarray(zs, dtype=want) if dtype == DTYPE_F64 else np.ascontiguousarray(zs)
    zt = np.ascontiguousarray(zt, dtype=want) if dtype == DTYPE_F64 else np.ascontiguousarray(zt)
    assert zs.shape == zt.shape and zs.ndim == 2
    assert zs.dtype == want and zt.dtype == want, (zs.dtype, want)
    r, v = zs.shape
    kl = np.empty(r, np.float64)
    g = np.empty((r, v), np.float64) if want_grad else None
    rc = _rows_lib().oracle_rows(zs.ctypes.data, v, zt.ctypes.data, v, dtype, r, v,
                                 kl.ctypes.data, None if g is None else g.ctypes.data, v,
                                 n_threads)
    if rc != 0:
        raise RuntimeError("oracle_rows failed")
    return kl, g


# ----------------------------------------------------------------------------
# loss and per-turn statistics


def losses(w_blend: np.ndarray, w_traj: np.ndarray, w_turn: np.ndarray, kl: np.ndarray):
    """(L_blend, L_traj, L_turn) = sum_i w_i * KL_i for the three weightings."""
    return (float(np.sum(w_blend * kl)), float(np.sum(w_traj * kl)), float(np.sum(w_turn * kl)))


def turn_stats(parts, max_turns: int) -> np.ndarray:
    """Per-turn-index statistics over one or more micro-batches.

    parts: iterable of (seg, loss_mask, kl, w) per micro-batch.  Everything is
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


def fwd_bwd(traj_id, turn_id, loss_mask, alpha: float, max_turns: int, row_source,
            dtype: int, grad_scale: float = 1.0, grad_rows=(), chunk_rows: int = 512,
            n_threads: int = 0) -> Result:
    """Reference for one call of the fused path.

    row_source(rows) -> (zs, zt): host arrays [len(rows), V] holding the
    listed rows (uint16 bf16 patterns or float32).  Only supervised rows are
    evaluated; rows listed in grad_rows also return their gradient.
    """
    traj_id = np.asarray(traj_id)
    loss_mask = np.asarray(loss_mask)
    n = int(traj_id.shape[0])
    seg = segments(traj_id, turn_id, loss_mask, max_turns)
    if seg.status != OK:
        return Result(seg.status, seg, np.zeros(n), np.zeros(n), (np.nan,) * 3,
                      np.zeros(max_turns, STAT_DTYPE), {})
    w = token_weights(seg, n, loss_mask, alpha)
    w0 = token_weights(seg, n, loss_mask, 0.0)
    w1 = token_weights(seg, n, loss_mask, 1.0)
    kl = np.zeros(n, np.float64)
    sup = np.nonzero(loss_mask)[0]
    for k0 in range(0, sup.shape[0], chunk_rows):
        rows = sup[k0:k0 + chunk_rows]
        zs, zt = row_source(rows)
        kl[rows], _ = row_kl(zs, zt, dtype, want_grad=False, n_threads=n_threads)
    grads = {}
    want = np.asarray(sorted(set(int(r) for r in grad_rows)), np.int64)
    for k0 in range(0, want.shape[0], chunk_rows):
        rows = want[k0:k0 + chunk_rows]
        zs, zt = row_source(rows)
        _, g = row_kl(zs, zt, dtype, want_grad=True, n_threads=n_threads)
        for k, r in enumerate(rows.tolist()):
            grads[r] = g[k]
    stats = turn_stats([(seg, loss_mask, kl, w)], max_turns)
    return Result(OK, seg, w, kl, losses(w, w0, w1, kl), stats, grads)
