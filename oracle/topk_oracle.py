"""CPU oracle for the top-K reverse-KL variant of TurnOPD's distillation loss
(arXiv 2607.05804).

TEST INFRASTRUCTURE.  Only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may import this module.  It shares no code with the HIP
path (paper_2607_05804_amd/) and imports nothing from it.

The paper trains with a reverse KL on the teacher's top-K support, K = 50
(App. D: Algorithm 1 computes "top-K reverse-KL token losses"; the
full-configuration table lists the teacher top-K support size and the
top-K reverse-KL loss mode).  It does not print the formula.  Reading used
here:
  * T1  the support S_i of token i is the set of K vocabulary ids the teacher
        ranks highest (passed in by the caller, distinct, in [0, V));
  * T2  both distributions are renormalised over S_i:
          p^_s(v) = exp(a_v) / sum_{u in S_i} exp(a_u),  p^_t likewise from the
          teacher's values on S_i (logits or log-probabilities: a per-row
          constant cancels),
        and the token loss is the reverse KL of the two, student first
        (Sec. 3, Eq. opd-rkl restricted to S_i):
          KL_i = sum_{v in S_i} p^_s(v) (log p^_s(v) - log p^_t(v));
  * T3  its gradient with respect to the student logits is
          dKL_i/da_v = p^_s(v) (d_v - KL_i),  d_v = log p^_s(v) - log p^_t(v)
        for v in S_i, and 0 for every other id;
  * the weights, loss, per-turn statistics and segment rules are those of the
    full-vocabulary path (oracle/turnkl_oracle.py), unchanged.
"""
from __future__ import annotations

import numpy as np

from . import turnkl_oracle as O


def support_lse(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """[n, 2]: log sum_{v in S_i} exp of the student and of the teacher values
    on each row's support (max shift, then log of the sum), in float64."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    ma = a.max(axis=1, keepdims=True)
    mb = b.max(axis=1, keepdims=True)
    return np.concatenate([ma + np.log(np.exp(a - ma).sum(axis=1, keepdims=True)),
                           mb + np.log(np.exp(b - mb).sum(axis=1, keepdims=True))], axis=1)


def topk_row_kl(a: np.ndarray, b: np.ndarray, want_grad: bool = True):
    """a, b: float64 [n, K] student and teacher values on each row's support.
    Returns (kl [n], g [n, K]) by the two-pass definition (max shift, lse,
    explicit probabilities), in float64."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    ma = a.max(axis=1, keepdims=True)
    mb = b.max(axis=1, keepdims=True)
    ls = a - (ma + np.log(np.exp(a - ma).sum(axis=1, keepdims=True)))
    lt = b - (mb + np.log(np.exp(b - mb).sum(axis=1, keepdims=True)))
    p = np.exp(ls)
    d = ls - lt
    kl = (p * d).sum(axis=1)
    g = p * (d - kl[:, None]) if want_grad else None
    return kl, g


def widen(values: np.ndarray, dtype: int) -> np.ndarray:
    """Logit storage (uint16 bf16 bit patterns, float32, or float64 for
    tests) to float64, exactly."""
    if dtype == O.DTYPE_F64:
        return np.asarray(values, np.float64)
    if dtype == O.DTYPE_BF16:
        return (np.asarray(values).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(values, np.float32).astype(np.float64)


def fwd_bwd_topk(traj_id, turn_id, loss_mask, alpha: float, max_turns: int, student_at,
                 teacher_ids: np.ndarray, teacher_vals: np.ndarray, dtype: int,
                 grad_scale: float = 1.0, chunk_rows: int = 4096, support_floor: int = 0,
                 support_frac: float = 0.0, success=None) -> O.Result:
    """Reference for one call of the top-K path.

    student_at(rows, ids) -> student logits [len(rows), K] at those ids (in
    the storage dtype); teacher_ids, teacher_vals: [N, K] (int, float).  The
    returned Result's grads map each supervised row to its unweighted
    gradient on the support, ordered as teacher_ids[row].  support_floor,
    support_frac and success act as in the full-vocabulary oracle."""
    traj_id = np.asarray(traj_id)
    loss_mask = np.asarray(loss_mask)
    n = int(traj_id.shape[0])
    seg = O.segments(traj_id, turn_id, loss_mask, max_turns, success)
    if seg.status != O.OK:
        return O.Result(seg.status, seg, np.zeros(n), np.zeros(n), (np.nan,) * 3,
                        np.zeros(max_turns, O.STAT_DTYPE), {})
    w = O.token_weights(seg, n, loss_mask, alpha, support_floor, support_frac)
    w0 = O.token_weights(seg, n, loss_mask, 0.0, support_floor, support_frac)
    w1 = O.token_weights(seg, n, loss_mask, 1.0, support_floor, support_frac)
    kl = np.zeros(n, np.float64)
    lse = np.full((n, 2), np.nan)
    grads = {}
    sup = np.nonzero(loss_mask)[0]
    for k0 in range(0, sup.shape[0], chunk_rows):
        rows = sup[k0:k0 + chunk_rows]
        ids = np.asarray(teacher_ids[rows], np.int64)
        a = widen(student_at(rows, ids), dtype)
        b = np.asarray(teacher_vals[rows], np.float64)
        k_, g = topk_row_kl(a, b)
        kl[rows] = k_
        lse[rows] = support_lse(a, b)
        for j, r in enumerate(rows.tolist()):
            grads[r] = g[j]
    stats = O.turn_stats([(seg, loss_mask, kl, w)], max_turns)
    return O.Result(O.OK, seg, w, kl, O.losses(w, w0, w1, kl), stats, grads,
                    O.outcome_split(seg, loss_mask, kl, w, max_turns), lse)
