"""Parity of the turn-support floor (App. D's internal-blend n_min) and of the
per-outcome statistics (Sec. 4.2) on the HIP path with the CPU oracle, for
the full-vocabulary and the top-K entry points, through the C ABI."""
import numpy as np
import pytest
import torch

import synth
from gpu_support import (check_grad_every_row_on_device, check_grad_rows,
                         check_grad_rows_batched, check_loss, check_segments, check_stats,
                         check_token_kl, device_row_source, ids_to_device, log, oracle_dtype,
                         sample_rows, to_device_logits)
from oracle import diagnostics as D
from oracle import topk_oracle as K
from oracle import turnkl_oracle as O
from paper_2607_05804_amd import turnkl as T
from test_gpu_edges import make_batch

pytestmark = pytest.mark.gpu


def _flags(traj, seed):
    """Per-token outcome flags, one random draw per trajectory (padding: random)."""
    rng = np.random.default_rng(seed)
    per = rng.integers(0, 2, int(traj.max()) + 2)
    f = per[np.maximum(traj, 0)].astype(np.uint8)
    pad = traj < 0
    f[pad] = rng.integers(0, 2, int(pad.sum())).astype(np.uint8)  # ignored by both sides
    return f


def _call(zs, zt, traj, turn, mask, alpha, max_turns, floor, frac, succ=None, grad="new",
          stats=None, ostats=None, accumulate=False):
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
    stats = T.new_turn_stats(max_turns) if stats is None else stats
    s_d = None
    if succ is not None:
        s_d = torch.from_numpy(succ).cuda()
        ostats = T.new_turn_stats(2 * max_turns) if ostats is None else ostats
    loss, g, _, kl, ws = T.fwd_bwd(zs, zt, turn_d, traj_d, mask_d, alpha, grad=grad,
                                   max_turns=max_turns, turn_stats=stats, token_kl=True,
                                   accumulate_stats=accumulate, support_floor=floor,
                                   support_frac=frac, success=s_d, outcome_stats=ostats)
    torch.cuda.synchronize()
    return loss, g, stats, kl, ws, ostats


def _check_outcome(ostats, ref_split, max_turns):
    half = 48 * max_turns
    check_stats(ostats[:half], ref_split[0])
    check_stats(ostats[half:], ref_split[1])


@pytest.mark.parametrize("floor,frac,dtype,V", [(2, 0.3, "bf16", 1000), (8, 0.15, "bf16", 4096),
                                                (3, 0.5, "f32", 3000), (99, 0.0, "bf16", 2048),
                                                (1, 0.0, "f32", 1000)])
def test_floor_and_outcome_parity(floor, frac, dtype, V, gpu):
    traj, turn, mask, zs_h, zt_h = make_batch(900 + floor, n_traj=14, max_turns=8, V=V,
                                              dtype=dtype, max_len=24)
    succ = _flags(traj, floor)
    log(f"floor={floor} frac={frac} {dtype} V={V} N={len(traj)}")
    zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    loss, g, stats, kl, ws, ostats = _call(zs, zt, traj, turn, mask, 0.6, 8, floor, frac, succ)
    rows = list(range(len(traj)))
    dt = O.DTYPE_BF16 if dtype == "bf16" else O.DTYPE_F32
    ref = O.fwd_bwd(traj, turn, mask, 0.6, 8, lambda r: (zs_h[r], zt_h[r]), dt, 1.0, rows,
                    support_floor=floor, support_frac=frac, success=succ)
    assert ref.status == O.OK
    check_segments(ws, ref.seg)
    check_loss(loss, ref.loss)
    check_token_kl(kl, ref.kl, mask)
    check_stats(stats, ref.stats)
    _check_outcome(ostats, ref.outcome_stats, 8)
    worst = check_grad_rows(g, ref, 1.0, rows, mask)
    surv = O.turn_survivors(ref.seg, 8)
    log(f"  survivors={surv.tolist()} loss gpu={loss.tolist()} ref={ref.loss} grad err={worst:.1e}")


def test_floor_off_forms_are_bit_identical_to_the_plain_call(gpu):
    """floor 0 / frac 0 (no floor) and floor 1 (every supervised turn valid,
    through the floor's kernels) reproduce the call without options bit for
    bit; so does an outcome split (it adds statistics only)."""
    traj, turn, mask, zs_h, zt_h = make_batch(950, n_traj=9, max_turns=6, V=2048)
    zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    base = _call(zs, zt, traj, turn, mask, 0.35, 6, 0, 0.0)
    for floor, frac, succ in ((0, 0.0, None), (1, 0.0, None), (0, 1e-9, None),
                              (0, 0.0, _flags(traj, 3))):
        got = _call(zs, zt, traj, turn, mask, 0.35, 6, floor, frac, succ)
        assert torch.equal(got[0], base[0]), (floor, frac)
        assert torch.equal(got[1].view(torch.int16), base[1].view(torch.int16))
        assert torch.equal(got[2], base[2]) and torch.equal(got[3], base[3])


def test_no_valid_turn_makes_the_turn_loss_the_trajectory_loss(gpu):
    traj, turn, mask, zs_h, zt_h = make_batch(951, n_traj=6, max_turns=5, V=1000)
    zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    loss, g, *_ = _call(zs, zt, traj, turn, mask, 0.8, 5, 1000, 0.0)
    l0, g0, *_ = _call(zs, zt, traj, turn, mask, 0.0, 5, 0, 0.0)
    lb, lt, lu = loss.tolist()
    assert lu == lt and lb == pytest.approx(lt, rel=1e-6)
    assert l0[1].item() == lt
    # every weight falls back to alpha = 0: the gradients agree to rounding
    d = (g.float() - g0.float()).abs().max().item()
    assert d <= 2 ** -8 * g0.float().abs().max().item()


def test_outcome_statistics_accumulate_over_micro_batches(gpu):
    parts_all, parts = [], []
    stats = T.new_turn_stats(7)
    ostats = T.new_turn_stats(14)
    for k in range(3):
        traj, turn, mask, zs_h, zt_h = make_batch(960 + k, n_traj=5, max_turns=7, V=1000)
        succ = _flags(traj, 40 + k)
        zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
        _call(zs, zt, traj, turn, mask, 0.5, 7, 2, 0.25, succ, grad=None, stats=stats,
              ostats=ostats, accumulate=k > 0)
        ref = O.fwd_bwd(traj, turn, mask, 0.5, 7, lambda r: (zs_h[r], zt_h[r]), O.DTYPE_BF16,
                        support_floor=2, support_frac=0.25, success=succ)
        parts.append((ref.seg, mask, ref.kl, ref.w))
    want = O.turn_stats(parts, 7)
    check_stats(stats, want)
    for f in (0, 1):
        check_stats(ostats[48 * 7 * f:48 * 7 * (f + 1)], O.turn_stats(parts, 7, outcome=f))


def test_outcome_flag_errors(gpu):
    z = lambda *a: np.array(a, np.int32)
    m = lambda *a: np.array(a, np.uint8)
    V = 256
    rng = np.random.default_rng(5)

    def run(traj, turn, mask, succ):
        n = len(traj)
        zs = to_device_logits(rng.normal(0, 1, (n, V)).astype(np.float32))
        turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
        o = T.new_turn_stats(2 * 4)
        try:
            T.fwd_bwd(zs, zs, turn_d, traj_d, mask_d, 0.5, max_turns=4,
                      success=torch.from_numpy(succ).cuda(), outcome_stats=o)
        except T.TurnKLError as e:
            return e.code
        return T.OK

    assert run(z(0, 0, 0), z(0, 0, 0), m(1, 1, 1), m(1, 1, 0)) == T.ERR_OUTCOME
    assert run(z(0, 0, 1), z(0, 1, 0), m(1, 1, 1), m(1, 0, 0)) == T.ERR_OUTCOME
    assert run(z(0, 0, 1), z(0, 1, 0), m(1, 1, 1), m(1, 7, 0)) == T.OK
    assert run(z(0, -1, 0), z(0, 0, 1), m(1, 0, 1), m(1, 0, 1)) == T.OK
    assert run(z(0, 0, 0), z(1, 1, 0), m(1, 1, 1), m(1, 1, 0)) == T.ERR_UNSORTED
    assert run(z(0, 0), z(0, 9), m(1, 1), m(1, 0)) == T.ERR_TURN_RANGE
    assert run(z(0, 0, 0), z(0, 0, 9), m(1, 1, 1), m(1, 0, 1)) == T.ERR_OUTCOME
    # the oracle reports the same codes on the same inputs
    assert O.segments(z(0, 0, 0), z(0, 0, 9), m(1, 1, 1), 4, m(1, 0, 1)).status == O.ERR_OUTCOME


def test_topk_floor_and_outcome_parity(gpu):
    traj, turn, mask, zs_h, zt_h = make_batch(970, n_traj=12, max_turns=8, V=4096, max_len=24)
    succ = _flags(traj, 9)
    zt_f = (zt_h.astype(np.uint32) << 16).view(np.float32)
    ids = np.argsort(-zt_f, axis=1, kind="stable")[:, :50].astype(np.int32)
    vals = np.take_along_axis(zt_f, ids.astype(np.int64), axis=1).astype(np.float32)
    zs = to_device_logits(zs_h)
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
    stats, ostats = T.new_turn_stats(8), T.new_turn_stats(16)
    loss, g, gk, _, kl, ws = T.fwd_bwd_topk(
        zs, torch.from_numpy(ids).cuda(), torch.from_numpy(vals).cuda(), turn_d, traj_d, mask_d,
        0.7, grad_topk=True, max_turns=8, turn_stats=stats, token_kl=True, support_floor=3,
        support_frac=0.2, success=torch.from_numpy(succ).cuda(), outcome_stats=ostats)
    torch.cuda.synchronize()
    ref = K.fwd_bwd_topk(traj, turn, mask, 0.7, 8,
                         lambda rows, i: np.take_along_axis(zs_h[rows], i, axis=1), ids, vals,
                         O.DTYPE_BF16, support_floor=3, support_frac=0.2, success=succ)
    check_segments(ws, ref.seg)
    check_loss(loss, ref.loss)
    check_token_kl(kl, ref.kl, mask)
    check_stats(stats, ref.stats)
    _check_outcome(ostats, ref.outcome_stats, 8)
    gk_h = gk.cpu().numpy().astype(np.float64)
    for r in np.nonzero(mask)[0]:
        want = ref.w[r] * ref.grads[int(r)]
        assert np.all(np.abs(gk_h[r] - want) <= 1e-4 * np.abs(want) + 2e-6 * ref.w[r]), r


def test_long_horizon_full_size_with_the_paper_floor(gpu):
    """65,536 tokens x V = 151,936 bf16 with App. D's floor (8, 0.15): n_min =
    8 over 30 trajectories leaves the deepest turns invalid.  Loss, per-token
    KL, both statistics over every row; every gradient row on the device and
    1,000 supervised rows against the oracle, half of them at invalid turns."""
    w = synth.make("long_horizon")
    zs, zt = w.device_logits()
    succ = (w.traj_id % 2 == 0).astype(np.uint8)
    ref = O.fwd_bwd(w.traj_id, w.turn_id, w.loss_mask, 0.5, w.max_turns,
                    device_row_source(zs, zt), oracle_dtype(zs.dtype), 1.0,
                    support_floor=8, support_frac=0.15, success=succ)
    log(f"  oracle done: loss={ref.loss}")
    surv = O.turn_survivors(ref.seg, w.max_turns)
    assert (surv[surv > 0] < 8).any()  # the floor removes some turns
    loss, g, stats, kl, ws, ostats = _call(zs, zt, w.traj_id, w.turn_id, w.loss_mask, 0.5,
                                           w.max_turns, 8, 0.15, succ)
    check_segments(ws, ref.seg)
    check_loss(loss, ref.loss)
    check_token_kl(kl, ref.kl, w.loss_mask)
    check_stats(stats, ref.stats)
    _check_outcome(ostats, ref.outcome_stats, w.max_turns)
    check_grad_every_row_on_device(g, w.loss_mask, ref.w, 1.0)
    # supervised rows at turns the floor invalidates (their weights keep only
    # the trajectory term) and others, from both ends of the ticket order
    sup = np.nonzero(w.loss_mask)[0]
    invalid = np.isin(w.turn_id[sup], np.nonzero((surv > 0) & (surv < 8))[0])
    rng = np.random.default_rng(3)
    pick = lambda a, k: a if a.size <= k else rng.choice(a, k, replace=False)
    rows = np.union1d(np.union1d(pick(sup[invalid], 500), pick(sup[~invalid], 400)),
                      np.concatenate([sup[:50], sup[-50:]]))
    worst = check_grad_rows_batched(g, ref.w, 1.0, rows, device_row_source(zs, zt),
                                    oracle_dtype(zs.dtype))
    log(f"  loss gpu={loss.tolist()} ref={ref.loss} {rows.size} oracle rows "
        f"({int(invalid.sum())} supervised tokens at invalid turns) grad err={worst:.1e}")
    # the host diagnostics on the device statistics agree with the oracle's
    # diagnostics on the oracle's statistics
    n_b = int(np.unique(w.traj_id[(w.traj_id >= 0) & (w.loss_mask > 0)]).size)
    got = T.budget_report(stats, n_b, 8, 0.15)
    want = D.budget_report(ref.stats, n_b, 8, 0.15)
    assert (got["n_min"], got["prefix"], got["third"]) == (want.n_min, want.prefix, want.third)
    for k in ("shallow_budget", "deep_budget", "deep_support", "deep_shallow_kl"):
        assert abs(got[k] - getattr(want, k)) <= 1e-4 * abs(getattr(want, k)) + 1e-7, k
    np.testing.assert_allclose(T.loss_share(stats), D.loss_share(ref.stats), rtol=1e-4, atol=1e-8)
    gap = T.outcome_gap(ostats)
    want_gap = D.outcome_gap(ref.outcome_stats)
    np.testing.assert_array_equal(np.isnan(gap), np.isnan(want_gap))
    ok = ~np.isnan(want_gap)
    np.testing.assert_allclose(gap[ok], want_gap[ok], rtol=1e-3, atol=1e-5)
    log(f"  budget {got}")
    del zs, zt, g
    torch.cuda.empty_cache()
