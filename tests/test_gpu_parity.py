"""Parity of the HIP path with the CPU oracle on the five seeded workloads.

The two small workloads are generated on the host and compared everywhere
(every row's KL, every gradient row of the tiny batch, sampled gradient rows
of the 4k-token batch).  The three vocabulary-151,936 workloads are generated
in HBM at full size and run with the launch configuration bench.py times; the
oracle reads every supervised row (copied from the generator's output before
the call) for the loss, the per-token KL and the per-turn statistics.  The
gradient is checked on every row on the device (unsupervised rows exactly
zero, supervised rows summing to zero as dKL/dz_s does) and against the
oracle element by element on 1,000 supervised rows per workload: the first
and the last 100 in token order, which are the two ends of the row kernel's
ticket order, and 800 more at random, each row covering all of its chunks.
"""
import numpy as np
import pytest
import torch

import synth
from gpu_support import (check_grad_every_row_on_device, check_grad_rows,
                         check_grad_rows_batched, check_loss, check_segments, check_stats,
                         check_token_kl, check_token_lse, check_token_weights, device_row_source,
                         ids_to_device, log, oracle_dtype, rows_bits_to_host,
                         ticket_order_rows, to_device_logits)
from oracle import turnkl_oracle as O
from paper_2607_05804_amd import turnkl as T

pytestmark = pytest.mark.gpu


def _run(zs, zt, w, alpha, grad_scale, grad="new", ws=None, **extra):
    turn, traj, mask = ids_to_device(w.traj_id, w.turn_id, w.loss_mask)
    stats = T.new_turn_stats(w.max_turns)
    loss, g, _, kl, ws = T.fwd_bwd(zs, zt, turn, traj, mask, alpha, grad_scale=grad_scale,
                                   grad=grad, max_turns=w.max_turns, turn_stats=stats,
                                   token_kl=True, workspace=ws, **extra)
    torch.cuda.synchronize()
    return loss, g, stats, kl, ws


@pytest.mark.parametrize("name,grad_scale", [("tiny", 1.0), ("agent", 0.5)])
def test_small_workloads(name, grad_scale, gpu):
    w = synth.make(name)
    alpha = w.alphas[0]
    log(f"parity {name}: N={w.n_tokens} V={w.vocab} {w.dtype} alpha={alpha}")
    zs_h, zt_h = w.host_logits(0, w.n_tokens)
    zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    loss, g, stats, kl, ws = _run(zs, zt, w, alpha, grad_scale)
    rows = list(range(w.n_tokens)) if name == "tiny" else []
    ref = O.fwd_bwd(w.traj_id, w.turn_id, w.loss_mask, alpha, w.max_turns,
                    lambda r: (zs_h[r], zt_h[r]), oracle_dtype(zs.dtype), grad_scale, rows)
    check_segments(ws, ref.seg)
    check_loss(loss, ref.loss)
    check_token_kl(kl, ref.kl, w.loss_mask)
    check_stats(stats, ref.stats)
    if rows:
        worst = check_grad_rows(g, ref, grad_scale, rows, w.loss_mask)
    else:  # every supervised row of the 4k-token batch, in batches
        worst = check_grad_rows_batched(g, ref.w, grad_scale, np.nonzero(w.loss_mask)[0],
                                        lambda r: (zs_h[r], zt_h[r]), oracle_dtype(zs.dtype))
        check_grad_every_row_on_device(g, w.loss_mask, ref.w, grad_scale)
    log(f"  loss gpu={loss.tolist()} ref={ref.loss} worst unweighted grad err={worst:.2e}")
    # every unsupervised row of the gradient is zero
    uns = np.nonzero(w.loss_mask == 0)[0]
    if uns.size:
        assert torch.count_nonzero(g[torch.from_numpy(uns).to(gpu)]).item() == 0


def _snapshot(zs, zt, rows):
    """Host copies of the listed rows, taken before any call (an in-place call
    overwrites the student logits), as an oracle row source for them."""
    rows = np.asarray(rows, np.int64)
    hs, ht = rows_bits_to_host(zs, rows), rows_bits_to_host(zt, rows)
    at = {int(r): k for k, r in enumerate(rows)}
    return lambda r: (hs[[at[int(x)] for x in r]], ht[[at[int(x)] for x in r]])


def _full_size(name, gpu, check_alphas=None):
    w = synth.make(name)
    log(f"parity {name}: N={w.n_tokens} V={w.vocab} sup={w.n_supervised} in_place={w.in_place}")
    zs, zt = w.device_logits()
    rows = ticket_order_rows(w.loss_mask, seed=1)
    host_rows = _snapshot(zs, zt, rows)
    alphas = check_alphas or w.alphas
    # oracle first: an in-place call overwrites the student logits
    ref = O.fwd_bwd(w.traj_id, w.turn_id, w.loss_mask, alphas[0], w.max_turns,
                    device_row_source(zs, zt), oracle_dtype(zs.dtype), 1.0)
    log(f"  oracle done: loss={ref.loss}")
    assert ref.status == O.OK
    ws = None
    for k, alpha in enumerate(alphas):
        last = k == len(alphas) - 1
        grad = "inplace" if (w.in_place and last) else "new"
        # the first call also returns the per-token weights and log-partition functions
        extra = {} if k else dict(
            token_weights=torch.empty(w.n_tokens, dtype=torch.float32, device=gpu),
            token_lse=torch.empty((w.n_tokens, 2), dtype=torch.float32, device=gpu))
        loss, g, stats, kl, ws = _run(zs, zt, w, alpha, 1.0, grad=grad, ws=ws, **extra)
        w_a = O.token_weights(ref.seg, w.n_tokens, w.loss_mask, alpha)
        if extra:
            check_token_weights(extra["token_weights"], w_a, w.loss_mask)
            check_token_lse(extra["token_lse"], ref.lse, w.loss_mask)
        w0 = O.token_weights(ref.seg, w.n_tokens, w.loss_mask, 0.0)
        w1 = O.token_weights(ref.seg, w.n_tokens, w.loss_mask, 1.0)
        ref_loss = O.losses(w_a, w0, w1, ref.kl)
        ref_stats = O.turn_stats([(ref.seg, w.loss_mask, ref.kl, w_a)], w.max_turns)
        check_segments(ws, ref.seg)
        check_loss(loss, ref_loss)
        check_token_kl(kl, ref.kl, w.loss_mask)
        check_stats(stats, ref_stats)
        check_grad_every_row_on_device(g, w.loss_mask, w_a, 1.0)
        # every selected row at the first alpha and in place, 64 of them otherwise
        sel = rows if (k == 0 or grad == "inplace") else rows[::len(rows) // 64]
        worst = check_grad_rows_batched(g, w_a, 1.0, sel, host_rows, oracle_dtype(zs.dtype))
        log(f"  alpha={alpha} ({grad}): loss gpu={loss.tolist()} ref={ref_loss} "
            f"{len(sel)} oracle rows, worst grad err={worst:.2e}")
        del g
    del zs, zt
    torch.cuda.empty_cache()


def test_peaked_full_size_alpha_sweep(gpu):
    _full_size("peaked", gpu)


def test_peaked_full_size_every_row_supervised(gpu):
    """The peaked batch (16,534 rows x V = 151,936) with every row supervised:
    the row kernel's alternating load order, chosen on the device when more
    than 90% of the rows are supervised, at full width against the oracle."""
    w = synth.make("peaked")
    mask_h = np.ones(w.n_tokens, np.uint8)
    log(f"parity peaked, every row supervised: N={w.n_tokens} V={w.vocab}")
    zs, zt = w.device_logits()
    rows = ticket_order_rows(mask_h, seed=2)
    ref = O.fwd_bwd(w.traj_id, w.turn_id, mask_h, w.alphas[0], w.max_turns,
                    device_row_source(zs, zt), oracle_dtype(zs.dtype), 1.0)
    assert ref.status == O.OK
    turn, traj, mask = ids_to_device(w.traj_id, w.turn_id, mask_h)
    stats = T.new_turn_stats(w.max_turns)
    loss, g, _, kl, ws = T.fwd_bwd(zs, zt, turn, traj, mask, w.alphas[0], max_turns=w.max_turns,
                                   turn_stats=stats, token_kl=True)
    torch.cuda.synchronize()
    check_segments(ws, ref.seg)
    check_loss(loss, ref.loss)
    check_token_kl(kl, ref.kl, mask_h)
    check_stats(stats, ref.stats)
    check_grad_every_row_on_device(g, mask_h, ref.w, 1.0)
    worst = check_grad_rows_batched(g, ref.w, 1.0, rows, device_row_source(zs, zt),
                                    oracle_dtype(zs.dtype))
    log(f"  loss gpu={loss.tolist()} ref={ref.loss} {len(rows)} oracle rows, "
        f"worst grad err={worst:.2e}")
    del g, zs, zt
    torch.cuda.empty_cache()


def test_long_horizon_full_size(gpu):
    _full_size("long_horizon", gpu)


def test_stress_full_size_in_place(gpu):
    _full_size("stress", gpu)
