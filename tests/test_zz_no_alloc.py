"""turnkl_fwd_bwd_noalloc, the fused call on the library's built-in scratch,
against turnkl_fwd_bwd on a caller workspace.

Both run the same kernels, so every output must agree bit for bit: loss,
gradient, per-token KL, weights and log-partition functions, per-turn and
per-outcome statistics.  The no-allocation calls come two in a row on one
GPU, the second with a smaller batch, so the second finds the first one's
contents in the scratch.  The batches are the long-horizon workload cut to a
few thousand tokens: vocabulary 151,936 in bf16, three chunks per row, so the
row kernel's exchange slots live in the scratch too.
"""
import numpy as np
import pytest
import torch

import synth
from gpu_support import ids_to_device, log
from paper_2607_05804_amd import turnkl as T

pytestmark = pytest.mark.gpu


def _batch(n, gpu):
    w = synth.make("long_horizon", n_tokens=n)
    zs, zt = w.device_logits(device=gpu)
    turn, traj, mask = ids_to_device(w.traj_id, w.turn_id, w.loss_mask, gpu)
    succ = torch.from_numpy((w.traj_id % 2 == 0).astype(np.uint8)).to(gpu)
    return w, zs, zt, turn, traj, mask, succ


def _outputs(w, gpu):
    n = w.n_tokens
    return dict(loss=torch.empty(3, dtype=torch.float32, device=gpu),
                grad=torch.empty((n, w.vocab), dtype=torch.bfloat16, device=gpu),
                kl=torch.empty(n, dtype=torch.float32, device=gpu),
                stats=T.new_turn_stats(w.max_turns, device=gpu),
                ostats=T.new_turn_stats(2 * w.max_turns, device=gpu),
                weights=torch.empty(n, dtype=torch.float32, device=gpu),
                lse=torch.empty((n, 2), dtype=torch.float32, device=gpu),
                status=torch.full((1,), 12345, dtype=torch.int32, device=gpu))


def _noalloc(b, out, alpha):
    w, zs, zt, turn, traj, mask, succ = b
    T.fwd_bwd_noalloc(zs, zt, turn, traj, mask, alpha, out["loss"], grad_scale=0.75,
                      grad=out["grad"], max_turns=w.max_turns, turn_stats=out["stats"],
                      token_kl=out["kl"], status=out["status"], support_floor=8,
                      support_frac=0.15, success=succ, outcome_stats=out["ostats"],
                      token_weights=out["weights"], token_lse=out["lse"])


def _with_workspace(b, out, alpha):
    w, zs, zt, turn, traj, mask, succ = b
    loss, _, _, _, ws = T.fwd_bwd(zs, zt, turn, traj, mask, alpha, grad_scale=0.75,
                                  grad=out["grad"], max_turns=w.max_turns,
                                  turn_stats=out["stats"], token_kl=out["kl"], support_floor=8,
                                  support_frac=0.15, success=succ, outcome_stats=out["ostats"],
                                  token_weights=out["weights"], token_lse=out["lse"])
    out["loss"].copy_(loss)
    out["status"].fill_(ws.status())


def _same(a, b, what):
    """Bit-for-bit equality of two output tensors (NaN where either has NaN
    must match: unsupervised rows' log-partition functions)."""
    x = a.contiguous().view(torch.uint8)
    y = b.contiguous().view(torch.uint8)
    assert torch.equal(x, y), what


def test_noalloc_matches_the_workspace_call_twice_in_a_row(gpu):
    outs = []
    batches = [_batch(3000, gpu), _batch(1100, gpu)]
    alphas = (0.5, 0.25)
    # the two no-allocation calls back to back, then the reference calls
    for b, a in zip(batches, alphas):
        log(f"noalloc: N={b[0].n_tokens} V={b[0].vocab} alpha={a}")
        out = _outputs(b[0], gpu)
        _noalloc(b, out, a)
        outs.append(out)
    torch.cuda.synchronize()
    for b, a, got in zip(batches, alphas, outs):
        ref = _outputs(b[0], gpu)
        _with_workspace(b, ref, a)
        torch.cuda.synchronize()
        assert int(got["status"].item()) == T.OK
        assert int(ref["status"].item()) == T.OK
        for k in ("loss", "grad", "kl", "stats", "ostats", "weights", "lse"):
            _same(got[k], ref[k], k)
        assert np.all(np.isfinite(got["loss"].cpu().numpy()))
        log(f"  N={b[0].n_tokens}: loss {got['loss'].tolist()} identical to the workspace call")


def test_noalloc_reports_device_errors_and_recovers(gpu):
    b = _batch(1500, gpu)
    w, zs, zt, turn, traj, mask, succ = b
    # trajectory ids out of order: swap two trajectories' ids
    bad_traj = traj.clone()
    first, last = int(w.traj_id[0]), int(w.traj_id[-1])
    bad_traj[traj == first] = last
    bad_traj[traj == last] = first
    out = _outputs(w, gpu)
    T.fwd_bwd_noalloc(zs, zt, turn, bad_traj, mask, 0.5, out["loss"], grad=out["grad"],
                      max_turns=w.max_turns, turn_stats=out["stats"], status=out["status"])
    torch.cuda.synchronize()
    assert int(out["status"].item()) == T.ERR_UNSORTED
    assert np.all(np.isnan(out["loss"].cpu().numpy()))
    # the next call on the same scratch is unaffected
    _noalloc(b, out, 0.5)
    ref = _outputs(w, gpu)
    _with_workspace(b, ref, 0.5)
    torch.cuda.synchronize()
    assert int(out["status"].item()) == T.OK
    for k in ("loss", "grad", "kl", "stats", "ostats", "weights", "lse"):
        _same(out[k], ref[k], k)
