"""Seeded random configurations of the fused call against the oracle: vocabulary
(vector and scalar paths), dtype, tiling, padded row stride, alpha, the sign
and size of grad_scale, in-place gradient, turn-support floor and outcome
split, all at once.  Every row, gradient and statistic is compared."""
import numpy as np
import pytest
import torch

from gpu_support import (check_grad_rows, check_loss, check_segments, check_stats,
                         check_token_kl, ids_to_device, log, to_device_logits)
from oracle import turnkl_oracle as O
from paper_2607_05804_amd import turnkl as T
from test_gpu_edges import make_batch

pytestmark = pytest.mark.gpu

N_CASES = 64


def _case(k):
    rng = np.random.default_rng(5000 + k)
    dtype = "bf16" if rng.uniform() < 0.6 else "f32"
    V = int(rng.choice([8, 24, 1000, 1001, 2048, 4392, 8240, 12296, 17003, 20000]))
    vpt = int(rng.choice([0, 0, 1, 2, 3, 5, 9, 13, 25]))
    ld = None if rng.uniform() < 0.7 else V + int(rng.choice([1, 8, 64]))
    alpha = float(rng.choice([0.0, 1.0, rng.uniform()]))
    grad_scale = float(rng.choice([1.0, -0.5, 3.0, 1e-3]))
    in_place = ld is None and rng.uniform() < 0.3
    floor = int(rng.choice([0, 0, 2, 8]))
    frac = float(rng.choice([0.0, 0.15, 0.5]))
    outcome = rng.uniform() < 0.5
    n_traj = int(rng.integers(1, 9))
    max_turns = int(rng.integers(1, 9))
    return dict(seed=6000 + k, dtype=dtype, V=V, vpt=vpt, ld=ld, alpha=alpha,
                grad_scale=grad_scale, in_place=in_place, floor=floor, frac=frac,
                outcome=outcome, n_traj=n_traj, max_turns=max_turns)


def _device(h, ld):
    if ld is None:
        return to_device_logits(h)
    full = torch.full((h.shape[0], ld), float("nan"), dtype=torch.float32, device="cuda")
    if h.dtype == np.uint16:
        full = full.to(torch.bfloat16)
    full[:, :h.shape[1]] = to_device_logits(h)
    return full[:, :h.shape[1]]


@pytest.mark.parametrize("k", range(N_CASES))
def test_random_configuration(k, gpu):
    c = _case(k)
    log(f"fuzz {k}: {c}")
    traj, turn, mask, zs_h, zt_h = make_batch(c["seed"], n_traj=c["n_traj"],
                                              max_turns=c["max_turns"], V=c["V"],
                                              dtype=c["dtype"], max_len=20)
    n = len(traj)
    rng = np.random.default_rng(c["seed"])
    succ = None
    if c["outcome"]:
        per = rng.integers(0, 2, int(traj.max()) + 2)
        succ = per[np.maximum(traj, 0)].astype(np.uint8)
    zs, zt = _device(zs_h, c["ld"]), _device(zt_h, c["ld"])
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
    stats = T.new_turn_stats(c["max_turns"])
    ostats = T.new_turn_stats(2 * c["max_turns"]) if succ is not None else None
    T.set_row_tiling(c["vpt"])
    try:
        loss, g, _, kl, ws = T.fwd_bwd(
            zs, zt, turn_d, traj_d, mask_d, c["alpha"], grad_scale=c["grad_scale"],
            grad="inplace" if c["in_place"] else "new", max_turns=c["max_turns"],
            turn_stats=stats, token_kl=True, support_floor=c["floor"], support_frac=c["frac"],
            success=None if succ is None else torch.from_numpy(succ).cuda(), outcome_stats=ostats)
    finally:
        T.set_row_tiling(0)
    torch.cuda.synchronize()
    dt = O.DTYPE_BF16 if c["dtype"] == "bf16" else O.DTYPE_F32
    rows = list(range(n))
    ref = O.fwd_bwd(traj, turn, mask, c["alpha"], c["max_turns"],
                    lambda r: (zs_h[r], zt_h[r]), dt, c["grad_scale"], rows,
                    support_floor=c["floor"], support_frac=c["frac"], success=succ)
    assert ref.status == O.OK
    check_segments(ws, ref.seg)
    check_loss(loss, ref.loss)
    check_token_kl(kl, ref.kl, mask)
    check_stats(stats, ref.stats)
    if succ is not None:
        half = 48 * c["max_turns"]
        check_stats(ostats[:half], ref.outcome_stats[0])
        check_stats(ostats[half:], ref.outcome_stats[1])
    if c["in_place"]:
        assert g.data_ptr() == zs.data_ptr()
    check_grad_rows(g, ref, c["grad_scale"], rows, mask)
