"""Seeded random configurations of the fused call against the oracle: vocabulary
(vector and scalar paths), dtype, tiling, padded row stride, alpha, the sign
and size of grad_scale, in-place gradient, turn-support floor and outcome
split, and the optional per-token weights and log-partition functions, all at
once.  Every row, gradient and statistic is compared."""
import numpy as np
import pytest
import torch

from gpu_support import (check_grad_rows, check_loss, check_segments, check_stats,
                         check_token_kl, check_token_lse, check_token_weights, ids_to_device, log,
                         to_device_logits)
from oracle import turnkl_oracle as O
from paper_2607_05804_amd import turnkl as T
from test_gpu_edges import make_batch

pytestmark = pytest.mark.gpu

N_CASES = 128


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
    per_token = rng.uniform() < 0.5
    return dict(seed=6000 + k, dtype=dtype, V=V, vpt=vpt, ld=ld, alpha=alpha,
                grad_scale=grad_scale, in_place=in_place, floor=floor, frac=frac,
                outcome=outcome, n_traj=n_traj, max_turns=max_turns, per_token=per_token)


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
    extra = {}
    if c["per_token"]:
        extra = dict(token_weights=torch.empty(n, dtype=torch.float32, device="cuda"),
                     token_lse=torch.empty((n, 2), dtype=torch.float32, device="cuda"))
    T.set_row_tiling(c["vpt"])
    try:
        loss, g, _, kl, ws = T.fwd_bwd(
            zs, zt, turn_d, traj_d, mask_d, c["alpha"], grad_scale=c["grad_scale"],
            grad="inplace" if c["in_place"] else "new", max_turns=c["max_turns"],
            turn_stats=stats, token_kl=True, support_floor=c["floor"], support_frac=c["frac"],
            success=None if succ is None else torch.from_numpy(succ).cuda(), outcome_stats=ostats,
            **extra)
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
    if extra:
        check_token_weights(extra["token_weights"], ref.w, mask)
        check_token_lse(extra["token_lse"], ref.lse, mask)
    if c["in_place"]:
        assert g.data_ptr() == zs.data_ptr()
    check_grad_rows(g, ref, c["grad_scale"], rows, mask)


N_TOPK_CASES = 48


@pytest.mark.parametrize("k", range(N_TOPK_CASES))
def test_random_topk_configuration(k, gpu):
    from oracle import topk_oracle as K
    rng = np.random.default_rng(7000 + k)
    dtype = "bf16" if rng.uniform() < 0.7 else "f32"
    V = int(rng.choice([64, 1000, 1001, 4096, 32000]))
    kk = int(min(V, rng.choice([1, 7, 50, 64, 65, 200])))
    alpha = float(rng.choice([0.0, 1.0, rng.uniform()]))
    grad_scale = float(rng.choice([1.0, -2.0]))
    mode = str(rng.choice(["new", "inplace", "none"]))
    floor = int(rng.choice([0, 2, 8]))
    outcome = rng.uniform() < 0.5
    max_turns = int(rng.integers(1, 8))
    log(f"topk fuzz {k}: {dtype} V={V} K={kk} alpha={alpha} scale={grad_scale} {mode} "
        f"floor={floor} outcome={outcome}")
    traj, turn, mask, zs_h, zt_h = make_batch(7100 + k, n_traj=int(rng.integers(1, 7)),
                                              max_turns=max_turns, V=V, dtype=dtype, max_len=20)
    zt_f = (zt_h.astype(np.uint32) << 16).view(np.float32) if dtype == "bf16" else zt_h
    order = np.argsort(-zt_f, axis=1, kind="stable")[:, :kk]
    order = np.take_along_axis(order, np.argsort(rng.random(order.shape), axis=1), axis=1)
    ids = order.astype(np.int32)
    vals = np.take_along_axis(zt_f, order, axis=1).astype(np.float32)
    succ = None
    if outcome:
        succ = rng.integers(0, 2, int(traj.max()) + 2)[np.maximum(traj, 0)].astype(np.uint8)
    zs = to_device_logits(zs_h)
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask)
    stats = T.new_turn_stats(max_turns)
    ostats = T.new_turn_stats(2 * max_turns) if outcome else None
    loss, g, gk, _, kl, ws = T.fwd_bwd_topk(
        zs, torch.from_numpy(ids).cuda(), torch.from_numpy(vals).cuda(), turn_d, traj_d, mask_d,
        alpha, grad_scale=grad_scale, grad=None if mode == "none" else mode, grad_topk=True,
        max_turns=max_turns, turn_stats=stats, token_kl=True, support_floor=floor,
        success=None if succ is None else torch.from_numpy(succ).cuda(), outcome_stats=ostats)
    torch.cuda.synchronize()
    dt = O.DTYPE_BF16 if dtype == "bf16" else O.DTYPE_F32
    ref = K.fwd_bwd_topk(traj, turn, mask, alpha, max_turns,
                         lambda rows, i: np.take_along_axis(zs_h[rows], i, axis=1), ids, vals, dt,
                         grad_scale, support_floor=floor, success=succ)
    assert ref.status == O.OK
    check_segments(ws, ref.seg)
    check_loss(loss, ref.loss)
    check_token_kl(kl, ref.kl, mask)
    check_stats(stats, ref.stats)
    if outcome:
        half = 48 * max_turns
        check_stats(ostats[:half], ref.outcome_stats[0])
        check_stats(ostats[half:], ref.outcome_stats[1])
    gk_h = gk.cpu().numpy().astype(np.float64)
    dense = None
    if g is not None:
        dense = g.float().cpu().numpy().astype(np.float64)
    bf16_dense = dtype == "bf16"
    for r in range(len(traj)):
        if not mask[r]:
            assert np.all(gk_h[r] == 0.0)
            if dense is not None:
                assert np.all(dense[r] == 0.0)
            continue
        want = grad_scale * ref.w[r] * ref.grads[r]
        assert np.all(np.abs(gk_h[r] - want) <= 1e-4 * np.abs(want) + 2e-6 * abs(grad_scale * ref.w[r])), r
        if dense is not None:
            row = dense[r]
            tol = (2.0 ** -8 * np.abs(want) + 2e-5 * abs(grad_scale * ref.w[r])) if bf16_dense else \
                (1e-4 * np.abs(want) + 2e-6 * abs(grad_scale * ref.w[r]))
            assert np.all(np.abs(row[ids[r]] - want) <= tol), r
            off = np.ones(V, bool)
            off[ids[r]] = False
            assert np.all(row[off] == 0.0), r
