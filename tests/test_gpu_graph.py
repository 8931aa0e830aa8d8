"""The fused call captured in a HIP graph: every replay equals the eager
call bit for bit (the library enqueues only kernels, allocates nothing and
never synchronises on the success path, and resets its ticket and exchange
state with kernels, so a captured call can be replayed)."""
import numpy as np
import pytest
import torch

import synth
from gpu_support import ids_to_device, log, to_device_logits
from paper_2607_05804_amd import turnkl as T

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("vpt,opts", [(0, False), (4, False), (0, True)])
def test_graph_replays_equal_eager(vpt, opts, gpu):
    w = synth.make("agent")
    zs_h, zt_h = w.host_logits(0, w.n_tokens)
    zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    turn, traj, mask = ids_to_device(w.traj_id, w.turn_id, w.loss_mask)
    n, V = zs.shape
    T.set_row_tiling(vpt)
    try:
        ws = T.Workspace(n, V, T.BF16, w.max_turns)
        grad = torch.empty_like(zs)
        kl = torch.empty(n, dtype=torch.float32, device=gpu)
        stats = T.new_turn_stats(w.max_turns)
        kw = {}
        if opts:  # turn-support floor and outcome split
            kw = dict(support_floor=8, support_frac=0.15,
                      success=torch.from_numpy((w.traj_id % 2).astype(np.uint8)).to(gpu),
                      outcome_stats=T.new_turn_stats(2 * w.max_turns))
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            # eager reference on the side stream
            loss, _, _, _, _ = T.fwd_bwd(zs, zt, turn, traj, mask, 0.3, grad=grad,
                                         max_turns=w.max_turns, turn_stats=stats, token_kl=kl,
                                         workspace=ws, check=False, **kw)
            s.synchronize()
            ref = (loss.clone(), grad.clone(), kl.clone(), stats.clone(),
                   kw["outcome_stats"].clone() if opts else None)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s):
                loss_g, _, _, _, _ = T.fwd_bwd(zs, zt, turn, traj, mask, 0.3, grad=grad,
                                               max_turns=w.max_turns, turn_stats=stats,
                                               token_kl=kl, workspace=ws, check=False, **kw)
        torch.cuda.current_stream().wait_stream(s)
        for r in range(4):
            grad.fill_(7)  # eager work between replays
            kl.zero_()
            stats.fill_(5)
            if opts:
                kw["outcome_stats"].fill_(3)
            g.replay()
            torch.cuda.synchronize()
            assert ws.status() == T.OK
            assert torch.equal(loss_g, ref[0]), r
            assert torch.equal(grad.view(torch.int16), ref[1].view(torch.int16)), r
            assert torch.equal(kl, ref[2]), r
            assert torch.equal(stats, ref[3]), r
            if opts:
                assert torch.equal(kw["outcome_stats"], ref[4]), r
        log(f"graph replays ok (vpt={vpt}, options={opts}): loss={loss_g.tolist()}")
    finally:
        T.set_row_tiling(0)


def test_topk_graph_replays_equal_eager(gpu):
    """The top-K call (support rows, dense zero-fill, scatter) captured in a
    graph: every replay equals the eager call bit for bit."""
    w = synth.make("agent")
    zs_h, zt_h = w.host_logits(0, w.n_tokens)
    zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    top_v, top_i = torch.topk(zt.float(), 50, dim=1)
    ids, vals = top_i.to(torch.int32).contiguous(), top_v.contiguous()
    turn, traj, mask = ids_to_device(w.traj_id, w.turn_id, w.loss_mask)
    n, V = zs.shape
    ws = T.TopkWorkspace(n, 50, w.max_turns)
    grad = torch.empty_like(zs)
    gk = torch.empty((n, 50), dtype=torch.float32, device=gpu)
    stats = T.new_turn_stats(w.max_turns)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        loss, *_ = T.fwd_bwd_topk(zs, ids, vals, turn, traj, mask, 0.4, grad=grad, grad_topk=gk,
                                  max_turns=w.max_turns, turn_stats=stats, workspace=ws,
                                  check=False)
        s.synchronize()
        ref = (loss.clone(), grad.clone(), gk.clone(), stats.clone())
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            loss_g, *_ = T.fwd_bwd_topk(zs, ids, vals, turn, traj, mask, 0.4, grad=grad,
                                        grad_topk=gk, max_turns=w.max_turns, turn_stats=stats,
                                        workspace=ws, check=False)
    torch.cuda.current_stream().wait_stream(s)
    for r in range(4):
        grad.fill_(7)
        gk.fill_(3)
        stats.fill_(5)
        g.replay()
        torch.cuda.synchronize()
        assert ws.status() == T.OK
        assert torch.equal(loss_g, ref[0]), r
        assert torch.equal(grad.view(torch.int16), ref[1].view(torch.int16)), r
        assert torch.equal(gk, ref[2]) and torch.equal(stats, ref[3]), r
    log(f"top-K graph replays ok: loss={loss_g.tolist()}")


def test_graph_replays_follow_the_mask(gpu):
    """The bf16 row kernel's load order is chosen on the device from the
    supervised share of the rows, so one captured call replayed with a mixed
    mask and with every row supervised (written into the same mask buffer
    between replays) equals the eager call for each mask, bit for bit."""
    w = synth.make("agent")
    zs_h, zt_h = w.host_logits(0, w.n_tokens)
    zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    turn, traj, mask = ids_to_device(w.traj_id, w.turn_id, w.loss_mask)
    masks = [mask.clone(), (traj >= 0).to(torch.uint8)]
    assert masks[0].float().mean().item() < 0.9 and masks[1].float().mean().item() > 0.9
    n, V = zs.shape
    ws = T.Workspace(n, V, T.BF16, w.max_turns)
    grad = torch.empty_like(zs)
    kl = torch.empty(n, dtype=torch.float32, device=gpu)
    stats = T.new_turn_stats(w.max_turns)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    refs = []
    with torch.cuda.stream(s):
        for m in masks:
            mask.copy_(m)
            loss, *_ = T.fwd_bwd(zs, zt, turn, traj, mask, 0.3, grad=grad, max_turns=w.max_turns,
                                 turn_stats=stats, token_kl=kl, workspace=ws, check=False)
            s.synchronize()
            assert ws.status() == T.OK
            refs.append((loss.clone(), grad.clone(), kl.clone(), stats.clone()))
        mask.copy_(masks[0])
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            loss_g, *_ = T.fwd_bwd(zs, zt, turn, traj, mask, 0.3, grad=grad,
                                   max_turns=w.max_turns, turn_stats=stats, token_kl=kl,
                                   workspace=ws, check=False)
    torch.cuda.current_stream().wait_stream(s)
    for r in range(6):
        k = r % 2
        mask.copy_(masks[k])  # eager work between replays
        grad.fill_(7)
        kl.zero_()
        stats.fill_(5)
        g.replay()
        torch.cuda.synchronize()
        assert ws.status() == T.OK
        ref = refs[k]
        assert torch.equal(loss_g, ref[0]), r
        assert torch.equal(grad.view(torch.int16), ref[1].view(torch.int16)), r
        assert torch.equal(kl, ref[2]) and torch.equal(stats, ref[3]), r
    log(f"graph replays follow the mask: losses {[x[0].tolist() for x in refs]}")
