"""The depth controller driven by the GPU path's per-turn statistics equals
the oracle controller driven by the oracle's statistics of the same probe
batch (Sec. 5.1: K_t and n_t of a probe batch feed the controller)."""
import numpy as np
import pytest
import torch

import synth
from gpu_support import ids_to_device, log, oracle_dtype, to_device_logits
from oracle import depth_controller as D
from oracle import turnkl_oracle as O
from paper_2607_05804_amd import turnkl as T

pytestmark = pytest.mark.gpu


def _success_lengths(w):
    """Turn counts of the even-numbered trajectories, standing in for the
    probe batch's successful completions."""
    out = []
    for b in np.unique(w.traj_id[w.traj_id >= 0]):
        if b % 2 == 0:
            out.append(int(np.unique(w.turn_id[w.traj_id == b]).size))
    return out


@pytest.mark.parametrize("name", ["agent", "tiny"])
def test_controller_on_gpu_stats_matches_oracle(name, gpu):
    w = synth.make(name)
    log(f"controller on {name}: N={w.n_tokens} V={w.vocab}")
    zs_h, zt_h = w.host_logits(0, w.n_tokens)
    zs, zt = to_device_logits(zs_h), to_device_logits(zt_h)
    turn, traj, mask = ids_to_device(w.traj_id, w.turn_id, w.loss_mask)
    stats = T.new_turn_stats(w.max_turns)
    T.fwd_bwd(zs, zt, turn, traj, mask, w.alphas[0], grad=None, max_turns=w.max_turns,
              turn_stats=stats)
    torch.cuda.synchronize()
    ref = O.fwd_bwd(w.traj_id, w.turn_id, w.loss_mask, w.alphas[0], w.max_turns,
                    lambda r: (zs_h[r], zt_h[r]), oracle_dtype(zs.dtype))
    succ = _success_lengths(w)
    ctl = T.DepthController(min_cov_traj=1, h_max=12)
    cfg = D.Config(min_cov_traj=1, h_max=12)
    st = D.init(cfg)
    for k in range(1, 25):
        want = D.plan(cfg, st, k)
        assert ctl.plan(k) == want
        if want[1]:
            ctl.update(stats, succ)
            st = D.update(cfg, st, list(ref.stats["kl_mean"]), list(ref.stats["n_traj"]), succ)
            s = ctl.state
            assert (s.h_eff, s.h_cov, s.h_ctrl) == (st.h_eff, st.h_cov, st.h_ctrl)
            assert abs(s.h_eff_bar - st.h_eff_bar) <= 1e-4 * max(1.0, st.h_eff_bar)
            assert abs(s.h_bar - st.h_bar) <= 1e-12 * st.h_bar
    log(f"  H_eff={ctl.state.h_eff} ({ctl.state.h_eff_bar:.4f}) H_cov={ctl.state.h_cov} "
        f"cap={ctl.plan(25)[0]}")
