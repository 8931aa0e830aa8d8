"""The device's segment table, per-turn counts and per-token weights on
hypothesis-generated batch layouts (padding between turns and trajectories,
skipped turn ids, sparse trajectory ids, fully masked turns and
trajectories, trailing padding), through the C ABI, against the oracle:
bit-exact for the integer tables, one float rounding for the weights."""
import numpy as np
import pytest
import torch
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from gpu_support import check_loss, check_segments, check_token_weights, ids_to_device
from oracle import turnkl_oracle as O
from paper_2607_05804_amd import turnkl as T
from test_oracle_hypothesis import _layout, build

pytestmark = pytest.mark.gpu

V = 8


@settings(max_examples=120, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.function_scoped_fixture])
@given(layout=_layout, tail=st.integers(0, 3), alpha=st.floats(0.0, 1.0),
       floor=st.integers(0, 4))
def test_segments_counts_and_weights_on_generated_layouts(gpu, layout, tail, alpha, floor):
    traj, turn, mask, max_turns = build(layout, tail)
    n = len(traj)
    rng = np.random.default_rng(n)
    zs = rng.normal(0.0, 3.0, (n, V)).astype(np.float32)
    zt = (zs + rng.normal(0.0, 1.0, zs.shape)).astype(np.float32)
    zs_d = torch.from_numpy(zs).to(gpu)
    zt_d = torch.from_numpy(zt).to(gpu)
    turn_d, traj_d, mask_d = ids_to_device(traj, turn, mask, gpu)
    stats = T.new_turn_stats(max_turns)
    w_d = torch.empty(n, dtype=torch.float32, device=gpu)
    loss, _, _, _, ws = T.fwd_bwd(zs_d, zt_d, turn_d, traj_d, mask_d, alpha, grad=None,
                                  max_turns=max_turns, turn_stats=stats, support_floor=floor,
                                  token_weights=w_d)
    torch.cuda.synchronize()
    ref = O.fwd_bwd(traj, turn, mask, alpha, max_turns, lambda r: (zs[r], zt[r]), O.DTYPE_F32,
                    support_floor=floor)
    assert ref.status == O.OK
    check_segments(ws, ref.seg)
    got = T.read_turn_stats(stats)
    assert np.array_equal(got["n_tokens"], ref.stats["n_tokens"])
    assert np.array_equal(got["n_traj"], ref.stats["n_traj"])
    check_token_weights(w_d, ref.w, mask)
    check_loss(loss, ref.loss)
