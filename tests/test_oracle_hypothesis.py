"""Property-based pins of the oracle's segment table, weights and per-turn
statistics on hypothesis-generated batch layouts: padding between turns and
trajectories, skipped turn ids, sparse trajectory ids, fully masked turns
and trajectories.  Expected values come from pandas group-bys and an
itertools run-length walk, not from the oracle."""
import itertools

import numpy as np
import pandas as pd
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from oracle import turnkl_oracle as O

# one turn: (turn-id step >= 1, tokens, observation tokens, padding before it)
_turn = st.tuples(st.integers(1, 3), st.integers(1, 6), st.integers(0, 6), st.integers(0, 2))
# one trajectory: (trajectory-id step >= 1, its turns)
_traj = st.tuples(st.integers(1, 4), st.lists(_turn, min_size=1, max_size=6))
_layout = st.lists(_traj, min_size=0, max_size=6)


def build(layout, trailing_pad=0):
    """Token arrays of a layout, and max_turns just above its largest turn id."""
    traj, turn, mask = [], [], []
    b = -1
    top = 0
    for db, turns in layout:
        b += db
        t = -1
        for dt, n, obs, pad in turns:
            t += dt
            traj += [-1] * pad
            turn += [0] * pad
            mask += [0] * pad
            o = min(obs, n)
            traj += [b] * n
            turn += [t] * n
            mask += [0] * o + [1] * (n - o)
            top = max(top, t)
    traj += [-1] * trailing_pad
    turn += [0] * trailing_pad
    mask += [0] * trailing_pad
    return (np.array(traj, np.int32), np.array(turn, np.int32), np.array(mask, np.uint8),
            top + 1)


def runs(traj, turn, mask):
    """(start, length, trajectory, turn, supervised) of every maximal run of
    equal (trajectory, turn) that is not padding."""
    out = []
    for key, grp in itertools.groupby(range(len(traj)), key=lambda k: (int(traj[k]), int(turn[k]))):
        idx = list(grp)
        if key[0] >= 0:
            out.append((idx[0], len(idx), key[0], key[1], sum(int(mask[k]) for k in idx)))
    return out


def frame(traj, turn, mask, kl, w=None):
    keep = mask.astype(bool)
    d = {"traj": traj[keep], "turn": turn[keep], "kl": kl[keep]}
    if w is not None:
        d["w"] = w[keep]
    return pd.DataFrame(d)


_settings = settings(max_examples=150, deadline=None, derandomize=True,
                     suppress_health_check=[HealthCheck.too_slow])


@_settings
@given(_layout, st.integers(0, 3))
def test_segments_are_the_runs_of_equal_ids(layout, tail):
    traj, turn, mask, max_turns = build(layout, tail)
    seg = O.segments(traj, turn, mask, max_turns)
    assert seg.status == O.OK
    got = list(zip(seg.start.tolist(), seg.length.tolist(), seg.traj.tolist(),
                   seg.turn.tolist(), seg.n_sup.tolist()))
    assert got == runs(traj, turn, mask)
    # with max_turns one below the largest turn id plus one, that turn is out of range
    if seg.count:
        assert O.segments(traj, turn, mask, max_turns - 1).status == O.ERR_TURN_RANGE


@_settings
@given(_layout, st.floats(0.0, 1.0))
def test_weights_sum_to_one_and_give_the_paper_means(layout, alpha):
    traj, turn, mask, max_turns = build(layout)
    seg = O.segments(traj, turn, mask, max_turns)
    n = len(traj)
    w = O.token_weights(seg, n, mask, alpha)
    kl = np.random.default_rng(n).uniform(0.0, 2.0, n)
    df = frame(traj, turn, mask, kl)
    assert np.all(w[mask == 0] == 0.0)
    if df.empty:  # no supervised token: no trajectory counts, every weight is zero
        assert not w.any()
        return
    assert abs(w.sum() - 1.0) < 1e-12
    w0 = O.token_weights(seg, n, mask, 0.0)
    w1 = O.token_weights(seg, n, mask, 1.0)
    np.testing.assert_allclose(w, (1 - alpha) * w0 + alpha * w1, rtol=1e-12, atol=1e-16)
    # alpha = 0: mean over trajectories of each one's token mean (Eq. opd-rkl);
    # alpha = 1: mean over trajectories of the mean of its supervised turns' means
    l0 = df.groupby("traj")["kl"].mean().mean()
    l1 = df.groupby(["traj", "turn"])["kl"].mean().groupby(level=0).mean().mean()
    assert abs(float(np.sum(w0 * kl)) - l0) < 1e-12
    assert abs(float(np.sum(w1 * kl)) - l1) < 1e-12


@_settings
@given(_layout)
def test_turn_stats_are_group_by_moments(layout):
    traj, turn, mask, max_turns = build(layout)
    seg = O.segments(traj, turn, mask, max_turns)
    n = len(traj)
    kl = np.random.default_rng(n + 1).gamma(2.0, 0.3, n)
    w = O.token_weights(seg, n, mask, 0.5)
    stt = O.turn_stats([(seg, mask, kl, w)], max_turns)
    df = frame(traj, turn, mask, kl, w)
    for t in range(max_turns):
        d = df[df["turn"] == t]
        assert stt["n_tokens"][t] == len(d)
        assert stt["n_traj"][t] == d["traj"].nunique()
        if len(d):
            assert abs(stt["kl_mean"][t] - d["kl"].mean()) < 1e-12
            assert abs(stt["kl_var"][t] - np.var(d["kl"].to_numpy(), ddof=0)) < 1e-12
            assert abs(stt["loss_mass"][t] - float((d["w"] * d["kl"]).sum())) < 1e-12
        else:
            assert stt["kl_mean"][t] == 0 and stt["kl_var"][t] == 0
