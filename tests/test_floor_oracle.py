"""Pins of the oracle's turn-support floor (App. D, internal blend: n_min =
max(min_floor, ceil(min_frac * n_traj))) and of its per-outcome statistics
(Sec. 4.2: K_t^fail, K_t^succ and G_t), against the hand-derived example in
tests/golden/, brute-force group-bys and invariants of the weights."""
import json
import os
from fractions import Fraction

import numpy as np
import pandas as pd
import pytest

from oracle import turnkl_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _ex():
    with open(os.path.join(GOLDEN, "support_floor_outcome_example.json")) as f:
        return json.load(f)


def _batch(ex):
    tok = ex["tokens"]
    return (np.array(tok["traj_id"], np.int32), np.array(tok["turn_id"], np.int32),
            np.array(tok["loss_mask"], np.uint8), np.array(tok["success"], np.uint8))


def _frac(xs):
    return np.array([float(Fraction(x)) for x in xs])


def test_n_min_of_the_paper_configuration():
    g = _ex()["paper_default_n_min"]
    for n_traj, want in g["n_traj_to_n_min"]:
        assert O.n_min_of(n_traj, g["floor"], g["frac"]) == want, n_traj


def test_worked_example_weights_with_a_floor():
    ex = _ex()
    traj, turn, mask, _ = _batch(ex)
    seg = O.segments(traj, turn, mask, ex["max_turns"])
    assert O.turn_survivors(seg, ex["max_turns"]).tolist() == ex["survivors_per_turn"]
    for case, per_alpha in ex["weights"].items():
        floor, frac = ex["floors"][case]
        for a, fr in per_alpha.items():
            w = O.token_weights(seg, len(traj), mask, float(a), floor, frac)
            np.testing.assert_allclose(w, _frac(fr), rtol=1e-15, atol=0, err_msg=f"{case} {a}")
    # floor 6: no valid turn anywhere, the turn term falls back to the trajectory term
    w0 = _frac(ex["weights"]["floor2_frac0.55"]["0.0"])
    for a in (0.0, 0.3, 1.0):
        np.testing.assert_allclose(O.token_weights(seg, len(traj), mask, a, 6, 0.0), w0,
                                   rtol=1e-15, atol=0)


def _random_layout(rng, n_traj, max_turns):
    traj, turn, mask = [], [], []
    for b in range(n_traj):
        depth = int(rng.integers(1, max_turns + 1))  # trajectories end at different depths
        for t in range(depth):
            if rng.uniform() < 0.15:
                continue  # a turn the trajectory skips
            n = int(rng.integers(1, 7))
            traj += [b] * (n + 1)
            turn += [t] * (n + 1)
            mask += [0] + [int(v) for v in (rng.uniform(size=n) < 0.8)]
    return np.array(traj, np.int32), np.array(turn, np.int32), np.array(mask, np.uint8)


@pytest.mark.parametrize("seed", range(6))
def test_floor_invariants(seed):
    """For every floor: the weights sum to one, each trajectory gets 1/B; alpha
    = 0 ignores the floor; at alpha = 1 every valid supervised turn of a
    trajectory gets the same total weight and invalid turns none (unless the
    trajectory has no valid turn, when it keeps its alpha = 0 weights);
    n_min <= 1 admits every supervised turn (the plain blend)."""
    rng = np.random.default_rng(700 + seed)
    mt = 9
    traj, turn, mask = _random_layout(rng, 12, mt)
    seg = O.segments(traj, turn, mask, mt)
    assert seg.status == O.OK
    n = len(traj)
    df = pd.DataFrame({"traj": traj, "turn": turn, "mask": mask})
    sup = df[df["mask"] == 1]
    B = sup["traj"].nunique()
    surv = sup.groupby("turn")["traj"].nunique().reindex(range(mt), fill_value=0).to_numpy()
    plain = {a: O.token_weights(seg, n, mask, a) for a in (0.0, 0.35, 1.0)}
    for floor, frac in ((0, 0.0), (1, 0.0), (3, 0.0), (2, 0.4), (8, 0.15), (99, 0.0)):
        n_min = max(floor, int(np.ceil(frac * B)))
        for a in (0.0, 0.35, 1.0):
            w = O.token_weights(seg, n, mask, a, floor, frac)
            assert abs(w.sum() - 1.0) < 1e-12
            per_traj = pd.Series(w).groupby(traj).sum()
            for b in sup["traj"].unique():
                assert abs(per_traj[b] - 1.0 / B) < 1e-13
            if a == 0.0 or n_min <= 1:
                np.testing.assert_allclose(w, plain[a], rtol=1e-13, atol=0)
            if a == 1.0:
                dfw = sup.assign(w=w[df.index[df["mask"] == 1]])
                for b, g in dfw.groupby("traj"):
                    per_turn = g.groupby("turn")["w"].sum()
                    valid = [t for t in per_turn.index if surv[t] >= n_min]
                    if not valid:
                        np.testing.assert_allclose(g["w"], plain[0.0][g.index], rtol=1e-13)
                        continue
                    for t in per_turn.index:
                        want = 1.0 / (B * len(valid)) if t in valid else 0.0
                        assert abs(per_turn[t] - want) < 1e-13, (floor, frac, b, t)


def test_floor_loss_reduces_when_no_turn_is_valid():
    """n_min above every survivor count: L_turn equals L_traj, and L_blend
    with it for every alpha; without the floor they differ."""
    rng = np.random.default_rng(11)
    traj, turn, mask = _random_layout(rng, 5, 6)
    zs = rng.normal(0, 1, (len(traj), 16)).astype(np.float32)
    zt = (zs + rng.normal(0, 1, zs.shape)).astype(np.float32)
    src = lambda r: (zs[r], zt[r])
    res = O.fwd_bwd(traj, turn, mask, 0.5, 6, src, O.DTYPE_F32, support_floor=50)
    assert res.status == O.OK
    lb, lt, lu = res.loss
    assert abs(lu - lt) < 1e-15 and abs(lb - lt) < 1e-15
    plain = O.fwd_bwd(traj, turn, mask, 0.5, 6, src, O.DTYPE_F32)
    assert abs(plain.loss[2] - plain.loss[1]) > 1e-4
    assert plain.loss[1] == lt


# ----------------------------------------------------------------------------
# per-outcome statistics (Sec. 4.2)


def test_worked_example_outcome_split():
    ex = _ex()
    traj, turn, mask, succ = _batch(ex)
    seg = O.segments(traj, turn, mask, ex["max_turns"], succ)
    assert seg.status == O.OK
    kl = np.arange(len(traj)) / 10.0
    w = O.token_weights(seg, len(traj), mask, 0.5, 2, 0.55)
    st = O.outcome_split(seg, mask, kl, w, ex["max_turns"])
    g = ex["outcome"]
    for row, key in ((0, "fail"), (1, "succ")):
        assert st[row]["n_tokens"].tolist() == g[key]["n_tokens"]
        assert st[row]["n_traj"].tolist() == g[key]["n_traj"]
        np.testing.assert_allclose(st[row]["kl_mean"], _frac(g[key]["kl_mean"]), rtol=1e-14,
                                   atol=1e-15)
    gap = st[0]["kl_mean"] - st[1]["kl_mean"]
    for t, want in enumerate(g["gap_fail_minus_succ"]):
        if want is not None:
            assert abs(gap[t] - float(Fraction(want))) < 1e-14


@pytest.mark.parametrize("seed", range(5))
def test_outcome_split_matches_group_by_and_partitions_the_batch(seed):
    rng = np.random.default_rng(800 + seed)
    mt = 7
    traj, turn, mask = _random_layout(rng, 10, mt)
    flag_of = rng.integers(0, 2, 10)
    succ = flag_of[traj].astype(np.uint8)
    seg = O.segments(traj, turn, mask, mt, succ)
    assert seg.status == O.OK
    kl = rng.gamma(2.0, 0.3, len(traj))
    w = O.token_weights(seg, len(traj), mask, 0.4, 2, 0.3)
    st = O.outcome_split(seg, mask, kl, w, mt)
    every = O.turn_stats([(seg, mask, kl, w)], mt)
    df = pd.DataFrame({"traj": traj, "turn": turn, "kl": kl, "w": w, "s": succ})[mask == 1]
    for f in (0, 1):
        d = df[df["s"] == f]
        for t in range(mt):
            e = d[d["turn"] == t]
            assert st[f]["n_tokens"][t] == len(e)
            assert st[f]["n_traj"][t] == e["traj"].nunique()
            if len(e):
                assert abs(st[f]["kl_mean"][t] - e["kl"].mean()) < 1e-12
                assert abs(st[f]["kl_var"][t] - np.var(e["kl"].to_numpy())) < 1e-12
                assert abs(st[f]["loss_mass"][t] - float((e["w"] * e["kl"]).sum())) < 1e-13
    # the two outcomes partition every turn's tokens, survivors and loss mass
    for k in ("n_tokens", "n_traj"):
        np.testing.assert_array_equal(st[0][k] + st[1][k], every[k])
    np.testing.assert_allclose(st[0]["loss_mass"] + st[1]["loss_mass"], every["loss_mass"],
                               rtol=1e-12, atol=1e-16)
    tot = st[0]["n_tokens"] * st[0]["kl_mean"] + st[1]["n_tokens"] * st[1]["kl_mean"]
    np.testing.assert_allclose(tot, every["n_tokens"] * every["kl_mean"], rtol=1e-12, atol=1e-14)


def test_outcome_flag_errors_first_in_token_order():
    z = lambda *a: np.array(a, np.int32)
    m = lambda *a: np.array(a, np.uint8)
    # a flag that changes inside a turn, or between turns of one trajectory
    assert O.segments(z(0, 0, 0), z(0, 0, 0), m(1, 1, 1), 4, m(1, 1, 0)).status == O.ERR_OUTCOME
    assert O.segments(z(0, 0, 1), z(0, 1, 0), m(1, 1, 1), 4, m(1, 0, 0)).status == O.ERR_OUTCOME
    # nonzero flags are all "success"; padding flags are ignored
    assert O.segments(z(0, 0, 1), z(0, 1, 0), m(1, 1, 1), 4, m(1, 7, 0)).status == O.OK
    assert O.segments(z(0, -1, 0), z(0, 0, 1), m(1, 0, 1), 4, m(1, 0, 1)).status == O.OK
    # earliest position wins; at one token the other checks come first
    assert O.segments(z(0, 0, 0), z(1, 1, 0), m(1, 1, 1), 4, m(1, 1, 0)).status == O.ERR_UNSORTED
    assert O.segments(z(0, 0), z(0, 9), m(1, 1), 4, m(1, 0)).status == O.ERR_TURN_RANGE
    assert O.segments(z(0, 0, 0), z(0, 0, 9), m(1, 1, 1), 4, m(1, 0, 1)).status == O.ERR_OUTCOME
    # no flags: no outcome check
    assert O.segments(z(0, 0), z(0, 1), m(1, 1), 4).status == O.OK


# ----------------------------------------------------------------------------
# the pins have teeth


def test_pins_catch_planted_mistakes():
    ex = _ex()
    traj, turn, mask, _ = _batch(ex)
    seg = O.segments(traj, turn, mask, ex["max_turns"])
    want = _frac(ex["weights"]["floor2_frac0.55"]["1.0"])
    surv = np.array(ex["survivors_per_turn"])
    B = ex["B"]

    def weights(n_min, valid_of, fallback):
        w = np.zeros(len(traj))
        for b in range(B):
            ss = [s for s in range(seg.count) if seg.traj[s] == b and seg.n_sup[s] > 0]
            nv = sum(valid_of(int(seg.turn[s]), n_min) for s in ss)
            tot = sum(int(seg.n_sup[s]) for s in ss)
            for s in ss:
                q = (1.0 / nv if valid_of(int(seg.turn[s]), n_min) else 0.0) if nv else \
                    fallback(int(seg.n_sup[s]) / tot, len(ss))
                lo, hi = int(seg.start[s]), int(seg.start[s] + seg.length[s])
                for i in range(lo, hi):
                    if mask[i]:
                        w[i] = q / seg.n_sup[s] / B
        return w

    ge = lambda t, k: surv[t] >= k
    gt = lambda t, k: surv[t] > k
    traj_term = lambda q_traj, T: q_traj
    ok = weights(3, ge, traj_term)
    np.testing.assert_allclose(ok, want, rtol=1e-15)  # the intended rule reproduces the golden
    bad = [
        weights(3, gt, traj_term),                              # strict > instead of >=
        weights(max(2, int(np.floor(0.55 * B))), ge, traj_term),  # floor instead of ceil
        weights(max(2, int(np.ceil(0.55 * (B + 1)))), ge, traj_term),  # dead trajectory counted
        weights(3, ge, lambda q, T: 0.0),                       # no fallback: weight dropped
        weights(3, ge, lambda q, T: 1.0 / T),                   # fallback ignores the floor
    ]
    for k, w in enumerate(bad):
        assert np.max(np.abs(w - want)) > 1e-3, k
    # survivors counted as supervised tokens instead of trajectories
    tokens_per_turn = np.bincount(turn[mask == 1], minlength=5)
    assert (tokens_per_turn >= 3).tolist() != (surv >= 3).tolist()
