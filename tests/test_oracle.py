"""Pins of the CPU oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: every expected value comes from
a closed form, a library routine (scipy), finite differences, a brute-force
group-by, the hand-derived worked example in tests/golden/, or a value the
paper prints.  test_pins_catch_planted_mistakes shows that plausible mistakes
in the oracle fail these pins.
"""
import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pandas as pd
import pytest
from scipy import special, stats

from oracle import turnkl_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def kl64(zs, zt, grad=True):
    return O.row_kl(np.atleast_2d(zs), np.atleast_2d(zt), O.DTYPE_F64, want_grad=grad)


def bf16_bits(x):
    """Round float32 values to bf16 (RNE) and return the 16-bit patterns."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def bf16_value(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32)


# ----------------------------------------------------------------------------
# per-token reverse KL (Sec. 3, Eq. opd-rkl)


def test_identical_logits_give_exact_zero():
    rng = np.random.default_rng(1)
    z = rng.normal(0.0, 3.0, (7, 301))
    kl, g = kl64(z, z)
    assert np.all(kl == 0.0) and np.all(g == 0.0)
    b = bf16_bits(z)
    kl, g = O.row_kl(b, b, O.DTYPE_BF16)
    assert np.all(kl == 0.0) and np.all(g == 0.0)
    f = z.astype(np.float32)
    kl, g = O.row_kl(f, f, O.DTYPE_F32)
    assert np.all(kl == 0.0) and np.all(g == 0.0)


@pytest.mark.parametrize("V", [1, 2, 3, 17, 300, 4099])
def test_kl_matches_scipy_relative_entropy(V):
    """KL(p_s || p_t), student first, equals scipy's relative entropy."""
    rng = np.random.default_rng(V)
    zs = rng.normal(0.0, 2.5, (5, V))
    zt = zs + rng.normal(0.0, 1.0, (5, V))
    kl, _ = kl64(zs, zt, grad=False)
    ref = stats.entropy(special.softmax(zs, axis=1), special.softmax(zt, axis=1), axis=1)
    np.testing.assert_allclose(kl, ref, rtol=1e-10, atol=1e-14)


def test_kl_uniform_teacher_is_log_v_minus_entropy():
    rng = np.random.default_rng(2)
    V = 1000
    zs = rng.normal(0.0, 3.0, (4, V))
    zt = np.full_like(zs, 0.7)
    kl, _ = kl64(zs, zt, grad=False)
    ref = np.log(V) - stats.entropy(special.softmax(zs, axis=1), axis=1)
    np.testing.assert_allclose(kl, ref, rtol=1e-11, atol=1e-13)


def test_kl_two_classes_is_bernoulli_kl():
    x = np.array([-3.0, -0.4, 0.0, 1.1, 5.0])
    y = np.array([2.0, -0.1, 0.3, -2.0, 4.0])
    zs = np.stack([np.zeros_like(x), x], 1)
    zt = np.stack([np.zeros_like(y), y], 1)
    kl, g = kl64(zs, zt)
    p, q = special.expit(x), special.expit(y)
    ref = p * np.log(p / q) + (1 - p) * np.log((1 - p) / (1 - q))
    np.testing.assert_allclose(kl, ref, rtol=1e-12)
    # d/dx of the Bernoulli KL with p = sigmoid(x): p(1-p)(logit p - logit q) = p(1-p)(x - y)
    dkl = p * (1 - p) * (x - y)
    np.testing.assert_allclose(g[:, 1], dkl, rtol=1e-11, atol=1e-15)
    np.testing.assert_allclose(g[:, 0], -dkl, rtol=1e-11, atol=1e-15)


@pytest.mark.parametrize("c", [-6.0, -0.5, 0.25, 10.0])
def test_kl_single_boosted_token_closed_form(c):
    """Teacher = student + c at one column k: KL = -c p_k + log(1 + p_k (e^c - 1))."""
    rng = np.random.default_rng(3)
    zs = rng.normal(0.0, 2.0, (3, 257))
    k = 41
    zt = zs.copy()
    zt[:, k] += c
    kl, _ = kl64(zs, zt, grad=False)
    pk = special.softmax(zs, axis=1)[:, k]
    ref = -c * pk + np.log1p(pk * np.expm1(c))
    np.testing.assert_allclose(kl, ref, rtol=1e-10, atol=1e-15)


def test_kl_nonnegative_and_shift_invariant():
    rng = np.random.default_rng(4)
    zs = rng.normal(0.0, 3.0, (16, 513))
    zt = zs + rng.normal(0.0, 1.5, zs.shape)
    kl, g = kl64(zs, zt)
    assert np.all(kl > 0)
    a = rng.normal(0, 50, (16, 1))
    b = rng.normal(0, 50, (16, 1))
    kl2, g2 = kl64(zs + a, zt + b)
    np.testing.assert_allclose(kl2, kl, rtol=1e-9)
    np.testing.assert_allclose(g2, g, rtol=1e-7, atol=1e-14)


def test_bf16_and_f32_inputs_widen_exactly():
    rng = np.random.default_rng(5)
    x = rng.normal(0.0, 3.0, (6, 777)).astype(np.float32)
    y = (x + rng.normal(0.0, 1.0, x.shape)).astype(np.float32)
    bs, bt = bf16_bits(x), bf16_bits(y)
    kl_b, g_b = O.row_kl(bs, bt, O.DTYPE_BF16)
    kl_w, g_w = kl64(bf16_value(bs).astype(np.float64), bf16_value(bt).astype(np.float64))
    assert np.array_equal(kl_b, kl_w) and np.array_equal(g_b, g_w)
    kl_f, g_f = O.row_kl(x, y, O.DTYPE_F32)
    kl_w, g_w = kl64(x.astype(np.float64), y.astype(np.float64))
    assert np.array_equal(kl_f, kl_w) and np.array_equal(g_f, g_w)


def test_contamination_compression_bound():
    """Prop. 1 (Sec. 4.3; proof App. B): with pi = lam p_F + (1 - lam) p_free for
    both models, KL(pi_S || pi_T) <= (1 - lam) KL(p_S_free || p_T_free)."""
    rng = np.random.default_rng(6)
    V = 64
    for trial in range(200):
        pf = rng.dirichlet(np.full(V, 0.3))
        ps = rng.dirichlet(np.full(V, 0.5))
        pt = rng.dirichlet(np.full(V, 0.5))
        lam = rng.uniform(0.0, 1.0)
        pis = lam * pf + (1 - lam) * ps
        pit = lam * pf + (1 - lam) * pt
        kl, _ = kl64(np.log(pis), np.log(pit), grad=False)
        bound = (1 - lam) * stats.entropy(ps, pt)
        assert kl[0] <= bound * (1 + 1e-12) + 1e-15, (trial, kl[0], bound)


# ----------------------------------------------------------------------------
# gradient with respect to the student logits (teacher frozen, Sec. 3)


def test_gradient_rows_sum_to_zero_and_permute_with_vocab():
    rng = np.random.default_rng(7)
    zs = rng.normal(0.0, 3.0, (5, 333))
    zt = zs + rng.normal(0.0, 1.0, zs.shape)
    kl, g = kl64(zs, zt)
    np.testing.assert_allclose(g.sum(axis=1), 0.0, atol=1e-13)
    perm = rng.permutation(333)
    kl2, g2 = kl64(zs[:, perm], zt[:, perm])
    np.testing.assert_allclose(kl2, kl, rtol=1e-12)
    np.testing.assert_allclose(g2, g[:, perm], rtol=1e-10, atol=1e-17)


def _tiny_batch(rng, n_traj=3, max_turn=4, V=12):
    traj, turn, mask = [], [], []
    for b in range(n_traj):
        for t in range(int(rng.integers(1, max_turn + 1))):
            n = int(rng.integers(1, 5))
            traj += [b] * n
            turn += [t] * n
            mask += [int(v) for v in rng.integers(0, 2, n)]
    mask[-1] = 1
    traj, turn, mask = (np.array(traj, np.int32), np.array(turn, np.int32),
                        np.array(mask, np.uint8))
    zs = rng.normal(0.0, 2.0, (len(traj), V))
    zt = zs + rng.normal(0.0, 1.0, zs.shape)
    return traj, turn, mask, zs, zt


@pytest.mark.parametrize("alpha", [0.0, 0.3, 1.0])
def test_gradient_matches_finite_differences_of_the_full_loss(alpha):
    """dL/dz_s by central differences of L = sum_i w_i KL_i (float64, V <= 64)."""
    rng = np.random.default_rng(8)
    traj, turn, mask, zs, zt = _tiny_batch(rng)
    seg = O.segments(traj, turn, mask, 8)
    assert seg.status == O.OK
    w = O.token_weights(seg, len(traj), mask, alpha)
    scale = 1.7
    kl, g = kl64(zs, zt)
    G = scale * w[:, None] * g

    def loss(z):
        k, _ = kl64(z, zt, grad=False)
        return scale * float(np.sum(w * np.where(mask == 1, k, 0.0)))

    h = 1e-5
    worst = 0.0
    for i in range(len(traj)):
        for v in range(zs.shape[1]):
            zp = zs.copy()
            zm = zs.copy()
            zp[i, v] += h
            zm[i, v] -= h
            fd = (loss(zp) - loss(zm)) / (2 * h)
            worst = max(worst, abs(fd - G[i, v]))
    assert worst <= 1e-8 * max(1e-3, np.abs(G).max()), worst


# ----------------------------------------------------------------------------
# segments, weights and loss (Sec. 3, Sec. 4.4, Sec. 5.2, App. D Algorithm 1)


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_worked_example_segments_and_weights():
    ex = _load("worked_example.json")
    tok = ex["tokens"]
    traj = np.array(tok["traj_id"], np.int32)
    turn = np.array(tok["turn_id"], np.int32)
    mask = np.array(tok["loss_mask"], np.uint8)
    seg = O.segments(traj, turn, mask, ex["max_turns"])
    assert seg.status == O.OK
    for k in ("start", "length", "traj", "turn", "n_sup"):
        assert getattr(seg, k).tolist() == ex["segments"][k], k
    for a, fr in ex["weights"].items():
        w = O.token_weights(seg, len(traj), mask, float(a))
        ref = np.array([float(Fraction(x)) for x in fr])
        np.testing.assert_allclose(w, ref, rtol=1e-15, atol=0)
    kl = np.linspace(0.1, 1.3, len(traj))
    st = O.turn_stats([(seg, mask, kl, np.zeros(len(traj)))], ex["max_turns"])
    assert st["n_traj"].tolist() == ex["survivors_per_turn"]
    assert st["n_tokens"].tolist() == ex["supervised_tokens_per_turn"]


def _random_layout(rng, n_traj, max_turns, pad_prob=0.0, masked_traj_prob=0.1):
    traj, turn, mask = [], [], []
    for b in range(n_traj):
        turns = np.sort(rng.choice(max_turns, size=int(rng.integers(1, max_turns + 1)),
                                   replace=False))
        dead = rng.uniform() < masked_traj_prob
        for t in turns:
            n = int(rng.integers(1, 9))
            if rng.uniform() < pad_prob:
                k = int(rng.integers(1, 3))
                traj += [-1] * k
                turn += [0] * k
                mask += [0] * k
            traj += [b] * n
            turn += [int(t)] * n
            mode = rng.integers(0, 3)
            if dead or mode == 0:
                mask += [0] * n
            elif mode == 1:
                mask += [1] * n
            else:
                mask += [int(v) for v in rng.integers(0, 2, n)]
    return (np.array(traj, np.int32), np.array(turn, np.int32), np.array(mask, np.uint8))


def _frame(traj, turn, mask, kl, w=None):
    df = pd.DataFrame({"traj": traj, "turn": turn, "mask": mask, "kl": kl})
    if w is not None:
        df["w"] = w
    return df[(df["traj"] >= 0) & (df["mask"] == 1)]


@pytest.mark.parametrize("seed", range(8))
def test_weights_sum_to_one_and_reduce_to_paper_forms(seed):
    rng = np.random.default_rng(100 + seed)
    traj, turn, mask = _random_layout(rng, 6, 7, pad_prob=0.2)
    seg = O.segments(traj, turn, mask, 7)
    assert seg.status == O.OK
    n = len(traj)
    kl = rng.uniform(0.0, 2.0, n)
    w0 = O.token_weights(seg, n, mask, 0.0)
    w1 = O.token_weights(seg, n, mask, 1.0)
    df = _frame(traj, turn, mask, kl)
    if df.empty:
        assert not w0.any()
        return
    for a in (0.0, 0.4, 1.0):
        w = O.token_weights(seg, n, mask, a)
        assert abs(w.sum() - 1.0) < 1e-12
        assert np.all(w[mask == 0] == 0)
        # affine in alpha
        np.testing.assert_allclose(w, (1 - a) * w0 + a * w1, rtol=1e-13, atol=1e-17)
    # alpha = 0: Eq. (opd-rkl): mean over trajectories of the per-trajectory token mean
    l0 = df.groupby("traj")["kl"].mean().mean()
    assert abs(float(np.sum(w0 * kl)) - l0) < 1e-12
    # alpha = 1: mean over trajectories of the mean over supervised turns of the turn mean
    l1 = df.groupby(["traj", "turn"])["kl"].mean().groupby(level=0).mean().mean()
    assert abs(float(np.sum(w1 * kl)) - l1) < 1e-12


def test_weights_independent_of_alpha_when_turns_have_equal_counts():
    """q_traj_t = n_t / N equals q_turn_t = 1 / T when all n_t are equal (Sec. 5.2)."""
    rng = np.random.default_rng(9)
    traj, turn, mask = [], [], []
    for b in range(5):
        n = int(rng.integers(1, 6))
        for t in range(int(rng.integers(1, 6))):
            traj += [b] * (n + 2)
            turn += [t] * (n + 2)
            mask += [0, 0] + [1] * n
    seg = O.segments(traj, turn, mask, 8)
    w0 = O.token_weights(seg, len(traj), mask, 0.0)
    for a in (0.25, 1.0):
        np.testing.assert_allclose(O.token_weights(seg, len(traj), mask, a), w0, rtol=1e-14)


def _brute_segments(traj, turn, mask):
    out = []
    i = 0
    for key, grp in itertools.groupby(range(len(traj)), key=lambda k: (int(traj[k]), int(turn[k]))):
        idx = list(grp)
        if key[0] < 0:
            continue
        out.append((idx[0], len(idx), key[0], key[1], int(sum(int(mask[k]) for k in idx))))
        i += len(idx)
    return out


@pytest.mark.parametrize("seed", range(10))
def test_segments_match_brute_force_group_by(seed):
    rng = np.random.default_rng(200 + seed)
    traj, turn, mask = _random_layout(rng, 7, 9, pad_prob=0.3)
    seg = O.segments(traj, turn, mask, 9)
    assert seg.status == O.OK
    got = list(zip(seg.start.tolist(), seg.length.tolist(), seg.traj.tolist(),
                   seg.turn.tolist(), seg.n_sup.tolist()))
    assert got == _brute_segments(traj, turn, mask)


def test_segment_errors_first_in_token_order():
    z = lambda *a: np.array(a, np.int32)
    m = lambda *a: np.array(a, np.uint8)
    # padding with mask 1
    assert O.segments(z(0, -1), z(0, 0), m(1, 1), 4).status == O.ERR_PAD_MASK
    # turn id out of range (either side)
    assert O.segments(z(0, 0), z(0, 4), m(1, 1), 4).status == O.ERR_TURN_RANGE
    assert O.segments(z(0, 0), z(-1, 0), m(1, 1), 4).status == O.ERR_TURN_RANGE
    # trajectory ids must increase; turn ids must increase within a trajectory
    assert O.segments(z(1, 1, 0), z(0, 0, 0), m(1, 1, 1), 4).status == O.ERR_UNSORTED
    assert O.segments(z(0, 0, 0), z(2, 2, 1), m(1, 1, 1), 4).status == O.ERR_UNSORTED
    # a turn split by padding is two runs of the same turn id
    assert O.segments(z(0, -1, 0), z(1, 0, 1), m(1, 0, 1), 4).status == O.ERR_UNSORTED
    # the earliest violation wins: unsorted at token 2 before range at token 4
    assert O.segments(z(0, 0, 0, 1, 1), z(1, 1, 0, 0, 9), m(1, 1, 1, 1, 1), 4).status == \
        O.ERR_UNSORTED
    # ... and a range error at token 1 before the unsorted run at token 2
    assert O.segments(z(0, 0, 0), z(1, 7, 0), m(1, 1, 1), 4).status == O.ERR_TURN_RANGE
    # empty and all-padding batches are valid and empty
    e = O.segments(z(), z(), m(), 4)
    assert e.status == O.OK and e.count == 0
    p = O.segments(z(-1, -1), z(0, 3), m(0, 0), 4)
    assert p.status == O.OK and p.count == 0


# ----------------------------------------------------------------------------
# per-turn statistics (Sec. 4.3 Eq. observed-turn-kl; Sec. 5.1; Sec. 4.4)


@pytest.mark.parametrize("seed", range(6))
def test_turn_stats_match_group_by(seed):
    rng = np.random.default_rng(300 + seed)
    traj, turn, mask = _random_layout(rng, 8, 6, pad_prob=0.1)
    seg = O.segments(traj, turn, mask, 6)
    n = len(traj)
    kl = rng.gamma(2.0, 0.3, n)
    w = O.token_weights(seg, n, mask, 0.6)
    st = O.turn_stats([(seg, mask, kl, w)], 6)
    df = _frame(traj, turn, mask, kl, w)
    for t in range(6):
        d = df[df["turn"] == t]
        assert st["n_tokens"][t] == len(d)
        assert st["n_traj"][t] == d["traj"].nunique()
        if len(d):
            assert abs(st["kl_mean"][t] - d["kl"].mean()) < 1e-12
            assert abs(st["kl_var"][t] - np.var(d["kl"].to_numpy(), ddof=0)) < 1e-12
            assert abs(st["kl_m2"][t] - st["kl_var"][t] * len(d)) < 1e-11
            assert abs(st["loss_mass"][t] - float((d["w"] * d["kl"]).sum())) < 1e-12
        else:
            assert st["kl_mean"][t] == 0 and st["kl_var"][t] == 0 and st["loss_mass"][t] == 0
    # totals: sum_t n_t mean_t = sum of supervised KL; sum_t loss_mass_t = L_blend
    assert abs(float((st["n_tokens"] * st["kl_mean"]).sum()) - float(df["kl"].sum())) < 1e-10
    assert abs(float(st["loss_mass"].sum()) - float(np.sum(w * kl))) < 1e-12


def test_turn_stats_pool_micro_batches():
    rng = np.random.default_rng(400)
    parts, frames = [], []
    for k in range(3):
        traj, turn, mask = _random_layout(rng, 4, 5)
        seg = O.segments(traj, turn, mask, 5)
        kl = rng.uniform(0, 1, len(traj))
        w = O.token_weights(seg, len(traj), mask, 0.5)
        parts.append((seg, mask, kl, w))
        f = _frame(traj + 100 * k, turn, mask, kl, w)
        frames.append(f)
    st = O.turn_stats(parts, 5)
    df = pd.concat(frames)
    for t in range(5):
        d = df[df["turn"] == t]
        assert st["n_tokens"][t] == len(d)
        assert st["n_traj"][t] == d["traj"].nunique()
        if len(d):
            assert abs(st["kl_mean"][t] - d["kl"].mean()) < 1e-12
            assert abs(st["kl_var"][t] - np.var(d["kl"].to_numpy())) < 1e-12


# ----------------------------------------------------------------------------
# alpha schedule (Sec. 5.2, App. D Algorithm 1) against the printed table


def test_alpha_schedule_reproduces_printed_phase_means():
    g = _load("alpha_schedule_table3.json")
    K = g["K"]
    alphas = [O.alpha_schedule(k, K, g["s"], g["e"]) for k in range(1, K + 1)]
    thirds = [alphas[0:33], alphas[33:66], alphas[66:100]]
    for part, printed in zip(thirds, g["alpha_early_mid_late"]):
        assert abs(np.mean(part) - printed) <= g["printed_precision"] + 1e-9
    assert O.alpha_schedule(0, 10) == 0.0 and O.alpha_schedule(10, 10) == 1.0
    assert O.alpha_schedule(5, 10, 0.6, 0.6) == 0.0 and O.alpha_schedule(7, 10, 0.6, 0.6) == 1.0
    assert O.alpha_schedule(3, 10, 0.2, 0.6) == pytest.approx(0.25)


# ----------------------------------------------------------------------------
# the pins have teeth: plausible mistakes planted in the oracle fail them


def test_pins_catch_planted_mistakes():
    rng = np.random.default_rng(500)
    zs = rng.normal(0.0, 2.0, (4, 50))
    zt = zs + rng.normal(0.0, 1.0, zs.shape)
    ps, pt = special.softmax(zs, axis=1), special.softmax(zt, axis=1)
    ref = stats.entropy(ps, pt, axis=1)
    # (1) KL direction reversed (teacher first)
    rev, _ = kl64(zt, zs, grad=False)
    assert np.max(np.abs(rev - ref)) > 1e-3
    # (2) gradient missing the -KL term, or with the sign flipped
    kl, g = kl64(zs, zt)
    no_kl = g + ps * kl[:, None]
    assert np.max(np.abs(no_kl.sum(axis=1))) > 1e-3          # rows no longer sum to 0
    x = np.array([0.8])
    zs2 = np.stack([np.zeros(1), x], 1)
    zt2 = np.stack([np.zeros(1), -x], 1)
    _, g2 = kl64(zs2, zt2)
    p = special.expit(x)
    assert abs(-g2[0, 1] - p * (1 - p) * (2 * x)) > 1e-3     # flipped sign fails V = 2
    # (3) trajectory token share and turn share swapped (alpha <-> 1 - alpha)
    ex = _load("worked_example.json")
    tok = ex["tokens"]
    seg = O.segments(tok["traj_id"], tok["turn_id"], tok["loss_mask"], 3)
    w_bad = O.token_weights(seg, 13, np.array(tok["loss_mask"]), 1.0 - 0.25)
    w_ref = np.array([float(Fraction(v)) for v in ex["weights"]["0.5"]])
    w_ok = O.token_weights(seg, 13, np.array(tok["loss_mask"]), 0.5)
    np.testing.assert_allclose(w_ok, w_ref, rtol=1e-15)
    assert np.max(np.abs(w_bad - w_ref)) > 1e-3
    # (4) sample variance (ddof = 1) instead of population variance
    v = np.array([0.1, 0.4, 0.7])
    assert abs(np.var(v, ddof=1) - np.var(v, ddof=0)) > 1e-3
