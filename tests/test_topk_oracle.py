"""Pins of the top-K reverse-KL oracle (reading T1-T3 of App. D's top-K
loss) against facts it does not compute itself: the full-vocabulary oracle
when the support is the whole vocabulary, closed forms, invariances and
finite differences of the full loss."""
import numpy as np
import pytest
from scipy import special, stats

from oracle import topk_oracle as K
from oracle import turnkl_oracle as O


def test_support_equal_to_the_vocabulary_gives_the_full_kl():
    rng = np.random.default_rng(3)
    n, V = 7, 40
    zs = rng.normal(0, 2, (n, V)).astype(np.float32)
    zt = (zs + rng.normal(0, 1, (n, V))).astype(np.float32)
    kl_full, g_full = O.row_kl(zs, zt, O.DTYPE_F32)
    perm = np.stack([rng.permutation(V) for _ in range(n)])
    a = np.take_along_axis(zs.astype(np.float64), perm, axis=1)
    b = np.take_along_axis(zt.astype(np.float64), perm, axis=1)
    kl, g = K.topk_row_kl(a, b)
    np.testing.assert_allclose(kl, kl_full, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(g, np.take_along_axis(g_full, perm, axis=1), rtol=1e-10, atol=1e-15)


def test_matches_scipy_on_the_renormalised_support():
    rng = np.random.default_rng(4)
    a = rng.normal(0, 3, (9, 50))
    b = rng.normal(0, 3, (9, 50))
    kl, _ = K.topk_row_kl(a, b)
    ref = stats.entropy(special.softmax(a, axis=1), special.softmax(b, axis=1), axis=1)
    np.testing.assert_allclose(kl, ref, rtol=1e-12)


def test_single_entry_support_has_no_loss_and_two_entries_are_bernoulli():
    kl, g = K.topk_row_kl(np.array([[3.0], [-1.0]]), np.array([[7.0], [0.5]]))
    assert np.all(kl == 0.0) and np.all(g == 0.0)
    a = np.array([[0.3, -0.4]])
    b = np.array([[1.1, 0.2]])
    p = special.expit(a[0, 0] - a[0, 1])
    q = special.expit(b[0, 0] - b[0, 1])
    want = p * np.log(p / q) + (1 - p) * np.log((1 - p) / (1 - q))
    kl, g = K.topk_row_kl(a, b)
    assert abs(kl[0] - want) < 1e-14
    # d KL / d a_0 for a Bernoulli: p (1 - p) (logit(p) - logit(q))
    dp = p * (1 - p) * (np.log(p / (1 - p)) - np.log(q / (1 - q)))
    assert abs(g[0, 0] - dp) < 1e-14 and abs(g[0, 0] + g[0, 1]) < 1e-15


def test_shift_and_order_invariance_and_gradient_sums_to_zero():
    rng = np.random.default_rng(5)
    a = rng.normal(0, 2, (6, 50))
    b = rng.normal(0, 2, (6, 50))
    kl, g = K.topk_row_kl(a, b)
    kl2, g2 = K.topk_row_kl(a + 11.0, b - 4.0)  # per-row constants cancel (T2)
    np.testing.assert_allclose(kl2, kl, rtol=1e-12)
    np.testing.assert_allclose(g2, g, rtol=1e-9, atol=1e-15)
    perm = rng.permutation(50)
    kl3, g3 = K.topk_row_kl(a[:, perm], b[:, perm])
    np.testing.assert_allclose(kl3, kl, rtol=1e-12)
    np.testing.assert_allclose(g3, g[:, perm], rtol=1e-12, atol=1e-16)
    assert np.all(np.abs(g.sum(axis=1)) < 1e-14)  # 50 fp64 terms of size <= 0.2
    assert np.all(kl >= 0.0)


def test_gradient_matches_finite_differences_of_the_full_loss():
    """Central differences of L_blend with respect to every student logit
    (those off the support must have zero derivative)."""
    rng = np.random.default_rng(6)
    V, Kk = 12, 5
    traj = np.array([0, 0, 0, 0, 1, 1, 1], np.int32)
    turn = np.array([0, 0, 1, 1, 0, 0, 1], np.int32)
    mask = np.array([1, 1, 0, 1, 1, 1, 1], np.uint8)
    n = traj.shape[0]
    zs = rng.normal(0, 1.5, (n, V))
    ids = np.stack([rng.choice(V, Kk, replace=False) for _ in range(n)])
    tv = rng.normal(0, 1.5, (n, Kk))

    def loss(z):
        r = K.fwd_bwd_topk(traj, turn, mask, 0.4, 4, lambda rows, i: np.take_along_axis(
            z[rows], i, axis=1), ids, tv, O.DTYPE_F64)
        return r.loss[0], r

    _, ref = loss(zs)
    h = 1e-6
    for i in range(n):
        for v in range(V):
            zp, zm = zs.copy(), zs.copy()
            zp[i, v] += h
            zm[i, v] -= h
            fd = (loss(zp)[0] - loss(zm)[0]) / (2 * h)
            if mask[i] and v in ids[i]:
                j = int(np.nonzero(ids[i] == v)[0][0])
                an = ref.w[i] * ref.grads[i][j]
            else:
                an = 0.0
            assert abs(fd - an) <= 1e-7 + 1e-6 * abs(an), (i, v, fd, an)


def test_pins_catch_planted_mistakes():
    rng = np.random.default_rng(7)
    a = rng.normal(0, 2, (5, 50))
    b = rng.normal(0, 2, (5, 50))
    kl, g = K.topk_row_kl(a, b)
    ref = stats.entropy(special.softmax(a, axis=1), special.softmax(b, axis=1), axis=1)
    # (1) no renormalisation of the teacher (full-vocabulary log-probs taken as is)
    lt_raw = b - np.log(np.exp(b).sum(axis=1, keepdims=True) * 3.0)
    p = special.softmax(a, axis=1)
    bad = (p * (np.log(p) - lt_raw)).sum(axis=1)
    assert np.max(np.abs(bad - ref)) > 1e-3
    # (2) forward instead of reverse direction
    fwd = stats.entropy(special.softmax(b, axis=1), special.softmax(a, axis=1), axis=1)
    assert np.max(np.abs(fwd - kl)) > 1e-3
    # (3) gradient without the -KL term no longer sums to zero
    assert np.max(np.abs((g + p * kl[:, None]).sum(axis=1))) > 1e-3
