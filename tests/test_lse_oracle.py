"""Pins of the oracle's per-token log-partition functions (lse) and of the
per-token weights it reports, for the optional per-token outputs of both
fused calls.

lse is log sum_v exp(z[v]) of a logit row (Sec. 3, Eq. opd-rkl: at
temperature 1, App. D, log p(v) = z[v] - lse).  Expected values come from
scipy's logsumexp, closed forms (a constant row, a row of one very large
logit), the shift identity lse(z + c) = lse(z) + c, the full-vocabulary
oracle for a top-K support that is the whole vocabulary, and KL's identity
KL = <p_s, zs - zt> - lse_s + lse_t evaluated with scipy's softmax.
"""
import numpy as np
import pytest
from scipy import special

from oracle import topk_oracle as K
from oracle import turnkl_oracle as O


def lse64(zs, zt):
    out = np.empty((np.atleast_2d(zs).shape[0], 2))
    O.row_kl(np.atleast_2d(zs), np.atleast_2d(zt), O.DTYPE_F64, want_grad=False, lse_out=out)
    return out


@pytest.mark.parametrize("V", [1, 2, 17, 1000, 4099])
def test_lse_matches_scipy_logsumexp(V):
    rng = np.random.default_rng(100 + V)
    zs = rng.normal(0.0, 3.0, (6, V))
    zt = rng.normal(1.0, 2.0, (6, V))
    got = lse64(zs, zt)
    np.testing.assert_allclose(got[:, 0], special.logsumexp(zs, axis=1), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(got[:, 1], special.logsumexp(zt, axis=1), rtol=1e-13, atol=1e-13)


def test_lse_closed_forms_and_shift():
    V = 257
    c = np.full((1, V), -3.25)
    got = lse64(c, c + 10.0)
    assert got[0, 0] == pytest.approx(-3.25 + np.log(V), abs=1e-13)
    assert got[0, 1] == pytest.approx(6.75 + np.log(V), abs=1e-13)
    # one logit far above the rest: lse equals it up to exp(-gap) V
    z = np.zeros((1, V))
    z[0, 17] = 800.0
    got = lse64(z, z)
    assert got[0, 0] == pytest.approx(800.0 + np.log1p((V - 1) * np.exp(-800.0)), abs=1e-12)
    rng = np.random.default_rng(7)
    a = rng.normal(0.0, 2.0, (4, 333))
    b = rng.normal(0.0, 2.0, (4, 333))
    np.testing.assert_allclose(lse64(a + 41.5, b - 7.0), lse64(a, b) + [41.5, -7.0], atol=1e-11)


def test_lse_is_consistent_with_the_kl_identity():
    """KL = sum_v p_s(v) (zs[v] - zt[v]) - lse_s + lse_t, with p_s from scipy."""
    rng = np.random.default_rng(8)
    zs = rng.normal(0.0, 3.0, (5, 2048))
    zt = zs + rng.normal(0.0, 1.0, zs.shape)
    kl, _ = O.row_kl(zs, zt, O.DTYPE_F64, want_grad=False)
    lse = lse64(zs, zt)
    p = special.softmax(zs, axis=1)
    want = (p * (zs - zt)).sum(axis=1) - lse[:, 0] + lse[:, 1]
    np.testing.assert_allclose(kl, want, rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("dtype", [O.DTYPE_BF16, O.DTYPE_F32])
def test_lse_of_stored_logits_widens_exactly(dtype):
    rng = np.random.default_rng(9)
    z = rng.normal(0.0, 3.0, (3, 999)).astype(np.float32)
    if dtype == O.DTYPE_BF16:
        u = z.view(np.uint32).astype(np.uint64)
        bits = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
        wide = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        stored = bits
    else:
        wide, stored = z.astype(np.float64), z
    out = np.empty((3, 2))
    O.row_kl(stored, stored, dtype, want_grad=False, lse_out=out)
    np.testing.assert_allclose(out[:, 0], special.logsumexp(wide, axis=1), rtol=1e-13)
    assert np.array_equal(out[:, 0], out[:, 1])


def test_whole_pass_reports_lse_of_supervised_rows_only():
    rng = np.random.default_rng(10)
    traj = np.array([0, 0, 0, -1, 1, 1], np.int32)
    turn = np.array([0, 0, 1, 0, 0, 0], np.int32)
    mask = np.array([1, 0, 1, 0, 1, 1], np.uint8)
    zs = rng.normal(0.0, 2.0, (6, 64)).astype(np.float32)
    zt = rng.normal(0.0, 2.0, (6, 64)).astype(np.float32)
    ref = O.fwd_bwd(traj, turn, mask, 0.5, 4, lambda r: (zs[r], zt[r]), O.DTYPE_F32)
    for i in range(6):
        if mask[i]:
            assert ref.lse[i, 0] == pytest.approx(special.logsumexp(zs[i].astype(np.float64)),
                                                  abs=1e-12)
            assert ref.lse[i, 1] == pytest.approx(special.logsumexp(zt[i].astype(np.float64)),
                                                  abs=1e-12)
        else:
            assert np.all(np.isnan(ref.lse[i]))
            assert ref.w[i] == 0.0


def test_topk_support_lse():
    """On the whole vocabulary the top-K lse is the full one; on a subset it
    is scipy's logsumexp over the support."""
    rng = np.random.default_rng(11)
    a = rng.normal(0.0, 2.0, (4, 50))
    b = rng.normal(0.0, 2.0, (4, 50))
    np.testing.assert_allclose(K.support_lse(a, b), lse64(a, b), rtol=1e-13, atol=1e-13)
    ids = np.argsort(-b, axis=1)[:, :7]
    sa, sb = np.take_along_axis(a, ids, 1), np.take_along_axis(b, ids, 1)
    got = K.support_lse(sa, sb)
    np.testing.assert_allclose(got[:, 0], special.logsumexp(sa, axis=1), rtol=1e-13)
    np.testing.assert_allclose(got[:, 1], special.logsumexp(sb, axis=1), rtol=1e-13)


def test_lse_pin_rejects_plausible_mistakes():
    """The scipy pin's tolerance separates the oracle from plausible wrong
    values: the log of the shifted sum without the maximum added back, or
    the student's and the teacher's values swapped."""
    rng = np.random.default_rng(12)
    zs = rng.normal(0.0, 3.0, (3, 500))
    zt = rng.normal(2.0, 3.0, (3, 500))
    want = np.stack([special.logsumexp(zs, axis=1), special.logsumexp(zt, axis=1)], 1)
    m = zs.max(axis=1)
    dropped_max = np.stack([np.log(np.exp(zs - m[:, None]).sum(1)),
                            special.logsumexp(zt, axis=1)], 1)
    swapped = want[:, ::-1]
    for bad in (dropped_max, swapped):
        assert not np.allclose(bad, want, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(lse64(zs, zt), want, rtol=1e-13, atol=1e-13)
