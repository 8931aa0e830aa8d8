"""The seeded input generator (synth/): its Box-Muller transform against the
platform's math library, and the logits it draws against N(0, sigma^2)."""
import ctypes
import math

import numpy as np
import pytest
from scipy import stats

import synth
from synth import _lib


def _lib_math():
    L = _lib.lib()
    L.synth_math.restype = None
    L.synth_math.argtypes = [ctypes.c_double, ctypes.c_double, ctypes.POINTER(ctypes.c_double)]
    L.synth_normal_pair.restype = None
    L.synth_normal_pair.argtypes = [ctypes.c_uint64, ctypes.c_uint64,
                                    ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(ctypes.c_double)]
    return L


def test_transform_helpers_match_libm():
    """ln, sqrt and (cos, sin) of a full turn, written from their series, agree
    with numpy to a few units in the last place over the ranges the transform
    uses (ln on (0, 1], sqrt on [0, 75], every octant of the turn)."""
    L = _lib_math()
    out = (ctypes.c_double * 4)()
    rng = np.random.default_rng(3)
    xs = np.concatenate([np.exp(rng.uniform(-37, 0, 3000)), rng.uniform(0, 75, 1000),
                         [2.0 ** -52, 1 - 2.0 ** -52, 1.0, 0.5, 2.0, 4.0, math.sqrt(2.0), 73.0]])
    vs = np.concatenate([rng.uniform(0, 1, xs.size - 16), np.arange(16) / 16.0])
    for x, v in zip(xs.tolist(), vs.tolist()):
        L.synth_math(x, v, out)
        assert abs(out[0] - math.log(x)) <= 4e-16 * max(abs(math.log(x)), 1e-300) + 1e-300
        assert abs(out[1] - math.sqrt(x)) <= 4e-16 * math.sqrt(x)
        assert abs(out[2] - math.cos(2 * math.pi * v)) <= 1e-15
        assert abs(out[3] - math.sin(2 * math.pi * v)) <= 1e-15
    L.synth_math(0.0, 0.0, out)
    assert out[1] == 0.0 and out[2] == 1.0 and out[3] == 0.0


def test_normal_pair_is_box_muller():
    """The pair equals sqrt(-2 ln u1) (cos, sin)(2 pi u2) with the uniforms
    taken from the top 52 bits of the two SplitMix64 outputs."""
    L = _lib_math()
    z1, z2 = ctypes.c_double(), ctypes.c_double()
    rng = np.random.default_rng(5)
    xs = rng.integers(0, 2 ** 63, size=(2000, 2), dtype=np.uint64) * np.uint64(2)
    xs[0] = (0, 0)                      # u1 = 1: r = 0
    xs[1] = (2 ** 64 - 1, 0)            # u1 = 2^-52: the largest radius
    for a, b in xs.tolist():
        L.synth_normal_pair(a, b, ctypes.byref(z1), ctypes.byref(z2))
        u1 = 1.0 - (a >> 12) * 2.0 ** -52
        u2 = (b >> 12) * 2.0 ** -52
        r = math.sqrt(-2.0 * math.log(u1)) if u1 < 1.0 else 0.0
        assert abs(z1.value - r * math.cos(2 * math.pi * u2)) <= 1e-14 * max(r, 1.0)
        assert abs(z2.value - r * math.sin(2 * math.pi * u2)) <= 1e-14 * max(r, 1.0)
    L.synth_normal_pair(2 ** 64 - 1, 0, ctypes.byref(z1), ctypes.byref(z2))
    assert abs(z1.value - math.sqrt(104 * math.log(2.0))) < 1e-12 and z2.value == 0.0


def test_logits_are_gaussian():
    """fp32 logits of the tiny batch (student sigma 2, teacher noise 0.5): the
    student values and the teacher-minus-student noise pass a
    Kolmogorov-Smirnov test against N(0, sigma^2), their moments are the
    Gaussian's, they are uncorrelated, and the tails reach past 4 sigma (a
    sum of a few uniforms could not)."""
    w = synth.make("tiny")
    zs, zt = w.host_logits(0, w.n_tokens)
    s = zs.astype(np.float64).ravel() / w.student_sigma
    d = (zt.astype(np.float64) - zs.astype(np.float64)).ravel() / float(w.teacher_sigma[0])
    for x in (s, d):
        assert stats.kstest(x, "norm").pvalue > 1e-3
        assert abs(x.mean()) < 5.0 / math.sqrt(x.size)
        assert abs(x.var() - 1.0) < 0.01
        assert abs(stats.kurtosis(x)) < 0.05
        assert np.abs(x).max() > 4.2
    assert abs(np.corrcoef(s, d)[0, 1]) < 0.01


@pytest.mark.parametrize("name", ["agent", "long_horizon"])
def test_row_maxima_follow_the_gaussian(name):
    """bf16 rows of V draws: the mean row maximum is the Gaussian's expected
    maximum of V draws (about 4.1 sigma at V = 32,000, 4.4 sigma at 151,936),
    within a few percent."""
    w = synth.make(name)
    zs, _ = w.host_logits(0, 16)
    x = (zs.astype(np.uint32) << 16).view(np.float32).astype(np.float64) / w.student_sigma
    # E[max of V standard normals] by numerical integration of 1 - Phi^V
    grid = np.linspace(0.0, 9.0, 20001)
    e_max = np.trapezoid(1.0 - stats.norm.cdf(grid) ** w.vocab, grid)
    got = x.max(axis=1).mean()
    assert abs(got - e_max) < 0.05 * e_max, (got, e_max)
