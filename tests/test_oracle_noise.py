"""Pins of the oracle's noise stream against references other than itself.

* Philox words: rocRAND's Philox4x32-10 engine (a third-party implementation),
  whose seed / subsequence / offset semantics define the element -> word map.
* Transforms: mpmath at 200 bits, correctly rounded to binary32.
* Scale: the closed-form moments and CDF of the Laplace and Gaussian laws
  (Prop. 2: Gaussian standard deviation Delta/eps; Laplace scale Delta/eps).
"""
import math

import numpy as np
import pytest

import oracle as O
from tests import pins


def test_philox_zero_block_matches_rocrand():
    ref = pins.rocrand_words(0, 0, 0, 4)
    got = O.philox4x32_10([0, 0, 0, 0], [0, 0])
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("seed,sid,block0", [
    (0, 0, 0), (1, 0, 5), (0xDEADBEEFCAFEF00D, 3, 123456789),
    (42, (27 << 8) | 3, 2**33 + 17), (2**64 - 1, 2**64 - 1, 2**62 - 8)])
def test_philox_blocks_match_rocrand(seed, sid, block0):
    nblk = 64
    ref = pins.rocrand_words(seed, sid, 4 * block0, 4 * nblk).reshape(nblk, 4)
    got = O.philox_blocks(np.arange(block0, block0 + nblk, dtype=np.uint64), seed, sid)
    assert np.array_equal(got, ref)


def _words_sample(n, seed):
    g = np.random.Generator(np.random.PCG64(seed))
    rnd = g.integers(0, 2**32, size=n, dtype=np.uint64).astype(np.uint32)
    return np.concatenate([pins.edge_words(), rnd])


@pytest.mark.parametrize("fn", [O.FN_LAPLACE_T, O.FN_GAUSS_R, O.FN_COS2PI, O.FN_SIN2PI])
def test_transform_correctly_rounded_vs_mpmath(fn):
    words = _words_sample(600, 100 + fn)
    got = O.transform(fn, words)
    ref = np.array([pins.cr32(pins.MP_FUNCS[fn](w)) for w in words], dtype=np.float32)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_laplace_transform_is_exactly_odd():
    # F^-1(u) = -F^-1(1-u) and u(2^32-1-w) = 1 - u(w): the two branches must
    # hit the same logarithm argument.
    w = _words_sample(20000, 7)
    a = O.transform(O.FN_LAPLACE_T, w)
    b = O.transform(O.FN_LAPLACE_T, (np.uint32(0xFFFFFFFF) - w).astype(np.uint32))
    assert np.array_equal(a.view(np.uint32), (-b).view(np.uint32))
    assert np.all((a < 0) == (w < 2**31))


def test_sincos_pythagoras_and_symmetry():
    w = _words_sample(20000, 8)
    c = O.transform(O.FN_COS2PI, w).astype(np.float64)
    s = O.transform(O.FN_SIN2PI, w).astype(np.float64)
    assert np.max(np.abs(c * c + s * s - 1.0)) < 4 * 2.0**-24
    wm = (np.uint32(0xFFFFFFFF) - w).astype(np.uint32)  # u -> 1 - u
    assert np.array_equal(O.transform(O.FN_COS2PI, wm), c.astype(np.float32))
    assert np.array_equal(O.transform(O.FN_SIN2PI, wm), (-s).astype(np.float32))


def _expected_noise_unit_scale(mech, words_by_elem):
    """Noise at Delta/eps = 1 from rocRAND words and mpmath transforms."""
    n = words_by_elem.size
    out = np.zeros(n, dtype=np.float32)
    for e in range(n):
        if mech == O.MECH_LAPLACE:
            out[e] = pins.cr32(pins.mp_laplace_t(words_by_elem[e]))
        else:
            base = e - (e % 2)  # lanes (0,1) pair words (0,1); lanes (2,3) pair (2,3)
            r = pins.cr32(pins.mp_gauss_r(words_by_elem[base]))
            f = pins.mp_sin2pi if e % 2 else pins.mp_cos2pi
            c = pins.cr32(f(words_by_elem[base + 1]))
            out[e] = np.float32(np.float64(r) * np.float64(c))  # product exact in binary64
    return out


@pytest.mark.parametrize("mech", [O.MECH_LAPLACE, O.MECH_GAUSSIAN])
@pytest.mark.parametrize("seed,sid,row0,M,K", [(0, 0, 0, 3, 8), (7, 259, 11, 2, 12),
                                               (2**40 + 3, 5, 2047, 2, 16)])
def test_noise_elements_from_independent_references(mech, seed, sid, row0, M, K):
    words = pins.rocrand_words(seed, sid, row0 * K, M * K)
    ref = _expected_noise_unit_scale(mech, words).reshape(M, K)
    got = O.noise(M, K, mech, 1.0, 1.0, seed, sid, row0)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_noise_scale_applied_in_binary64_then_rounded():
    # eta = RN32(fl64(s * t)); with s = 1 the transform value comes back unchanged.
    unit = O.noise(4, 64, O.MECH_LAPLACE, 1.0, 1.0, 3, 1)
    scaled = O.noise(4, 64, O.MECH_LAPLACE, 825.27, 0.5, 3, 1)
    s = np.float64(825.27) / np.float64(0.5)
    assert np.array_equal(scaled, (s * unit.astype(np.float64)).astype(np.float32))


def test_noise_row_slicing_and_streams():
    full = O.noise(40, 96, O.MECH_GAUSSIAN, 1.0, 2.0, 11, 3, 0)
    part = O.noise(9, 96, O.MECH_GAUSSIAN, 1.0, 2.0, 11, 3, 17)
    assert np.array_equal(full[17:26], part)
    other = O.noise(40, 96, O.MECH_GAUSSIAN, 1.0, 2.0, 11, 4, 0)
    assert np.mean(full == other) < 0.001
    assert not np.any(O.noise(5, 8, O.MECH_NONE, 1.0, 1.0, 0, 0))


def test_noise_rejects_bad_arguments():
    with pytest.raises(ValueError):
        O.noise(2, 6, O.MECH_LAPLACE, 1.0, 1.0, 0, 0)  # K % 4 != 0
    for d, e in [(1.0, 0.0), (1.0, -1.0), (-1.0, 1.0), (1.0, float("nan")), (float("inf"), 1.0)]:
        with pytest.raises(ValueError):
            O.noise(2, 8, O.MECH_LAPLACE, d, e, 0, 0)


N_STAT = (512, 1024)


@pytest.mark.parametrize("delta,eps", [(1.0, 1.0), (825.27, 0.5), (1.0, 16.0)])
def test_laplace_scale_moments_and_ks(delta, eps):
    b = delta / eps
    eta = O.noise(*N_STAT, O.MECH_LAPLACE, delta, eps, 0, 0).astype(np.float64).ravel()
    n = eta.size
    # E|eta| = b (Var|eta| = b^2); Var(eta) = 2 b^2 (Var of eta^2 = 20 b^4)
    assert abs(np.mean(np.abs(eta)) - b) < 6 * b / math.sqrt(n)
    assert abs(np.mean(eta * eta) - 2 * b * b) < 6 * math.sqrt(20) * b * b / math.sqrt(n)
    assert abs(np.mean(eta)) < 6 * math.sqrt(2) * b / math.sqrt(n)
    d = O.ks_statistic(eta, lambda x: O.laplace_cdf(x, b))
    assert d < 1.95 / math.sqrt(n)


@pytest.mark.parametrize("delta,eps", [(1.0, 1.0), (719.8, 2.0), (1.0, 4.0)])
def test_gaussian_scale_moments_and_ks(delta, eps):
    sg = delta / eps
    eta = O.noise(*N_STAT, O.MECH_GAUSSIAN, delta, eps, 5, 2).astype(np.float64).ravel()
    n = eta.size
    assert abs(np.mean(eta * eta) - sg * sg) < 6 * math.sqrt(2) * sg * sg / math.sqrt(n)
    assert abs(np.mean(np.abs(eta)) - sg * math.sqrt(2 / math.pi)) < 6 * sg / math.sqrt(n)
    assert abs(np.mean(eta)) < 6 * sg / math.sqrt(n)
    d = O.ks_statistic(eta, lambda x: O.gauss_cdf(x, sg))
    assert d < 1.95 / math.sqrt(n)


def test_ks_detects_wrong_scale():
    # The statistical pins are not vacuous: noise at scale 1.02 b fails the KS gate.
    eta = O.noise(*N_STAT, O.MECH_LAPLACE, 1.0, 1.0, 0, 0).astype(np.float64).ravel()
    d = O.ks_statistic(eta * 1.02, lambda x: O.laplace_cdf(x, 1.0))
    assert d > 1.95 / math.sqrt(eta.size)
