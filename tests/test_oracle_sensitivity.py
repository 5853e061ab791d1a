"""Pins of the noise-scale oracle (oracle/sensitivity.py) against what the paper
and the mathematics fix: the bounds of Theorems 1-3 are never exceeded by the
functions they bound (sampled and adversarial neighbouring inputs), are
attained by constructed inputs where the proofs' inequalities are equalities,
the spectral norm meets its closed forms, the power method approaches it from
below, and the per-token eps composes back to the total (Prop. "Sequential
Composition")."""
import math

import numpy as np
import pytest

from oracle import sensitivity as S


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


# ------------------------------------------------------------- normalisation

@pytest.mark.parametrize("rms", [True, False])
def test_normalized_vectors_have_norm_sqrt_d(rms):
    # Prop. "z-standard-norm" (gamma = 0) and Prop. "standard-norm-bound" (gamma > 0)
    g = rng(1)
    for d in (4, 37, 3072):
        x = g.standard_normal(d) * 3 + 1
        assert np.linalg.norm(S.normalize(x, 0.0, rms)) == pytest.approx(math.sqrt(d), rel=1e-12)
        assert np.linalg.norm(S.normalize(x, 1e-3, rms)) <= math.sqrt(d)


# ----------------------------------------------------------------- Theorem 1

@pytest.mark.parametrize("d,j,c", [(8, 3, 1.0), (3072, 17, 0.37), (2560, 0, -2.5)])
def test_ln_bound_attained_for_one_hot_alpha(d, j, c):
    # alpha = c e_j, x = e_j, y = -e_j (gamma = 0): LN(x) - LN(y) = 2 c sqrt(d) e_j, every
    # inequality of the proof is an equality
    alpha = np.zeros(d)
    alpha[j] = c
    e = np.zeros(d)
    e[j] = 1.0
    diff = np.linalg.norm(S.layer_norm(e, alpha) - S.layer_norm(-e, alpha))
    assert diff == pytest.approx(S.delta_ln(d, alpha), rel=1e-12)
    assert S.delta_ln(d, alpha) == pytest.approx(2 * abs(c) * math.sqrt(d), rel=1e-12)


def test_ln_bound_with_unit_alpha_is_2_d_three_quarters():
    # ||1||_4 = d^(1/4): the bound for an untrained RMSNorm scale is 2 d^(3/4)
    for d in (16, 2560, 3072):
        assert S.delta_ln(d, np.ones(d)) == pytest.approx(2 * d ** 0.75, rel=1e-12)


@pytest.mark.parametrize("rms", [True, False])
def test_ln_bound_holds_on_samples(rms):
    g = rng(2)
    d = 64
    for trial in range(200):
        alpha = g.standard_normal(d) * (0.1 + trial % 5)
        beta = g.standard_normal(d)
        x, y = g.standard_normal(d) * 10, g.standard_normal(d) ** 3
        if trial % 3 == 0:  # adversarial: all mass on the largest |alpha| coordinate, opposite signs
            j = int(np.argmax(np.abs(alpha)))
            x = np.zeros(d)
            x[j] = 1.0
            y = -x
        diff = np.linalg.norm(S.layer_norm(x, alpha, beta, 1e-6, rms) - S.layer_norm(y, alpha, beta, 1e-6, rms))
        assert diff <= S.delta_ln(d, alpha) * (1 + 1e-12)


# ----------------------------------------------------------------- Theorem 2

def test_att_bound_attained_with_one_token():
    # n = 1: att(x) - att(y) = W_val (alpha (.) (xhat - yhat)); alpha = e_j and
    # W_val = diag(s) with s_j its largest entry make every inequality an equality
    d, j = 16, 5
    alpha = np.zeros(d)
    alpha[j] = 1.5
    s = np.linspace(0.1, 1.0, d)
    s[j] = 3.0
    w_val = np.diag(s)
    w = rng(3).standard_normal((d, d))
    e = np.zeros(d)
    e[j] = 1.0
    diff = np.linalg.norm(S.attention(e, [e], w, w, w_val, alpha) - S.attention(-e, [-e], w, w, w_val, alpha))
    assert diff == pytest.approx(S.delta_att(d, alpha, S.spectral_norm(w_val)), rel=1e-12)


def test_att_bound_holds_on_neighbouring_prompts():
    g = rng(4)
    d, n = 12, 6
    for trial in range(100):
        alpha = g.standard_normal(d)
        beta = g.standard_normal(d) * 0.3
        wq, wk, wv = (g.standard_normal((d, d)) for _ in range(3))
        xs = [g.standard_normal(d) * 2 for _ in range(n)]
        pos = trial % n
        y = g.standard_normal(d) * 5 if trial % 2 else -xs[pos]
        ys = list(xs)
        ys[pos] = y  # neighbouring prompt: one token replaced, also as the query
        diff = np.linalg.norm(S.attention(xs[pos], xs, wq, wk, wv, alpha, beta, 1e-6)
                              - S.attention(y, ys, wq, wk, wv, alpha, beta, 1e-6))
        assert diff <= S.delta_att(d, alpha, S.spectral_norm(wv)) * (1 + 1e-12)


# ----------------------------------------------------------------- Theorem 3

def test_act_bound_holds_on_samples():
    g = rng(5)
    d = 16
    worst = 0.0
    for trial in range(200):
        alpha = g.standard_normal(d)
        beta = g.standard_normal(d) * 0.5
        wu, wg = g.standard_normal((d, d)), g.standard_normal((d, d))
        x, y = g.standard_normal(d) * 3, g.standard_normal(d) * 3
        if trial % 4 == 0:
            y = -x
        diff = np.linalg.norm(S.activation(x, wu, wg, alpha, beta, 1e-6) - S.activation(y, wu, wg, alpha, beta, 1e-6))
        bound = S.delta_act(d, alpha, beta, S.spectral_norm(wu), S.spectral_norm(wg))
        assert diff <= bound * (1 + 1e-12)
        worst = max(worst, diff / bound)
    assert worst > 0.0


def test_act_bound_grows_with_beta_and_both_norms():
    d = 32
    alpha = np.ones(d)
    base = S.delta_act(d, alpha, None, 1.0, 1.0)
    assert base == pytest.approx(2 * math.sqrt(d) * (math.sqrt(d) * d ** 0.25) ** 2, rel=1e-12)
    assert S.delta_act(d, alpha, np.ones(d), 1.0, 1.0) > base
    assert S.delta_act(d, alpha, None, 2.0, 3.0) == pytest.approx(6 * base, rel=1e-12)


# ------------------------------------------------------------- spectral norm

def test_spectral_norm_closed_forms():
    g = rng(6)
    dvals = g.standard_normal(40)
    assert S.spectral_norm(np.diag(dvals)) == pytest.approx(np.max(np.abs(dvals)), rel=1e-13)
    q, _ = np.linalg.qr(g.standard_normal((50, 50)))
    assert S.spectral_norm(-3.25 * q) == pytest.approx(3.25, rel=1e-12)
    u, v = g.standard_normal(30), g.standard_normal(70)
    assert S.spectral_norm(np.outer(u, v)) == pytest.approx(np.linalg.norm(u) * np.linalg.norm(v), rel=1e-12)
    w = g.standard_normal((60, 90))
    s = S.spectral_norm(w)
    assert s <= np.linalg.norm(w) <= math.sqrt(60) * s


def test_power_iteration_rises_to_the_spectral_norm():
    g = rng(7)
    m, n = 80, 120
    uu, _ = np.linalg.qr(g.standard_normal((m, m)))
    vv, _ = np.linalg.qr(g.standard_normal((n, n)))
    s = np.linspace(1.0, 0.1, m)
    s[0] = 2.0  # a spectral gap of 2: the method converges fast
    w = uu @ np.diag(s) @ vv[:m]
    sig = S.power_iteration(w, g.standard_normal(n), 60)
    assert np.all(np.diff(sig) >= -1e-14)
    assert np.all(sig <= 2.0 * (1 + 1e-12))
    assert sig[-1] == pytest.approx(2.0, rel=1e-12)


# ------------------------------------------------------------- composition

@pytest.mark.parametrize("eps,n", [(1.0, 1), (4.0, 128), (16.0, 1000)])
def test_per_token_eps_composes_to_the_total(eps, n):
    e = S.eps_per_token(eps, n)
    assert math.sqrt(sum([e * e] * n)) == pytest.approx(eps, rel=1e-12)
