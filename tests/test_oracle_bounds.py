"""Pins of the oracle's error bounds from above: their values, and inputs that come
close to them.

``oracle.error_bounds`` (Theorem 4, Eq. fp-log-bound and the gate) and
``oracle.error_bounds_f64`` are checked elsewhere never to be exceeded by real
binary32 / binary64 executions.  That alone would let a bound that is 2x or 10x too
loose pass.  Here:

* values worked out by hand from Def. 6 (gamma_n = n u / (1 - n u)), Theorem 4 and
  Eq. fp-log-bound for a tiny dyadic case are written into the test as numbers;
* constructed inputs make a real execution of mask -> dot product -> unmask reach
  most of the bound: the correction's sum drops each small term (every addition
  rounds down by almost u of the running sum) while the masked product's sum rounds
  each one up, so the two errors add; a sequential sum nearly attains Theorem 4
  (gamma_K), a pairwise sum nearly attains Eq. fp-log-bound (gamma_{ceil(log2 K)+1}),
  a single bfloat16 rounding of the masked input nearly attains the extra term of the
  single-pass mode, and the binary64 path nearly attains its own bound;
* the same checks run against a copy of the oracle whose bound is loosened by 2x
  fail, so they would catch a bound that is too loose (a planted mistake, in the
  oracle, on the CPU).

The real executions are IEEE binary32 / binary64 operations in numpy scalars and
torch's bfloat16 conversion, not oracle code.
"""
import math
from fractions import Fraction as F

import numpy as np
import pytest
import torch

import oracle as O

U = 2.0 ** -24
DELTA = 2.0 ** -10  # the offset of the small terms in the constructions below


# ---------------------------------------------------------------- hand-derived values

def _tiny():
    # K = 4, one token, one output; every value dyadic so that Xt = X + eta is exact
    X = np.array([[1.0, -2.0, 0.5, 0.0]], dtype=np.float32)
    eta = np.array([[0.25, 1.0, -0.5, 4.0]], dtype=np.float32)
    W = np.array([[1.0, 0.5, -2.0, 0.25]], dtype=np.float32)
    Xt = O.mask(X, eta)
    return X, eta, Xt, W


def test_tiny_case_sums_by_hand():
    X, eta, Xt, W = _tiny()
    assert Xt.tolist() == [[1.25, -1.0, 0.0, 4.0]]
    b = O.error_bounds(X, eta, Xt, W)
    # S_x = 1 + 1 + 1 + 0, S_t = 1.25 + 0.5 + 0 + 1, S_eta = 0.25 + 0.5 + 1 + 1
    assert (b["Sx"][0, 0], b["St"][0, 0], b["Se"][0, 0]) == (3.0, 2.75, 2.75)


def test_theorem4_value_by_hand():
    X, eta, Xt, W = _tiny()
    b = O.error_bounds(X, eta, Xt, W)
    # gamma_4 = 4 2^-24 / (1 - 4 2^-24) = 1 / 4194303;  Theorem 4:
    # gamma_4 (3 + 2.75 + 2.75) + 2^-24 3 = 17 / 8388606 + 3 / 16777216
    thm4 = F(17, 8388606) + F(3, 16777216)
    assert F(float(b["thm4"][0, 0])) == pytest.approx(thm4, rel=1e-15)
    assert float(b["thm4"][0, 0]) == pytest.approx(2.20537234e-06, rel=1e-8)


def test_fp_log_bound_value_by_hand():
    X, eta, Xt, W = _tiny()
    b = O.error_bounds(X, eta, Xt, W)
    # ceil(log2 4) + 1 = 3;  gamma_3 = 3 / 16777213;  8.5 gamma_3 + 3 2^-24
    logb = F(51, 33554426) + F(3, 16777216)
    assert F(float(b["logb"][0, 0])) == pytest.approx(logb, rel=1e-15)
    assert float(b["logb"][0, 0]) == pytest.approx(1.69873265e-06, rel=1e-8)


def test_gate_and_rigorous_term_by_hand():
    X, eta, Xt, W = _tiny()
    b = O.error_bounds(X, eta, Xt, W)
    # precondition S_eta <= (K - 1) S_x: 2.75 <= 9
    assert bool(b["precond"][0, 0])
    u = F(1, 2 ** 24)
    g4 = F(1, 4194303)
    # R in binary32 (a fused multiply-add chain): c_R = gamma_4.  C may come from the
    # bfloat16 matrix cores on three planes: 4 group steps (3 planes x 1 group + 1 extra),
    # c_C = (gamma_4 + 8 u (1 + gamma_4)) (1 + 2^-6), which exceeds gamma_4 at this tiny K
    cC = (g4 + 8 * u * (1 + g4)) * F(65, 64)
    assert F(b["c_R"]) == pytest.approx(g4, rel=1e-15)
    assert F(b["c_C"]) == pytest.approx(cC, rel=1e-15)
    # rigorous term: (1 + u) (c_R S_t + c_C S_eta + u (S_x + S_eta)) + u S_x
    rig = (1 + u) * (g4 * F(11, 4) + cC * F(11, 4) + u * F(23, 4)) + 3 * u
    assert F(float(b["rigor"][0, 0])) == pytest.approx(rig, rel=1e-15)
    # so at K = 4 the gate is the rigorous term, above Theorem 4 (17/8388606 + 3/2^24)
    assert b["gate"][0, 0] == b["rigor"][0, 0] > b["thm4"][0, 0]


def test_gate_is_theorem4_from_moderate_k():
    # from K = 16 on every kernel's accumulation coefficient is gamma_K, so wherever the
    # precondition holds the gate is Theorem 4 itself
    for K in (16, 64, 2560, 9728):
        assert O.acc_coeff(K, 3) == O.gamma(K) and O.acc_coeff(K, 1) == O.gamma(K)
    assert O.acc_coeff(8, 3) > O.gamma(8)


def test_bf16_terms_by_hand():
    X, eta, Xt, W = _tiny()
    b = O.error_bounds(X, eta, Xt, W, O.PREC_BF16)
    # single pass adds u_bf16 S_t (1 + gamma_4) = 2^-8 2.75 (1 + 1/4194303) to both bounds
    extra = F(11, 4 * 256) * (1 + F(1, 4194303))
    assert F(float(b["thm4"][0, 0])) == pytest.approx(F(17, 8388606) + F(3, 16777216) + extra, rel=1e-15)
    # and u_bf16 S_t (1 + gamma_3) to Eq. fp-log-bound
    extra3 = F(11, 4 * 256) * (1 + F(3, 16777213))
    assert F(float(b["logb"][0, 0])) == pytest.approx(F(51, 33554426) + F(3, 16777216) + extra3, rel=1e-15)


def test_f64_bound_by_hand():
    X, eta, Xt, W = _tiny()
    b = O.error_bounds_f64(X, eta, W)
    u = F(1, 2 ** 53)
    g4 = 4 * u / (1 - 4 * u)
    # E = gamma_4(u64) (S_t + S_eta) + 2 u64 S_t; bound = E + (2^-24 + 2 u64)(S_x + E);
    # Theorem 4 at u64: gamma_4(u64) (S_x + S_t + S_eta) + u64 S_x
    E = g4 * F(11, 2) + 2 * u * F(11, 4)
    assert F(float(b["E"][0, 0])) == pytest.approx(E, rel=1e-15)
    assert F(float(b["bound"][0, 0])) == pytest.approx(E + (F(1, 2 ** 24) + 2 * u) * (3 + E), rel=1e-15)
    assert F(float(b["thm4"][0, 0])) == pytest.approx(g4 * F(17, 2) + 3 * u, rel=1e-15)


@pytest.mark.parametrize("K,idx", [(1, 1), (2, 2), (3, 3), (4, 3), (5, 4), (8, 4), (9, 5), (2560, 13),
                                   (3072, 13), (4096, 13), (9728, 15)])
def test_fp_log_bound_index(K, idx):
    # Eq. fp-log-bound replaces gamma_d by gamma_{ceil(log2 d)+1}: with every sum 1 it is
    # (3 gamma_idx + u) exactly; at K <= 2 the two indices agree, so the bound equals Theorem 4's
    X = np.ones((1, K), dtype=np.float32)
    eta = np.zeros((1, K), dtype=np.float32)
    W = np.full((1, K), 1.0 / K, dtype=np.float32) if K & (K - 1) == 0 else np.ones((1, K), np.float32)
    b = O.error_bounds(X, eta, X, W)
    s = float(b["Sx"][0, 0])
    want = (2 * s) * (idx * U / (1 - idx * U)) + U * s
    assert float(b["logb"][0, 0]) == pytest.approx(want, rel=1e-13)
    if K <= 2:
        assert b["logb"][0, 0] == b["thm4"][0, 0]


# ------------------------------------------------------------- near-attaining inputs

def _construction(K, positions, u=U, dtype=np.float32):
    """X, eta, W (all ones) for which both sums of the unmask err the same way.

    eta: 1 at k = 0 and u (1 - DELTA) at `positions`, zero elsewhere -- each small term
    is below half an ulp of the running sum 1, so adding it rounds down to 1.
    Xt = X + eta: 1 at k = 0 and u (1 + DELTA) at `positions` -- above half an ulp, so
    each addition rounds up by a whole ulp (2u) and gains u (1 - DELTA).
    X = Xt - eta: 2 u DELTA at `positions`; all values exact in the format."""
    eta = np.zeros((1, K), dtype=dtype)
    xt = np.zeros((1, K), dtype=dtype)
    eta[0, 0] = xt[0, 0] = 1.0
    eta[0, positions] = u * (1 - DELTA)
    xt[0, positions] = u * (1 + DELTA)
    X = (xt - eta).astype(dtype)
    assert np.array_equal((X + eta).astype(dtype), xt)  # the mask is exact
    W = np.ones((1, K), dtype=dtype)
    return X, eta, xt, W


def _seq(v, dtype):
    acc = dtype(0)
    for x in v:
        acc = dtype(acc + dtype(x))
    return acc


def _pairwise(v, dtype):
    v = [dtype(x) for x in v]
    while len(v) > 1:
        v = [dtype(v[i] + v[i + 1]) for i in range(0, len(v), 2)]
    return v[0]


def _unmask_error(X, eta, xt, W, summ, dtype):
    """|fl(fl(Xt . w) - fl(eta . w)) - x . w| for one output, products w x exact (w = 1)."""
    R = summ((xt[0] * W[0]).astype(dtype), dtype)
    C = summ((eta[0] * W[0]).astype(dtype), dtype)
    Y = dtype(R - C)
    exact = sum(F(float(a)) * F(float(w)) for a, w in zip(X[0], W[0]))
    return float(abs(F(float(Y)) - exact))


def _loose(bounds_fn, factor=2.0, keys=("thm4", "logb", "gate", "rigor", "bound", "E")):
    """A copy of a bound function with its bounds multiplied by `factor`: a planted mistake."""
    def fn(*args, **kw):
        b = dict(bounds_fn(*args, **kw))
        for k in keys:
            if k in b:
                b[k] = b[k] * factor
        return b
    return fn


def _attains(bounds_fn, key, K, summ, frac, u=U, dtype=np.float32, f64=False):
    positions = list(range(1, K)) if summ is _seq else [1 << j for j in range(int(math.log2(K)))]
    X, eta, xt, W = _construction(K, positions, u, dtype)
    err = _unmask_error(X, eta, xt, W, summ, dtype)
    b = bounds_fn(X, eta, W) if f64 else bounds_fn(X, eta, xt, W)
    bound = float(b[key][0, 0])
    return err <= bound and err >= frac * bound, err, bound


@pytest.mark.parametrize("K", [64, 512])
@pytest.mark.parametrize("key", ["thm4", "gate"])
def test_theorem4_nearly_attained_by_sequential_sums(K, key):
    # error 2 (K - 1) u (1 - DELTA) against about 2 K u: Theorem 4 is within (K - 1) / K of tight
    ok, err, bound = _attains(O.error_bounds, key, K, _seq, 0.95)
    assert ok, (err, bound, err / bound)
    assert not _attains(_loose(O.error_bounds), key, K, _seq, 0.95)[0]


@pytest.mark.parametrize("K", [64, 1024])
def test_fp_log_bound_nearly_attained_by_pairwise_sums(K):
    # pairwise summation puts log2 K additions on each path, all rounding the same way:
    # error 2 log2(K) u (1 - DELTA) against about 2 (log2(K) + 1) u
    L = int(math.log2(K))
    ok, err, bound = _attains(O.error_bounds, "logb", K, _pairwise, 0.97 * L / (L + 1))
    assert ok, (err, bound, err / bound)
    assert not _attains(_loose(O.error_bounds), "logb", K, _pairwise, 0.97 * L / (L + 1))[0]
    # the same input summed sequentially exceeds Eq. fp-log-bound: that bound is the
    # paper's tighter form for a pairwise (library) order, not a bound for every order
    ok_seq, err_seq, bound_seq = _attains(O.error_bounds, "logb", K, _seq, 0.0)
    assert err_seq > bound_seq


def test_bf16_input_rounding_term_nearly_attained():
    # single pass: every masked value 1 + 2^-8 (1 - DELTA) rounds down to the bfloat16 1,
    # so R = K exactly while X W^T = K 2^-8 (1 - DELTA); the u_bf16 S_t term is tight
    K = 64
    eta = np.ones((1, K), dtype=np.float32)
    X = np.full((1, K), 2.0 ** -8 * (1 - DELTA), dtype=np.float32)
    Xt = O.mask(X, eta)
    W = np.ones((1, K), dtype=np.float32)
    xb = torch.from_numpy(Xt).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.all(xb == 1.0)
    R = _seq(xb[0], np.float32)
    C = _seq(eta[0], np.float32)
    err = float(abs(F(float(np.float32(R - C))) - sum(F(float(x)) for x in X[0])))
    for fn, frac in ((O.error_bounds, 0.98), (_loose(O.error_bounds), None)):
        b = fn(X, eta, Xt, W, O.PREC_BF16)
        for key in ("thm4", "gate"):
            bound = float(b[key][0, 0])
            if frac is None:
                assert err < 0.98 * bound
            else:
                assert frac * bound <= err <= bound, (key, err, bound)


@pytest.mark.parametrize("K", [64, 512])
def test_f64_bound_nearly_attained_by_sequential_sums(K):
    # the binary64 path (mask, both products and the unmask in binary64, then one rounding
    # to binary32) on the construction at u = 2^-53: error 2 (K - 1) u64 (1 - DELTA), about
    # (K - 1) / (K + 1) of the bound (whose mask term adds 2 u64 S_t)
    u64 = 2.0 ** -53
    positions = list(range(1, K))
    X, eta, xt, W = _construction(K, positions, u64, np.float64)
    X32, eta32 = X.astype(np.float32), eta.astype(np.float32)
    assert np.array_equal(X32.astype(np.float64), X) and np.array_equal(eta32.astype(np.float64), eta)
    assert np.array_equal(O.mask64(X32, eta32), xt)
    R = _seq(xt[0], np.float64)
    C = _seq(eta[0], np.float64)
    Y = np.float32(np.float64(R - C))
    err = float(abs(F(float(Y)) - sum(F(float(x)) for x in X[0])))
    b = O.error_bounds_f64(X32, eta32, W.astype(np.float32))
    bound = float(b["bound"][0, 0])
    assert 0.95 * (K - 1) / (K + 1) * bound <= err <= bound, (err, bound, err / bound)
    lb = _loose(O.error_bounds_f64)(X32, eta32, W.astype(np.float32))
    assert err < 0.95 * (K - 1) / (K + 1) * float(lb["bound"][0, 0])
