"""Pins of the oracle's mask, split, GEMM, unmask and error bounds.

References other than the oracle itself:
* torch's float32 -> bfloat16 conversion (round to nearest even) and float32 add /
  subtract on the CPU;
* exact rational arithmetic (fractions) for the GEMM on tiny inputs;
* the identity W(x + eta) - W eta = W x (Eq. add-and-then-subtract), exact in
  binary32 for small integers;
* real binary32 computations (numpy's float32 GEMM, sequential float32 loops)
  that Theorem 4's bound must cover, and the paper's observation (Table 4) that
  the masking error scales as 1/eps.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle as O
import workloads as WL


def _torch_bf16(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).to(
        torch.float32).numpy()


def test_bf16_rne_matches_torch_on_random_and_ties():
    g = np.random.Generator(np.random.PCG64(3))
    x = (g.standard_normal(200000) * np.exp(g.uniform(-30, 30, 200000))).astype(np.float32)
    # exact ties: bf16 value + half a bf16 ulp (low 16 bits = 0x8000), odd and even
    bits = (g.integers(0x00800000, 0x7F000000, 20000, dtype=np.int64).astype(np.uint32)
            & np.uint32(0xFFFF0000)) | np.uint32(0x8000)
    ties = np.concatenate([bits.view(np.float32), -bits.view(np.float32)])
    special = np.array([0.0, -0.0, 1.0, -1.0, 3.3895314e38, 1e-40, -1e-42], dtype=np.float32)
    for arr in (x, ties, special):
        assert np.array_equal(O.bf16_rne(arr).view(np.uint32), _torch_bf16(arr).view(np.uint32))


def test_split3_reconstructs_exactly():
    g = np.random.Generator(np.random.PCG64(4))
    xt = (g.standard_normal(100000) * np.exp(g.uniform(-20, 20, 100000))).astype(np.float32)
    hi, mid, lo = O.split3(xt)
    for part in (hi, mid, lo):
        assert np.array_equal(part, O.bf16_rne(part))  # each term is a bfloat16 value
    total = hi.astype(np.float64) + mid.astype(np.float64) + lo.astype(np.float64)
    assert np.array_equal(total, xt.astype(np.float64))
    assert np.all(np.abs(mid.astype(np.float64)) <= 2.0**-8 * np.abs(xt.astype(np.float64)) * 1.01)


def test_mask_and_unmask_are_single_ieee_operations():
    g = np.random.Generator(np.random.PCG64(5))
    a = (g.standard_normal(50000) * 10.0 ** g.uniform(-6, 6, 50000)).astype(np.float32)
    b = (g.standard_normal(50000) * 10.0 ** g.uniform(-6, 6, 50000)).astype(np.float32)
    ta, tb = torch.from_numpy(a), torch.from_numpy(b)
    assert np.array_equal(O.mask(a, b), (ta + tb).numpy())
    assert np.array_equal(O.unmask(a, b), (ta - tb).numpy())


def test_gemm64_exact_against_rationals():
    g = np.random.Generator(np.random.PCG64(6))
    A = g.standard_normal((3, 7)).astype(np.float32)
    W = WL.gen_w(4, 7, seed=9)
    got = O.gemm64(A, W)
    for i in range(3):
        for j in range(4):
            exact = sum(Fraction(float(A[i, k])) * Fraction(float(W[j, k])) for k in range(7))
            assert abs(Fraction(float(got[i, j])) - exact) <= abs(exact) * Fraction(1, 2**50) + \
                Fraction(1, 2**80)


@pytest.mark.parametrize("prec", [O.PREC_F32, O.PREC_BF16, O.PREC_BF16X3])
def test_exact_cancellation_on_small_integers(prec):
    # Every product and partial sum is an integer below 2^24 (and the operands
    # fit in bfloat16), so each precision mode reproduces X W^T exactly.
    M, K, N = 16, 256, 24
    X = WL.gen_int((M, K), -8, 8, 10)
    eta = WL.gen_int((M, K), -8, 8, 11)
    W = WL.gen_int((N, K), -4, 4, 12)
    r = O.masked_linear(X, W, O.MECH_NONE, 1.0, 1.0, 0, 0, prec=prec, eta=eta)
    assert np.array_equal(r["Y"].astype(np.float64), r["Yref"])
    # planted mistake: subtracting the mask instead of adding it is caught
    bad = O.unmask(O.gemm64(O.mask(X, -eta), W).astype(np.float32),
                   O.gemm64(eta, W).astype(np.float32))
    assert not np.array_equal(bad.astype(np.float64), r["Yref"])


def _fp32_path(X, eta, W, seq=False):
    """A real binary32 execution of mask -> GEMM -> unmask (float32 BLAS or a
    sequential float32 loop) -- what Theorem 4 has to bound."""
    Xt = O.mask(X, eta)
    W32 = np.asarray(W, dtype=np.float32)
    if not seq:
        R = (Xt @ W32.T).astype(np.float32)
        C = (eta @ W32.T).astype(np.float32)
    else:
        def seqdot(A):
            acc = np.zeros((A.shape[0], W32.shape[0]), dtype=np.float32)
            for k in range(A.shape[1]):
                acc = (acc + (A[:, k:k + 1] * W32[:, k][None, :]).astype(np.float32)).astype(
                    np.float32)
            return acc
        R, C = seqdot(Xt), seqdot(eta)
    return Xt, O.unmask(R, C)


@pytest.mark.parametrize("mech", [O.MECH_LAPLACE, O.MECH_GAUSSIAN])
@pytest.mark.parametrize("delta,eps", [(1.0, 1.0), (1.0, 16.0), (825.27, 0.5), (825.27, 8.0)])
@pytest.mark.parametrize("seq", [False, True])
def test_theorem4_bounds_real_binary32_execution(mech, delta, eps, seq):
    M, K, N = 8, 768 if seq else 3072, 40
    X = WL.gen_x(M, K, seed=1)
    W = WL.gen_w(N, K, seed=2)
    eta = O.noise(M, K, mech, delta, eps, 0, 1)
    Xt, Y = _fp32_path(X, eta, W, seq)
    Yref = O.gemm64(X, W)
    b = O.error_bounds(X, eta, Xt, W)
    err = np.abs(Y.astype(np.float64) - Yref)
    assert np.all(err <= b["gate"])
    pre = b["precond"]
    assert np.all(err[pre] <= b["thm4"][pre])
    assert np.mean(err) <= np.mean(b["logb"])  # Table 4: mean error below mean Eq. fp-log-bound
    # the gate is Theorem 4 wherever its precondition holds
    assert np.array_equal(b["gate"][pre], np.maximum(b["thm4"], b["rigor"])[pre])
    assert np.all(b["rigor"][pre] <= b["thm4"][pre] * (1 + 1e-6))


def test_bound_with_dropped_noise_term_is_violated():
    # planted mistake in the bound: without the S_eta term the bound fails at
    # paper-scale noise, so the gate's noise terms are load-bearing.
    M, K, N = 8, 3072, 64
    X = WL.gen_x(M, K, seed=1)
    W = WL.gen_w(N, K, seed=2)
    eta = O.noise(M, K, O.MECH_GAUSSIAN, 825.27, 0.5, 0, 1)
    Xt, Y = _fp32_path(X, eta, W)
    err = np.abs(Y.astype(np.float64) - O.gemm64(X, W))
    b = O.error_bounds(X, eta, Xt, W)
    too_tight = O.U32 * (b["Sx"] + b["St"])
    assert np.any(err > too_tight)


def test_error_scales_as_one_over_eps():
    # Table 4: in the noise-dominated regime mean |error| * eps is constant.
    M, K, N = 16, 3072, 64
    X = WL.gen_x(M, K, seed=1)
    W = WL.gen_w(N, K, seed=2)
    Yref = O.gemm64(X, W)
    means = {}
    for eps in (0.5, 2.0, 8.0):
        eta = O.noise(M, K, O.MECH_GAUSSIAN, 825.27, eps, 0, 1)
        _, Y = _fp32_path(X, eta, W)
        means[eps] = float(np.mean(np.abs(Y.astype(np.float64) - Yref)))
    assert 0.75 < (means[0.5] * 0.5) / (means[2.0] * 2.0) < 1.33
    assert 0.75 < (means[2.0] * 2.0) / (means[8.0] * 8.0) < 1.33


@pytest.mark.parametrize("K", [256, 3072])
def test_bf16_single_pass_needs_its_own_term(K):
    # Rounding the masked input to bfloat16 adds u_bf16 * S_t; at paper-scale noise
    # the binary32 bounds alone do not cover it (Eq. fp-log-bound at any K; the
    # Theorem 4 gate at small K, where gamma_K is small).
    M, N = 8, 64
    X = WL.gen_x(M, K, seed=1)
    W = WL.gen_w(N, K, seed=2)
    eta = O.noise(M, K, O.MECH_GAUSSIAN, 825.27, 2.0, 0, 1)
    Xt = O.mask(X, eta)
    R = (O.bf16_rne(Xt) @ W.T).astype(np.float32)
    C = (eta @ W.T).astype(np.float32)
    Y = O.unmask(R, C)
    err = np.abs(Y.astype(np.float64) - O.gemm64(X, W))
    b32 = O.error_bounds(X, eta, Xt, W, O.PREC_F32)
    bb = O.error_bounds(X, eta, Xt, W, O.PREC_BF16)
    assert np.mean(err > b32["logb"]) > 0.5
    if K == 256:
        assert np.any(err > b32["gate"])
    assert np.all(err <= bb["gate"])


def test_gamma_definition_domain():
    assert O.gamma(1) == pytest.approx(2.0**-24 / (1 - 2.0**-24), rel=0, abs=0)
    with pytest.raises(ValueError):
        O.gamma(2**24)
    # Eq. fp-log-bound uses gamma_{ceil(log2 d)+1}: d = 3072 -> gamma_13
    assert math.ceil(math.log2(3072)) + 1 == 13


# ------------------------------------------------------------------ binary64 path

DELTA_ACT = 1.66e8  # Theorem 3 for a Llama-3.2-3B-shaped layer with random weights


def _fp64_path(X, eta, W, seq=False):
    Xt = O.mask64(X, eta)
    W64 = np.asarray(W, dtype=np.float64)
    e64 = np.asarray(eta, dtype=np.float64)
    if not seq:
        R, C = Xt @ W64.T, e64 @ W64.T
    else:
        def seqdot(A):
            acc = np.zeros((A.shape[0], W64.shape[0]))
            for k in range(A.shape[1]):
                acc = acc + A[:, k:k + 1] * W64[:, k][None, :]
            return acc
        R, C = seqdot(Xt), seqdot(e64)
    return (R - C).astype(np.float32)


def test_mask64_is_one_binary64_addition():
    g = np.random.Generator(np.random.PCG64(4))
    x = g.standard_normal(4096).astype(np.float32)
    e = (g.standard_normal(4096) * DELTA_ACT).astype(np.float32)
    got = O.mask64(x, e)
    want = np.array([float(Fraction(float(a)) + Fraction(float(b))) for a, b in zip(x[:64], e[:64])])
    assert np.array_equal(got[:64], want)  # correctly rounded sum
    # where |eta| < 2^28 |x| the sum is exact, so x comes back unchanged
    back = (got - e.astype(np.float64)).astype(np.float32)
    exact = np.abs(e) < np.abs(x) * 2.0 ** 28
    assert exact.mean() > 0.5 and np.array_equal(back[exact], x[exact])


@pytest.mark.parametrize("delta,eps", [(1.0, 1.0), (825.27, 0.5), (DELTA_ACT, 1.0), (DELTA_ACT, 0.25)])
@pytest.mark.parametrize("seq", [False, True])
def test_f64_bound_covers_real_binary64_execution(delta, eps, seq):
    M, K, N = 4, 1024 if seq else 8192, 24
    X = WL.gen_x(M, K, seed=1)
    W = WL.gen_w(N, K, seed=2)
    eta = O.noise(M, K, O.MECH_GAUSSIAN, delta, eps, 0, 3)
    Y = _fp64_path(X, eta, W, seq)
    err = np.abs(Y.astype(np.float64) - O.gemm64(X, W))
    b = O.error_bounds_f64(X, eta, W)
    assert np.all(err <= b["bound"])
    # Theorem 4 at u = 2^-53 is gamma_K(u64) / gamma_K(u32) ~ 2^-29 of the binary32 bound
    b32 = O.error_bounds(X, eta, O.mask(X, eta), W)
    assert np.allclose(b["thm4"] / b32["thm4"], 2.0 ** -29, rtol=1e-3)


def test_f64_bound_noise_terms_are_load_bearing():
    # at the sensitivity of Theorem 3 the binary64 product roundings show: the error is
    # more than the final rounding of the exact result to binary32 could explain
    M, K, N = 4, 8192, 32
    X = WL.gen_x(M, K, seed=1)
    W = WL.gen_w(N, K, seed=2)
    eta = O.noise(M, K, O.MECH_GAUSSIAN, DELTA_ACT, 1.0, 0, 3)
    y = O.gemm64(X, W)
    err = np.abs(_fp64_path(X, eta, W, seq=True).astype(np.float64) - y)
    b = O.error_bounds_f64(X, eta, W)
    assert np.any(err > 4 * O.U32 * np.abs(y))
    assert np.all(err <= b["bound"])


def test_binary64_remedies_the_down_projection():
    # the paper's case against offloading Down in binary32: at Theorem 3's sensitivity the
    # binary32 masked product loses X entirely, the binary64 one keeps it
    M, K, N = 4, 8192, 32
    X = WL.gen_x(M, K, seed=1)
    W = WL.gen_w(N, K, seed=2)
    eta = O.noise(M, K, O.MECH_GAUSSIAN, DELTA_ACT, 1.0, 0, 3)
    y = O.gemm64(X, W)
    _, Y32 = _fp32_path(X, eta, W)
    Y64 = _fp64_path(X, eta, W)
    rel32 = np.median(np.abs(Y32 - y) / np.abs(y))
    rel64 = np.median(np.abs(Y64 - y) / np.abs(y))
    assert rel32 > 0.5  # fl32(x + eta) drops x: the binary32 result is about 0, error ~ |y|
    assert rel64 < 1e-3
