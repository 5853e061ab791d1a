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
