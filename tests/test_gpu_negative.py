"""The parity comparisons fail when they should.

Each test runs the correct GPU call, then repeats the comparison that the parity
suite makes against a copy of the oracle's computation with one mistake planted in
it (on the CPU): the wrong seed, a row offset of +-1, W transposed, one correction
element moved by 2^10 ulps, the noise added twice, the unmask left out.  The
comparison it targets must reject the planted copy and accept the correct one.
Since Theorem 4's gate is loose at these sizes (errors sit far below it), the
bit-exact comparisons of the noise, the mask and the unmask carry most of the
weight; the tests show which comparison catches which mistake.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_15039_amd as sp
import workloads as WL

pytestmark = pytest.mark.gpu

M, K, N = 37, 264, 264  # square W, so that the transposed matrix has the same shape
DELTA, EPS, SEED, SID, ROW0 = 825.27, 2.0, 3, WL.stream_id(2, 1), 40
G, OG = sp.SPLITEE_MECH_GAUSSIAN, O.MECH_GAUSSIAN


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


@pytest.fixture(scope="module")
def run():
    """The GPU path on one seeded case: eta, Xt (F32 and BF16X3), R, C and Y."""
    X = WL.gen_x(M, K, seed=1)
    W = WL.gen_w(N, K, seed=2)
    assert not np.array_equal(W, W.T)
    Xd, Wd = dev(X), dev(W).to(torch.bfloat16)
    eta = host(sp.noise(M, K, G, DELTA, EPS, SEED, SID, ROW0))
    Xt = host(sp.noise_mask(Xd, sp.SPLITEE_PREC_F32, G, DELTA, EPS, SEED, SID, ROW0))[0]
    P = sp.SPLITEE_PREC_BF16X3
    Xt3 = sp.noise_mask(Xd, P, G, DELTA, EPS, SEED, SID, ROW0)
    R = sp.masked_linear(Xt3, P, Wd)
    C = sp.correction(Wd, M, G, DELTA, EPS, SEED, SID, ROW0, P)
    Yu = host(sp.unmask(R, C))
    Y = host(sp.masked_linear_fused(Xd, Wd, C, G, DELTA, EPS, SEED, SID, ROW0, P))
    return dict(X=X, W=W, eta=eta, Xt=Xt, R=host(R), C=host(C), Yu=Yu, Y=Y)


def _noise_matches(r, seed=SEED, row0=ROW0):
    return np.array_equal(bits(r["eta"]), bits(O.noise(M, K, OG, DELTA, EPS, seed, SID, row0)))


def _gate_holds(r, W_ref):
    eta = O.noise(M, K, OG, DELTA, EPS, SEED, SID, ROW0)
    b = O.error_bounds(r["X"], eta, O.mask(r["X"], eta), W_ref, O.PREC_BF16X3)
    return bool(np.all(np.abs(r["Y"].astype(np.float64) - O.gemm64(r["X"], W_ref)) <= b["gate"]))


def test_wrong_seed_fails_the_noise_comparison(run):
    assert _noise_matches(run)
    assert not _noise_matches(run, seed=SEED + 1)


@pytest.mark.parametrize("shift", [1, -1])
def test_row_offset_fails_the_noise_comparison(run, shift):
    assert not _noise_matches(run, row0=ROW0 + shift)
    # the rows themselves are right, only placed one row over
    ref = O.noise(M, K, OG, DELTA, EPS, SEED, SID, ROW0 + shift)
    got = run["eta"]
    if shift > 0:
        assert np.array_equal(bits(got[1:]), bits(ref[:-1]))
    else:
        assert np.array_equal(bits(got[:-1]), bits(ref[1:]))


def test_transposed_w_fails_the_theorem4_gate(run):
    assert _gate_holds(run, run["W"])
    assert not _gate_holds(run, np.ascontiguousarray(run["W"].T))


def test_perturbed_correction_element_fails_the_unmask_comparison(run):
    R, C = run["R"], run["C"]
    assert np.array_equal(bits(run["Yu"]), bits(O.unmask(R, C)))
    Cp = C.copy()
    i, j = 11, 123
    Cp[i, j] = (C[i, j].view(np.uint32) + np.uint32(1 << 10)).view(np.float32)  # 2^10 ulps up
    bad = bits(run["Yu"]) != bits(O.unmask(R, Cp))
    assert bad.sum() == 1 and bad[i, j]


def test_noise_added_twice_fails_the_mask_and_product_comparisons(run):
    X, eta, W = run["X"], run["eta"], run["W"]
    once, twice = O.mask(X, eta), O.mask(O.mask(X, eta), eta)
    assert np.array_equal(bits(run["Xt"]), bits(once))
    assert not np.array_equal(bits(run["Xt"]), bits(twice))
    # R against the oracle's product within the dot-product bound (three bfloat16 passes)
    for xt, ok in ((once, True), (twice, False)):
        A = O.gemm_operand(xt, O.PREC_BF16X3)
        within = np.all(np.abs(run["R"].astype(np.float64) - O.gemm64(A, W)) <= O.dot_bound(A, W, planes=3))
        assert bool(within) == ok


def test_missing_unmask_fails_the_theorem4_gate(run):
    # comparing R (the masked product, no correction subtracted) with X W^T
    X, W = run["X"], run["W"]
    eta = O.noise(M, K, OG, DELTA, EPS, SEED, SID, ROW0)
    b = O.error_bounds(X, eta, O.mask(X, eta), W, O.PREC_BF16X3)
    err = np.abs(run["R"].astype(np.float64) - O.gemm64(X, W))
    assert np.mean(err > b["gate"]) > 0.9
