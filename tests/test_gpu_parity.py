"""GPU parity: every C entry point against the oracle on the same seeded inputs.

Bar: bit-exact for the noise, the mask / split and the unmask given (R, C);
the Higham dot-product bound for R and C alone; the Theorem-4 gate (never
looser than the paper's bound where it applies) for the unmasked output.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_15039_amd as sp
import workloads as WL

pytestmark = pytest.mark.gpu

DEV = "cuda"
MECH = {"laplace": (sp.SPLITEE_MECH_LAPLACE, O.MECH_LAPLACE),
        "gaussian": (sp.SPLITEE_MECH_GAUSSIAN, O.MECH_GAUSSIAN),
        "none": (sp.SPLITEE_MECH_NONE, O.MECH_NONE)}
PREC = {"f32": (sp.SPLITEE_PREC_F32, O.PREC_F32), "bf16": (sp.SPLITEE_PREC_BF16, O.PREC_BF16),
        "bf16x3": (sp.SPLITEE_PREC_BF16X3, O.PREC_BF16X3)}


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def dev_w(W, w_dtype="bf16"):
    t = dev(W)
    return t.to(torch.bfloat16) if w_dtype == "bf16" else t


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


# ------------------------------------------------------------------------ noise

@pytest.mark.parametrize("mech", ["laplace", "gaussian", "none"])
@pytest.mark.parametrize("delta,eps,seed,sid,row0,M,K,ld", [
    (1.0, 1.0, 0, 0, 0, 32, 512, 512),
    (825.27, 0.5, 7, (3 << 8) | 2, 5, 37, 20, 24),
    (1.0, 16.0, 2**63 + 11, 2**40, 2**33 + 1, 3, 3072, 3072),
    (0.0, 1.0, 1, 1, 0, 4, 8, 8)])
def test_noise_bit_exact(mech, delta, eps, seed, sid, row0, M, K, ld):
    g, o = MECH[mech]
    eta = torch.full((M, ld), float("nan"), device=DEV)
    sp.splitee_noise_gen(eta, ld, M, K, g, delta, eps, seed, sid, row0)
    got = host(eta)
    ref = O.noise(M, K, o, delta, eps, seed, sid, row0)
    assert np.array_equal(bits(got[:, :K]), bits(ref))
    assert np.all(np.isnan(got[:, K:]))  # padding columns untouched


# Launch shapes of the row-walking noise kernel: below 2^17 Philox blocks a launch
# gives each lane half a block, above it a whole block; rows past 65535 are walked
# by the y dimension's stride.  Every shape must give the oracle's bits.
@pytest.mark.parametrize("mech", ["laplace", "gaussian"])
@pytest.mark.parametrize("M,K", [(130, 4104), (127, 4104), (65537, 8), (70001, 4)])
def test_noise_bit_exact_launch_shapes(mech, M, K):
    g, o = MECH[mech]
    eta = torch.full((M, K), float("nan"), device=DEV)
    sp.splitee_noise_gen(eta, K, M, K, g, 3.5, 0.75, 21, 6, 9)
    ref = O.noise(M, K, o, 3.5, 0.75, 21, 6, 9)
    assert np.array_equal(bits(host(eta)), bits(ref))


def _words(n, seed):
    from tests import pins
    g = np.random.Generator(np.random.PCG64(seed))
    return np.concatenate([pins.edge_words(), g.integers(0, 2**32, n, dtype=np.uint64).astype(np.uint32)])


@pytest.mark.parametrize("fn", [0, 1, 2, 3])
@pytest.mark.parametrize("force_slow", [0, 1])
def test_transform_correctly_rounded(fn, force_slow):
    w = _words(100000 if not force_slow else 20000, 40 + fn)
    wd = dev(w.view(np.int32))
    out = torch.empty(w.size, dtype=torch.float32, device=DEV)
    sp.splitee_transform_probe(wd, w.size, fn, force_slow, out)
    assert np.array_equal(bits(host(out)), bits(O.transform(fn, w)))


@pytest.mark.parametrize("fn", [0, 1, 2, 3])
def test_transform_fast_and_slow_paths_agree_on_all_words(fn):
    # every 32-bit word: the binary64 path (with its boundary check) and the
    # double-double path give the same binary32 value
    chunk = 1 << 28
    out_f = torch.empty(chunk, dtype=torch.float32, device=DEV)
    out_s = torch.empty(chunk, dtype=torch.float32, device=DEV)
    for c in range((1 << 32) // chunk):
        w = torch.arange(c * chunk, (c + 1) * chunk, dtype=torch.int64, device=DEV)
        w = (w - (1 << 32) * (w >= (1 << 31)).to(torch.int64)).to(torch.int32)
        sp.splitee_transform_probe(w, chunk, fn, 0, out_f)
        sp.splitee_transform_probe(w, chunk, fn, 1, out_s)
        bad = int((out_f.view(torch.int32) != out_s.view(torch.int32)).sum().item())
        assert bad == 0, "chunk %d: %d words differ" % (c, bad)
        del w


def test_noise_rows_are_bank_rows():
    # a decode step at positions [t, t+M) draws exactly rows t..t+M-1 of the bank's mask
    K, t, M = 2560, 1500, 16
    bank = sp.noise(2048, K, sp.SPLITEE_MECH_GAUSSIAN, 719.8, 2.0, 0, WL.stream_id(3, 0))
    step = sp.noise(M, K, sp.SPLITEE_MECH_GAUSSIAN, 719.8, 2.0, 0, WL.stream_id(3, 0), row0=t)
    assert torch.equal(bank[t:t + M].view(torch.int32), step.view(torch.int32))


@pytest.mark.parametrize("mech", ["laplace", "gaussian", "none"])
def test_noise_gen_multi_bit_exact(mech):
    # the blocks of one launch are the single-block noise, element for element
    g, o = MECH[mech]
    M, row0, seed = 7, 123, 2**40 + 9
    Ks = (3072, 264, 8192, 8)
    lds = (3072, 272, 8200, 12)
    sids = (WL.stream_id(1, 0), WL.stream_id(1, 1), 99, 2**50 + 3)
    etas = [torch.full((M, ld), float("nan"), device=DEV) for ld in lds]
    sp.splitee_noise_gen_multi(etas, lds, Ks, sids, M, g, 825.27, 2.0, seed, row0)
    for eta, K, sid in zip(etas, Ks, sids):
        got = host(eta)
        assert np.array_equal(bits(got[:, :K]), bits(O.noise(M, K, o, 825.27, 2.0, seed, sid, row0)))
        assert np.all(np.isnan(got[:, K:]))


def test_noise_gen_multi_eight_blocks_equal_single_calls():
    M, K = 16, 2560
    sids = [WL.stream_id(5, q) for q in range(8)]
    etas = [torch.empty((M, K), device=DEV) for _ in sids]
    sp.splitee_noise_gen_multi(etas, [K] * 8, [K] * 8, sids, M, sp.SPLITEE_MECH_GAUSSIAN, 719.8, 2.0, 4, 1000)
    for eta, sid in zip(etas, sids):
        one = sp.noise(M, K, sp.SPLITEE_MECH_GAUSSIAN, 719.8, 2.0, 4, sid, row0=1000)
        assert torch.equal(eta.view(torch.int32), one.view(torch.int32))


@pytest.mark.parametrize("mech", ["laplace", "gaussian"])
def test_noise_gen_multi_repetitions_are_layers(mech):
    # repetition r of block q: output at eta[q] + r * rep_strides[q], stream id sid[q] + 256 r,
    # i.e. the masks of layer r when stream ids are (layer << 8) | group
    g, o = MECH[mech]
    M, L, row0, seed = 3, 5, 1024, 11
    Ks = (2560, 4096, 9728)
    bufs = [torch.full((L, M, K + 4), float("nan"), device=DEV) for K in Ks]
    sids = [WL.stream_id(0, q) for q in range(len(Ks))]
    sp.splitee_noise_gen_multi(bufs, [K + 4 for K in Ks], Ks, sids, M, g, 719.8, 2.0, seed, row0, reps=L,
                               rep_strides=[M * (K + 4) for K in Ks], rep_sid_step=256)
    for q, (buf, K) in enumerate(zip(bufs, Ks)):
        got = host(buf)
        for r in range(L):
            ref = O.noise(M, K, o, 719.8, 2.0, seed, WL.stream_id(r, q), row0)
            assert np.array_equal(bits(got[r, :, :K]), bits(ref)), (q, r)
        assert np.all(np.isnan(got[:, :, K:]))


# ------------------------------------------------------------------------- mask

@pytest.mark.parametrize("prec", ["f32", "bf16", "bf16x3"])
@pytest.mark.parametrize("M,K", [(32, 512), (37, 264), (1, 8)])
def test_mask_bit_exact(prec, M, K):
    gp, op = PREC[prec]
    X = WL.gen_x(M, K, seed=3)
    eta = O.noise(M, K, O.MECH_LAPLACE, 825.27, 0.5, 0, 9)
    Xt = sp.mask(dev(X), dev(eta), gp)
    got = host(Xt)
    xt = O.mask(X, eta)
    if prec == "f32":
        assert np.array_equal(bits(got[0]), bits(xt))
    elif prec == "bf16":
        assert np.array_equal(got[0].view(np.uint16), O.bf16_bits(O.bf16_rne(xt)))
    else:
        for p, ref in enumerate(O.split3(xt)):
            assert np.array_equal(got[p].view(np.uint16), O.bf16_bits(ref))


def test_unmask_bit_exact():
    g = np.random.Generator(np.random.PCG64(12))
    R = (g.standard_normal((33, 300)) * 1e3).astype(np.float32)
    C = (R + g.standard_normal((33, 300)).astype(np.float32)).astype(np.float32)
    Y = sp.unmask(dev(R), dev(C))
    assert np.array_equal(bits(host(Y)), bits(O.unmask(R, C)))


# ------------------------------------------------------------- GEMM alone (R, C)

@pytest.mark.parametrize("prec,w_dtype", [("f32", "f32"), ("f32", "bf16"), ("bf16", "bf16"),
                                          ("bf16x3", "bf16")])
@pytest.mark.parametrize("M,N,K", [(32, 512, 512), (37, 100, 264), (130, 300, 1032), (1, 16, 8)])
def test_masked_linear_within_dot_bound(prec, w_dtype, M, N, K):
    gp, op = PREC[prec]
    X = WL.gen_x(M, K, seed=4)
    W = WL.gen_w(N, K, seed=5, dtype=w_dtype)
    eta = O.noise(M, K, O.MECH_GAUSSIAN, 4.0, 1.0, 1, 2)
    Xt = sp.mask(dev(X), dev(eta), gp)
    R = host(sp.masked_linear(Xt, gp, dev_w(W, w_dtype)))
    xt = O.mask(X, eta)
    A = O.gemm_operand(xt, op)
    err = np.abs(R.astype(np.float64) - O.gemm64(A, W))
    planes = {"bf16x3": 3, "bf16": 1}.get(prec)
    assert np.all(err <= O.dot_bound(A, W, planes=planes))
    # not vacuous: typical error at the float32 level
    assert np.median(err / np.maximum(O.dot_bound(A, W), 1e-30)) < 0.05


@pytest.mark.parametrize("prec", ["f32", "bf16x3"])
@pytest.mark.parametrize("mech", ["laplace", "gaussian"])
@pytest.mark.parametrize("M,N,K", [(32, 512, 512), (130, 200, 776), (5, 300, 2560), (64, 96, 4096)])
def test_correction_within_dot_bound(prec, mech, M, N, K):
    gp, op = PREC[prec]
    g, o = MECH[mech]
    W = WL.gen_w(N, K, seed=6)
    C = host(sp.correction(dev_w(W), M, g, 825.27, 2.0, 3, 77, 10, gp))
    eta = O.noise(M, K, o, 825.27, 2.0, 3, 77, 10)
    err = np.abs(C.astype(np.float64) - O.gemm64(eta, W))
    assert np.all(err <= O.dot_bound(eta, W, planes=3 if prec == "bf16x3" else None))


# --------------------------------------------------------------- fused, end to end

def _fused_case(M, N, K, mech, delta, eps, prec, w_dtype="bf16", seed=0, sid=5, row0=0,
                corr_prec="bf16x3"):
    gm, om = MECH[mech]
    gp, op = PREC[prec]
    cp = PREC["f32" if w_dtype == "f32" else corr_prec][0]
    X = WL.gen_x(M, K, seed=1)
    W = WL.gen_w(N, K, seed=2, dtype=w_dtype)
    Wd = dev_w(W, w_dtype)
    C = sp.correction(Wd, M, gm, delta, eps, seed, sid, row0, cp)
    Y = sp.masked_linear_fused(dev(X), Wd, C, gm, delta, eps, seed, sid, row0, gp)
    Yg = host(Y).astype(np.float64)
    eta = O.noise(M, K, om, delta, eps, seed, sid, row0)
    Xt = O.mask(X, eta)
    b = O.error_bounds(X, eta, Xt, W, op)
    err = np.abs(Yg - O.gemm64(X, W))
    return err, b, host(C), Y


@pytest.mark.parametrize("mech", ["laplace", "gaussian"])
def test_single_fp32_projection(mech):
    # 32 x 512 activations, 512 x 512 float32 weights, Delta = 1, eps = 1, seed 0
    err, b, _, _ = _fused_case(32, 512, 512, mech, 1.0, 1.0, "f32", w_dtype="f32")
    assert np.all(err <= b["gate"])
    assert np.mean(err) <= np.mean(b["logb"])


@pytest.mark.parametrize("prec", ["f32", "bf16", "bf16x3"])
@pytest.mark.parametrize("mech", ["laplace", "gaussian", "none"])
@pytest.mark.parametrize("M,N,K", [(37, 100, 264), (130, 300, 1032), (64, 96, 4096), (256, 640, 512)])
@pytest.mark.parametrize("delta,eps", [(1.0, 1.0), (825.27, 2.0)])
def test_fused_within_theorem4_gate(prec, mech, M, N, K, delta, eps):
    err, b, _, _ = _fused_case(M, N, K, mech, delta, eps, prec)
    assert np.all(err <= b["gate"]), "max err/gate %.3g" % np.max(err / b["gate"])
    if prec != "bf16":
        assert np.mean(err) <= np.mean(b["logb"])


@pytest.mark.parametrize("prec", ["bf16", "bf16x3"])
@pytest.mark.parametrize("M", [1, 4, 16])
@pytest.mark.parametrize("N,K", [(6144, 2560), (200, 9728), (40, 264), (72, 16400)])
def test_fused_skinny_decode(prec, M, N, K):
    err, b, _, _ = _fused_case(M, N, K, "gaussian", 719.8, 2.0, prec, row0=1000 + M)
    assert np.all(err <= b["gate"])


@pytest.mark.parametrize("prec", ["bf16", "bf16x3"])
@pytest.mark.parametrize("M", [1, 2, 3, 16])
@pytest.mark.parametrize("N,K,xpad", [(6144, 2560, 0), (200, 9728, 8), (40, 264, 0), (72, 16400, 0)])
def test_fused_precomputed_mask_is_the_two_launch_path(prec, M, N, K, xpad):
    # decode with a precomputed mask forms fl32(X + eta) inside the GEMM: bit for
    # bit the mask kernel followed by the GEMM, and the in-stream-noise fused call
    gp, op = PREC[prec]
    gm, om = MECH["gaussian"]
    sid, row0 = WL.stream_id(2, 1), 500 + M
    X = WL.gen_x(M, K, seed=31)
    W = WL.gen_w(N, K, seed=32)
    Wd = dev_w(W)
    Xd = torch.zeros((M, K + xpad), device=DEV)
    Xd[:, :K] = dev(X)
    Xd = Xd[:, :K]
    eta = sp.noise(M, K, gm, 719.8, 2.0, 0, sid, row0=row0)
    C = sp.correction(Wd, M, gm, 719.8, 2.0, 0, sid, row0, sp.SPLITEE_PREC_BF16X3)
    Y = host(sp.masked_linear_fused(Xd, Wd, C, gm, 719.8, 2.0, 0, sid, row0, gp, eta_override=eta))
    Y2 = host(sp.masked_linear_unmask(sp.mask(Xd, eta, gp), gp, Wd, C))
    Y3 = host(sp.masked_linear_fused(Xd, Wd, C, gm, 719.8, 2.0, 0, sid, row0, gp))
    assert np.array_equal(bits(Y), bits(Y2))
    assert np.array_equal(bits(Y), bits(Y3))
    eta_o = O.noise(M, K, om, 719.8, 2.0, 0, sid, row0)
    b = O.error_bounds(X, eta_o, O.mask(X, eta_o), W, op)
    assert np.all(np.abs(Y.astype(np.float64) - O.gemm64(X, W)) <= b["gate"])


@pytest.mark.parametrize("prec", ["f32", "bf16", "bf16x3"])
@pytest.mark.parametrize("M", [1, 16, 64, 130])
def test_exact_cancellation_integer_mask(prec, M):
    # integer X, eta, W with every partial sum below 2^24: Y == X W^T exactly
    gp, _ = PREC[prec]
    K, N = 256, 72
    X = WL.gen_int((M, K), -8, 8, 20)
    eta = WL.gen_int((M, K), -8, 8, 21)
    W = WL.gen_int((N, K), -4, 4, 22)
    Wd = dev_w(W)
    Cd = dev(O.gemm64(eta, W).astype(np.float32))  # exact integers
    Y = sp.masked_linear_fused(dev(X), Wd, Cd, sp.SPLITEE_MECH_NONE, 1.0, 1.0, 0, 0, 0, gp,
                               eta_override=dev(eta))
    assert np.array_equal(host(Y).astype(np.float64), O.gemm64(X, W))


@pytest.mark.parametrize("M,prec", [(4, "bf16x3"), (128, "bf16x3"), (128, "f32")])
def test_fused_deterministic(M, prec):
    gp, _ = PREC[prec]
    N, K = 2048, 3072
    X = dev(WL.gen_x(M, K))
    Wd = dev_w(WL.gen_w(N, K))
    C = sp.correction(Wd, M, sp.SPLITEE_MECH_LAPLACE, 1.0, 4.0, 0, 1, 0, sp.SPLITEE_PREC_BF16X3)
    ws = sp.workspace(M, N, K, gp)
    Y1 = sp.masked_linear_fused(X, Wd, C, sp.SPLITEE_MECH_LAPLACE, 1.0, 4.0, 0, 1, 0, gp, ws=ws).clone()
    Y2 = sp.masked_linear_fused(X, Wd, C, sp.SPLITEE_MECH_LAPLACE, 1.0, 4.0, 0, 1, 0, gp, ws=ws)
    assert torch.equal(Y1.view(torch.int32), Y2.view(torch.int32))


@pytest.mark.parametrize("M", [4, 64, 128])
def test_fused_unmask_is_exact_given_r_and_c(M):
    # Y == fl32(R - C) bit for bit, R from the same GEMM kernel without the epilogue
    N, K = 1280, 3072
    X = WL.gen_x(M, K)
    Wd = dev_w(WL.gen_w(N, K))
    gp = sp.SPLITEE_PREC_BF16X3
    mech = sp.SPLITEE_MECH_GAUSSIAN
    C = sp.correction(Wd, M, mech, 1.0, 1.0, 0, 3, 0, gp)
    Y = host(sp.masked_linear_fused(dev(X), Wd, C, mech, 1.0, 1.0, 0, 3, 0, gp))
    Xt = sp.noise_mask(dev(X), gp, mech, 1.0, 1.0, 0, 3, 0)
    R = host(sp.masked_linear_unmask(Xt, gp, Wd, None))
    assert np.array_equal(bits(Y), bits(O.unmask(R, host(C))))
    # and the two halves compose to the fused call exactly
    Y2 = host(sp.masked_linear_unmask(Xt, gp, Wd, C))
    assert np.array_equal(bits(Y), bits(Y2))


@pytest.mark.parametrize("prec", ["f32", "bf16", "bf16x3"])
@pytest.mark.parametrize("mech", ["laplace", "gaussian"])
def test_noise_mask_bit_exact(prec, mech):
    gp, op = PREC[prec]
    g, o = MECH[mech]
    M, K = 19, 1032
    X = WL.gen_x(M, K, seed=8)
    got = host(sp.noise_mask(dev(X), gp, g, 825.27, 0.5, 4, 300, 77))
    xt = O.mask(X, O.noise(M, K, o, 825.27, 0.5, 4, 300, 77))
    if prec == "f32":
        assert np.array_equal(bits(got[0]), bits(xt))
    elif prec == "bf16":
        assert np.array_equal(got[0].view(np.uint16), O.bf16_bits(O.bf16_rne(xt)))
    else:
        for p, ref in enumerate(O.split3(xt)):
            assert np.array_equal(got[p].view(np.uint16), O.bf16_bits(ref))


@pytest.mark.parametrize("prec,M,K", [(p, M, K) for p in ("f32", "bf16", "bf16x3") for M, K in ((130, 4104), (65537, 8))]
                         + [("f32", 70001, 4)])  # bfloat16 rows of 4 elements are not 16-byte aligned
def test_noise_mask_bit_exact_launch_shapes(prec, M, K):
    # the generated-noise mask at both lane mappings and past 65535 rows (see above)
    gp, op = PREC[prec]
    X = WL.gen_x(M, K, seed=13)
    got = host(sp.noise_mask(dev(X), gp, sp.SPLITEE_MECH_GAUSSIAN, 2.0, 1.0, 3, 41, 5))
    xt = O.mask(X, O.noise(M, K, O.MECH_GAUSSIAN, 2.0, 1.0, 3, 41, 5))
    if prec == "f32":
        assert np.array_equal(bits(got[0]), bits(xt))
    elif prec == "bf16":
        assert np.array_equal(got[0].view(np.uint16), O.bf16_bits(O.bf16_rne(xt)))
    else:
        for p, ref in enumerate(O.split3(xt)):
            assert np.array_equal(got[p].view(np.uint16), O.bf16_bits(ref))


@pytest.mark.parametrize("M,N,K,prec", [(128, 5120, 3072, "bf16x3"), (128, 3072, 8192, "bf16"),
                                        (1, 6144, 2560, "bf16x3"), (64, 2560, 4096, "f32")])
def test_split_k_reduction_matches_single_pass_bound_and_repeats(M, N, K, prec):
    # the split-K hand-off: repeated calls on one workspace give identical bits
    # and stay within the dot-product bound of the exact product
    gp, op = PREC[prec]
    X = WL.gen_x(M, K, seed=11)
    W = WL.gen_w(N, K, seed=12)
    Wd = dev_w(W)
    eta = O.noise(M, K, O.MECH_LAPLACE, 1.0, 1.0, 0, 1)
    Xt = sp.mask(dev(X), dev(eta), gp)
    ws = sp.workspace(M, N, K, gp, gemm_only=True)
    outs = [host(sp.masked_linear_unmask(Xt, gp, Wd, None, ws=ws)) for _ in range(3)]
    assert all(np.array_equal(bits(outs[0]), bits(o)) for o in outs[1:])
    A = O.gemm_operand(O.mask(X, eta), op)
    planes = {"bf16x3": 3, "bf16": 1}.get(prec)
    assert np.all(np.abs(outs[0].astype(np.float64) - O.gemm64(A, W)) <= O.dot_bound(A, W, planes=planes))


# ----------------------------------------------------- full-size sampled parity

def _sampled_full_size(model, M, prec, mech, delta, eps, nsample=256, nrows=16):
    gm, om = MECH[mech]
    gp, op = PREC[prec]
    g = np.random.Generator(np.random.PCG64(99))
    for proj in model.projections():
        K, N = proj.K, proj.N
        sid = WL.stream_id(0, proj.group)
        X = WL.gen_x(M, K, seed=1)
        W = WL.gen_w(N, K, seed=2)
        Wd = dev_w(W)
        C = sp.correction(Wd, M, gm, delta, eps, 0, sid, 0, sp.SPLITEE_PREC_BF16X3)
        Y = host(sp.masked_linear_fused(dev(X), Wd, C, gm, delta, eps, 0, sid, 0, gp))
        # the first and last row and column (the edge tiles) and random others
        rows = np.unique(np.concatenate([[0, M - 1], g.choice(M, size=min(M, nrows - 2), replace=False)]))
        cols = np.unique(np.concatenate([[0, N - 1], g.choice(N, size=nsample - 2, replace=False)]))
        for i in rows:
            eta = O.noise(1, K, om, delta, eps, 0, sid, int(i))
            xt = O.mask(X[i:i + 1], eta)
            Ws = W[cols]
            b = O.error_bounds(X[i:i + 1], eta, xt, Ws, op)
            err = np.abs(Y[i, cols].astype(np.float64) - O.gemm64(X[i:i + 1], Ws)[0])
            assert np.all(err <= b["gate"][0]), (proj.name, i)


@pytest.mark.parametrize("mech,eps", [("laplace", 1.0), ("gaussian", 4.0), ("laplace", 16.0)])
def test_llama_layer_m128_sampled(mech, eps):
    _sampled_full_size(WL.LLAMA_3B, 128, "bf16x3", mech, 1.0, eps)


def test_llama_layer_m512_sampled_paper_delta():
    _sampled_full_size(WL.LLAMA_3B, 512, "bf16x3", "gaussian", 825.27, 2.0)


@pytest.mark.parametrize("M", [1, 4, 16, 64])
def test_qwen_decode_bank_rows(M):
    # correction bank for 2048 positions; a decode step at t uses bank rows [t, t+M)
    proj = WL.QWEN3_4B.projections()[0]
    K, N = proj.K, proj.N
    sid = WL.stream_id(0, proj.group)
    W = WL.gen_w(N, K)
    Wd = dev_w(W)
    gm = sp.SPLITEE_MECH_GAUSSIAN
    bank = sp.correction(Wd, 2048, gm, 719.8, 2.0, 0, sid, 0, sp.SPLITEE_PREC_BF16X3)
    t = 2048 - M - 3
    X = WL.gen_x(M, K, seed=7)
    Y = host(sp.masked_linear_fused(dev(X), Wd, bank[t:t + M], gm, 719.8, 2.0, 0, sid, t,
                                    sp.SPLITEE_PREC_BF16X3))
    eta = O.noise(M, K, O.MECH_GAUSSIAN, 719.8, 2.0, 0, sid, t)
    b = O.error_bounds(X, eta, O.mask(X, eta), W, O.PREC_BF16X3)
    err = np.abs(Y.astype(np.float64) - O.gemm64(X, W))
    assert np.all(err <= b["gate"])


@pytest.mark.parametrize("M,prec", [(128, "bf16x3"), (4, "bf16x3"), (64, "f32")])
def test_graph_replay_matches_eager(M, prec):
    # noise + mask and GEMM + unmask captured in a HIP graph: every replay, with
    # eager work and synchronisations in between, equals the eager result
    gp, _ = PREC[prec]
    N, K = 3072, 3072
    X = dev(WL.gen_x(M, K))
    Wd = dev_w(WL.gen_w(N, K))
    mech = sp.SPLITEE_MECH_GAUSSIAN
    C = sp.correction(Wd, M, mech, 1.0, 1.0, 0, 9, 0, sp.SPLITEE_PREC_BF16X3)
    planes = 3 if gp == sp.SPLITEE_PREC_BF16X3 else 1
    Xt = torch.empty((planes, M, K), dtype=torch.float32 if gp == sp.SPLITEE_PREC_F32 else torch.int16,
                     device=DEV)
    Y = torch.empty((M, N), device=DEV)
    ws = sp.workspace(M, N, K, gp, gemm_only=True)

    def step():
        sp.splitee_noise_mask(X, K, Xt, gp, K, M, K, mech, 1.0, 1.0, 0, 9, 0)
        sp.splitee_masked_linear_unmask(Xt, gp, K, Wd, sp.SPLITEE_BF16, K, C, N, Y, N, M, N, K,
                                        ws[0], ws[1])

    step()
    ref = host(Y).copy()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for r in range(4):
        Y.fill_(float("nan"))
        g.replay()
        got = host(Y)
        assert np.array_equal(bits(got), bits(ref)), "replay %d" % r
        step()  # eager work between replays
        torch.cuda.synchronize()
