"""GPU parity of the tiled weight order (splitee_tile_weights, SPLITEE_BF16_TILED).

The tiling is a copy: bit-exact against the element index the header defines.
Every GEMM entry point that takes tiled W is held to the same bar as with
row-major W: the dot-product bound for R and the correction, the Theorem-4 gate
for the unmasked output, exact equality on small-integer inputs, bit-identical
repeats of the split-K path and bit-identity of the in-kernel decode mask with
the two-launch path.  Shapes span several tiles with ragged tails in M, N and K,
and every plan of the tiled path (decode kernel for M <= 16, 64-, 128- and
256-column streamed tiles, split and unsplit K).
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_15039_amd as sp
import workloads as WL

pytestmark = pytest.mark.gpu

DEV = "cuda"
PREC = {"bf16": (sp.SPLITEE_PREC_BF16, O.PREC_BF16), "bf16x3": (sp.SPLITEE_PREC_BF16X3, O.PREC_BF16X3)}


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def tiled_reference(Wbits, N, K):
    """The tiled buffer of the header's definition, built element by element from
    the index formula (uint16 bfloat16 bits in, uint16 out)."""
    N32, KT = -(-N // 32), -(-K // 64)
    out = np.zeros(N32 * KT * 2048, dtype=np.uint16)
    n = np.arange(N)[:, None]
    k = np.arange(K)[None, :]
    idx = ((((n // 32) * KT + k // 64) * 4 + (k % 64) // 16) * 64 + ((k % 16) // 8) * 32 + n % 32) * 8 + k % 8
    out[idx] = Wbits
    return out


@pytest.mark.parametrize("N,K,ldw", [(1, 8, 8), (32, 64, 64), (37, 264, 272), (200, 1032, 1032), (5120, 3072, 3072)])
def test_tile_weights_is_the_defined_permutation(N, K, ldw):
    W = WL.gen_w(N, K, seed=3)
    Wd = torch.zeros((N, ldw), dtype=torch.bfloat16, device=DEV)
    Wd[:, :K] = dev(W).to(torch.bfloat16)
    Wd[:, K:] = 7.0  # padding columns of W must not reach the tiled buffer
    T = sp.tile_weights(Wd[:, :K])
    got = host(T.data.view(torch.int16)).view(np.uint16)
    ref = tiled_reference(host(Wd[:, :K].contiguous().view(torch.int16)).view(np.uint16), N, K)
    assert got.size == sp.splitee_tiled_weights_bytes(N, K) // 2
    assert np.array_equal(got, ref)


def _tiled_case(M, N, K, prec, mech=sp.SPLITEE_MECH_GAUSSIAN, omech=O.MECH_GAUSSIAN, delta=1.0, eps=1.0,
                sid=5, row0=0):
    gp, op = PREC[prec]
    X = WL.gen_x(M, K, seed=1)
    W = WL.gen_w(N, K, seed=2)
    T = sp.tile_weights(dev(W).to(torch.bfloat16))
    C = sp.correction(T, M, mech, delta, eps, 0, sid, row0, sp.SPLITEE_PREC_BF16X3)
    Y = host(sp.masked_linear_fused(dev(X), T, C, mech, delta, eps, 0, sid, row0, gp)).astype(np.float64)
    eta = O.noise(M, K, omech, delta, eps, 0, sid, row0)
    b = O.error_bounds(X, eta, O.mask(X, eta), W, op)
    Cref = O.gemm64(eta, W)
    return np.abs(Y - O.gemm64(X, W)), b, np.abs(host(C).astype(np.float64) - Cref), O.dot_bound(eta, W, planes=3)


@pytest.mark.parametrize("prec", ["bf16", "bf16x3"])
@pytest.mark.parametrize("M", [1, 2, 3, 16, 17, 64, 65, 130, 257])
@pytest.mark.parametrize("N,K", [(300, 1032), (96, 4096), (200, 264)])
def test_tiled_fused_within_theorem4_gate(prec, M, N, K):
    err, b, cerr, cbound = _tiled_case(M, N, K, prec, delta=825.27, eps=2.0, row0=M)
    assert np.all(cerr <= cbound), "correction outside the dot-product bound"
    assert np.all(err <= b["gate"]), "max err/gate %.3g" % np.max(err / b["gate"])
    if prec == "bf16x3":
        assert np.mean(err) <= np.mean(b["logb"])


@pytest.mark.parametrize("prec", ["bf16", "bf16x3"])
def test_tiled_half_height_tiles_above_128_rows(prec):
    # more than 256 tiles of 128 x 256 whose 64-row halves end in a fuller last round:
    # 64 x 256 tiles on 4-wave workgroups, ragged in M (300 = 4 x 64 + 44), N (22052 =
    # 86 x 256 + 36; row pitches are whole 16-byte units) and K (200 = 3 x 64 + 8)
    err, b, cerr, cbound = _tiled_case(300, 22052, 200, prec, delta=825.27, eps=2.0, row0=7)
    assert np.all(cerr <= cbound), "correction outside the dot-product bound"
    assert np.all(err <= b["gate"]), "max err/gate %.3g" % np.max(err / b["gate"])
    # the same plan on small integers: every element exact, so a misplaced tile shows
    gp, _ = PREC[prec]
    M, N, K = 300, 22052, 200
    X = WL.gen_int((M, K), -8, 8, 40)
    eta = WL.gen_int((M, K), -8, 8, 41)
    W = WL.gen_int((N, K), -4, 4, 42)
    T = sp.tile_weights(dev(W).to(torch.bfloat16))
    Cd = dev(O.gemm64(eta, W).astype(np.float32))
    Y = sp.masked_linear_fused(dev(X), T, Cd, sp.SPLITEE_MECH_NONE, 1.0, 1.0, 0, 0, 0, gp, eta_override=dev(eta))
    assert np.array_equal(host(Y).astype(np.float64), O.gemm64(X, W))


@pytest.mark.parametrize("prec", ["bf16", "bf16x3"])
@pytest.mark.parametrize("M,N,K", [(37, 100, 264), (130, 300, 1032), (1, 16, 8), (300, 520, 200)])
def test_tiled_masked_linear_within_dot_bound(prec, M, N, K):
    gp, op = PREC[prec]
    X = WL.gen_x(M, K, seed=4)
    W = WL.gen_w(N, K, seed=5)
    eta = O.noise(M, K, O.MECH_GAUSSIAN, 4.0, 1.0, 1, 2)
    Xt = sp.mask(dev(X), dev(eta), gp)
    R = host(sp.masked_linear(Xt, gp, sp.tile_weights(dev(W).to(torch.bfloat16))))
    A = O.gemm_operand(O.mask(X, eta), op)
    err = np.abs(R.astype(np.float64) - O.gemm64(A, W))
    assert np.all(err <= O.dot_bound(A, W, planes=3 if prec == "bf16x3" else 1))


@pytest.mark.parametrize("prec", ["bf16", "bf16x3"])
@pytest.mark.parametrize("M", [1, 2, 16, 64, 130])
def test_tiled_exact_cancellation_integer_mask(prec, M):
    # integer X, eta, W with every partial sum below 2^24: Y == X W^T exactly
    gp, _ = PREC[prec]
    K, N = 256, 72
    X = WL.gen_int((M, K), -8, 8, 20)
    eta = WL.gen_int((M, K), -8, 8, 21)
    W = WL.gen_int((N, K), -4, 4, 22)
    T = sp.tile_weights(dev(W).to(torch.bfloat16))
    Cd = dev(O.gemm64(eta, W).astype(np.float32))
    Y = sp.masked_linear_fused(dev(X), T, Cd, sp.SPLITEE_MECH_NONE, 1.0, 1.0, 0, 0, 0, gp, eta_override=dev(eta))
    assert np.array_equal(host(Y).astype(np.float64), O.gemm64(X, W))


@pytest.mark.parametrize("prec", ["bf16", "bf16x3"])
@pytest.mark.parametrize("M", [1, 2, 3, 16, 17, 64, 100, 128])
@pytest.mark.parametrize("N,K", [(6144, 2560), (200, 9728), (40, 264)])
def test_tiled_precomputed_mask_is_the_two_launch_path(prec, M, N, K):
    # the decode kernels (M <= 16) and the streamed kernel with 64-row tiles (M <= 128)
    # form fl32(X + eta) themselves: bit for bit the mask kernel followed by the GEMM, on
    # tiled W
    gp, op = PREC[prec]
    gm = sp.SPLITEE_MECH_GAUSSIAN
    sid, row0 = WL.stream_id(2, 1), 500 + M
    X = WL.gen_x(M, K, seed=31)
    W = WL.gen_w(N, K, seed=32)
    T = sp.tile_weights(dev(W).to(torch.bfloat16))
    Xd = dev(X)
    eta = sp.noise(M, K, gm, 719.8, 2.0, 0, sid, row0=row0)
    C = sp.correction(T, M, gm, 719.8, 2.0, 0, sid, row0, sp.SPLITEE_PREC_BF16X3)
    Y = host(sp.masked_linear_fused(Xd, T, C, gm, 719.8, 2.0, 0, sid, row0, gp, eta_override=eta))
    Y2 = host(sp.masked_linear_unmask(sp.mask(Xd, eta, gp), gp, T, C))
    assert np.array_equal(bits(Y), bits(Y2))
    eta_o = O.noise(M, K, O.MECH_GAUSSIAN, 719.8, 2.0, 0, sid, row0)
    b = O.error_bounds(X, eta_o, O.mask(X, eta_o), W, op)
    assert np.all(np.abs(Y.astype(np.float64) - O.gemm64(X, W)) <= b["gate"])


@pytest.mark.parametrize("prec", ["bf16", "bf16x3"])
@pytest.mark.parametrize("M", [64, 128])
def test_tiled_precomputed_mask_wide_n_is_the_two_launch_path(prec, M):
    # the 64 x 256 tiles of the in-kernel mask (gate/up widths), split over K
    gp, _ = PREC[prec]
    gm = sp.SPLITEE_MECH_GAUSSIAN
    N, K = 19456, 2560
    sid, row0 = WL.stream_id(4, 2), 300
    X = WL.gen_x(M, K, seed=33)
    T = sp.tile_weights(dev(WL.gen_w(N, K, seed=34)).to(torch.bfloat16))
    Xd = dev(X)
    eta = sp.noise(M, K, gm, 719.8, 2.0, 0, sid, row0=row0)
    C = sp.correction(T, M, gm, 719.8, 2.0, 0, sid, row0, sp.SPLITEE_PREC_BF16X3)
    Y = host(sp.masked_linear_fused(Xd, T, C, gm, 719.8, 2.0, 0, sid, row0, gp, eta_override=eta))
    Y2 = host(sp.masked_linear_unmask(sp.mask(Xd, eta, gp), gp, T, C))
    assert np.array_equal(bits(Y), bits(Y2))


@pytest.mark.parametrize("M,N,K,prec", [(128, 16384, 3072, "bf16x3"), (128, 5120, 3072, "bf16x3"),
                                        (512, 3072, 8192, "bf16"), (4, 6144, 2560, "bf16x3"),
                                        (64, 2560, 9728, "bf16x3")])
def test_tiled_split_k_repeats_and_matches_row_major_bound(M, N, K, prec):
    # repeated calls on one workspace give identical bits; both layouts stay
    # within the dot-product bound of the exact product
    gp, op = PREC[prec]
    X = WL.gen_x(M, K, seed=11)
    W = WL.gen_w(N, K, seed=12)
    Wd = dev(W).to(torch.bfloat16)
    T = sp.tile_weights(Wd)
    eta = O.noise(M, K, O.MECH_LAPLACE, 1.0, 1.0, 0, 1)
    Xt = sp.mask(dev(X), dev(eta), gp)
    ws = sp.workspace(M, N, K, gp, gemm_only=True)
    outs = [host(sp.masked_linear_unmask(Xt, gp, T, None, ws=ws)) for _ in range(3)]
    assert all(np.array_equal(bits(outs[0]), bits(o)) for o in outs[1:])
    rowmajor = host(sp.masked_linear_unmask(Xt, gp, Wd, None, ws=ws))
    A = O.gemm_operand(O.mask(X, eta), op)
    ref = O.gemm64(A, W)
    bound = O.dot_bound(A, W, planes=3 if prec == "bf16x3" else 1)
    assert np.all(np.abs(outs[0].astype(np.float64) - ref) <= bound)
    assert np.all(np.abs(rowmajor.astype(np.float64) - ref) <= bound)


def _sampled_full_size_tiled(model, M, prec, mech, omech, delta, eps, nsample=256, nrows=16):
    # the launch configuration of the bench: full projection shapes, tiled W,
    # outputs checked on sampled rows and columns
    gp, op = PREC[prec]
    g = np.random.Generator(np.random.PCG64(98))
    for proj in model.projections():
        K, N = proj.K, proj.N
        sid = WL.stream_id(0, proj.group)
        X = WL.gen_x(M, K, seed=1)
        W = WL.gen_w(N, K, seed=2)
        T = sp.tile_weights(dev(W).to(torch.bfloat16))
        C = sp.correction(T, M, mech, delta, eps, 0, sid, 0, sp.SPLITEE_PREC_BF16X3)
        Y = host(sp.masked_linear_fused(dev(X), T, C, mech, delta, eps, 0, sid, 0, gp))
        # the first and last row and column (the edge tiles) and random others
        rows = np.unique(np.concatenate([[0, M - 1], g.choice(M, size=min(M, nrows - 2), replace=False)]))
        cols = np.unique(np.concatenate([[0, N - 1], g.choice(N, size=nsample - 2, replace=False)]))
        for i in rows:
            eta = O.noise(1, K, omech, delta, eps, 0, sid, int(i))
            Ws = W[cols]
            b = O.error_bounds(X[i:i + 1], eta, O.mask(X[i:i + 1], eta), Ws, op)
            err = np.abs(Y[i, cols].astype(np.float64) - O.gemm64(X[i:i + 1], Ws)[0])
            assert np.all(err <= b["gate"][0]), (proj.name, i)


@pytest.mark.parametrize("M", [128, 512])
def test_tiled_llama_layer_sampled(M):
    _sampled_full_size_tiled(WL.LLAMA_3B, M, "bf16x3", sp.SPLITEE_MECH_GAUSSIAN, O.MECH_GAUSSIAN, 1.0, 1.0)


@pytest.mark.parametrize("M", [1, 4, 16, 64, 1024])
def test_tiled_qwen_layer_sampled(M):
    _sampled_full_size_tiled(WL.QWEN3_4B, M, "bf16x3", sp.SPLITEE_MECH_LAPLACE, O.MECH_LAPLACE, 719.8, 2.0)


def test_tiled_qwen_headline_configuration_sampled():
    # the bench's default launch configuration: 1024 tokens, Gaussian noise, Delta = eps = 1
    _sampled_full_size_tiled(WL.QWEN3_4B, 1024, "bf16x3", sp.SPLITEE_MECH_GAUSSIAN, O.MECH_GAUSSIAN, 1.0, 1.0)


@pytest.mark.parametrize("model,M,layout", [("qwen", 1024, "tiled"), ("llama", 512, "tiled"), ("llama", 128, "tiled"),
                                            ("qwen", 64, "tiled"), ("qwen", 16, "tiled"), ("qwen", 4, "tiled"),
                                            ("qwen", 2, "tiled"), ("qwen", 2, "row"), ("qwen", 1, "tiled"),
                                            ("qwen", 1, "row")])
@pytest.mark.parametrize("mech,omech,delta,eps", [(sp.SPLITEE_MECH_GAUSSIAN, O.MECH_GAUSSIAN, 1.0, 1.0),
                                                   (sp.SPLITEE_MECH_LAPLACE, O.MECH_LAPLACE, 719.8, 2.0)])
def test_tiled_full_size_every_element(model, M, layout, mech, omech, delta, eps):
    # the bench's workloads at full size in its launch configuration (one layer of the model,
    # bf16x3; tiled W, and at one and two tokens also the row-major W of the decode GEMV):
    # every output element of every projection against its Theorem-4 gate
    gp, op = PREC["bf16x3"]
    shape = WL.QWEN3_4B if model == "qwen" else WL.LLAMA_3B
    for proj in shape.projections():
        K, N = proj.K, proj.N
        sid = WL.stream_id(0, proj.group)
        X = WL.gen_x(M, K, seed=1)
        W = WL.gen_w(N, K, seed=2)
        T = sp.tile_weights(dev(W).to(torch.bfloat16)) if layout == "tiled" else dev(W).to(torch.bfloat16)
        C = sp.correction(T, M, mech, delta, eps, 0, sid, 0, sp.SPLITEE_PREC_BF16X3)
        Y = host(sp.masked_linear_fused(dev(X), T, C, mech, delta, eps, 0, sid, 0, gp)).astype(np.float64)
        del T, C
        eta = O.noise(M, K, omech, delta, eps, 0, sid, 0)
        gate = O.error_bounds(X, eta, O.mask(X, eta), W, op)["gate"]
        err = np.abs(Y - O.gemm64(X, W))
        bad = int((err > gate).sum())
        assert bad == 0, "%s: %d of %d elements above the gate (max err/gate %.3g)" % (
            proj.name, bad, err.size, float((err / gate).max()))


@pytest.mark.parametrize("prec,layout", [("bf16", "tiled"), ("f32", "row")])
@pytest.mark.parametrize("M", [1024, 64])
def test_full_size_every_element_other_modes(prec, layout, M):
    # the bench's other precision modes at the headline shapes (one Qwen3-4B layer): single-pass
    # bfloat16 on tiled W, and the binary32 MFMA path on row-major bfloat16 W; every element
    gp, op = {"bf16": (sp.SPLITEE_PREC_BF16, O.PREC_BF16), "f32": (sp.SPLITEE_PREC_F32, O.PREC_F32)}[prec]
    for proj in WL.QWEN3_4B.projections():
        K, N = proj.K, proj.N
        sid = WL.stream_id(0, proj.group)
        X = WL.gen_x(M, K, seed=1)
        W = WL.gen_w(N, K, seed=2)
        Wd = dev(W).to(torch.bfloat16)
        T = sp.tile_weights(Wd) if layout == "tiled" else Wd
        cprec = sp.SPLITEE_PREC_F32 if prec == "f32" else sp.SPLITEE_PREC_BF16X3
        C = sp.correction(T, M, sp.SPLITEE_MECH_GAUSSIAN, 1.0, 1.0, 0, sid, 0, cprec)
        Y = host(sp.masked_linear_fused(dev(X), T, C, sp.SPLITEE_MECH_GAUSSIAN, 1.0, 1.0, 0, sid, 0, gp))
        del T, C, Wd
        eta = O.noise(M, K, O.MECH_GAUSSIAN, 1.0, 1.0, 0, sid, 0)
        gate = O.error_bounds(X, eta, O.mask(X, eta), W, op)["gate"]
        err = np.abs(Y.astype(np.float64) - O.gemm64(X, W))
        bad = int((err > gate).sum())
        assert bad == 0, "%s %s: %d of %d elements above the gate (max err/gate %.3g)" % (
            prec, proj.name, bad, err.size, float((err / gate).max()))


@pytest.mark.parametrize("M", [128, 4, 64])
def test_tiled_graph_replay_matches_eager(M):
    # noise + mask and GEMM + unmask on tiled W captured in a HIP graph: every replay,
    # with eager work and synchronisations in between, equals the eager result
    gp = sp.SPLITEE_PREC_BF16X3
    N, K = 3072, 3072
    X = dev(WL.gen_x(M, K))
    T = sp.tile_weights(dev(WL.gen_w(N, K)).to(torch.bfloat16))
    mech = sp.SPLITEE_MECH_GAUSSIAN
    C = sp.correction(T, M, mech, 1.0, 1.0, 0, 9, 0, sp.SPLITEE_PREC_BF16X3)
    Xt = torch.empty((3, M, K), dtype=torch.int16, device=DEV)
    Y = torch.empty((M, N), device=DEV)
    ws = sp.workspace(M, N, K, gp, gemm_only=True)

    def step():
        sp.splitee_noise_mask(X, K, Xt, gp, K, M, K, mech, 1.0, 1.0, 0, 9, 0)
        sp.splitee_masked_linear_unmask(Xt, gp, K, T, sp.SPLITEE_BF16_TILED, K, C, N, Y, N, M, N, K, ws[0], ws[1])

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
        step()
        torch.cuda.synchronize()
