"""The no-allocation variant of the fused call (splitee_masked_linear_fused_noalloc):
through the C ABI, on two calls in a row with the second one smaller, its output is
bit-identical to splitee_masked_linear_fused's with a caller-owned workspace (the same
kernels run on the library's static scratch buffer), for the prefill path (noise + mask
+ GEMM + unmask, split over K), the decode path with a precomputed mask, and both
weight layouts; a shape that needs more scratch than the buffer holds is refused."""
import numpy as np
import pytest
import torch

import paper_2609_15039_amd as sp
import workloads as WL

pytestmark = pytest.mark.gpu

G = sp.SPLITEE_MECH_GAUSSIAN
P3 = sp.SPLITEE_PREC_BF16X3


def _inputs(M, N, K, tiled, seed):
    X = torch.from_numpy(WL.gen_x(M, K, seed=seed)).cuda()
    W = torch.from_numpy(WL.gen_w(N, K, seed=seed + 1)).cuda().to(torch.bfloat16)
    if tiled:
        W = sp.tile_weights(W)
    return X, W


def _both(X, W, C, M, N, K, prec, sid, row0, eta=None):
    wt = sp._wtype(W)
    Y_ref = sp.masked_linear_fused(X, W, C, G, 825.27, 2.0, 0, sid, row0, prec, eta_override=eta)
    Y = torch.full((M, N), float("nan"), device="cuda")
    sp.splitee_masked_linear_fused_noalloc(X, X.stride(0), W, wt, W.stride(0), C, C.stride(0), Y, N, M, N, K, G,
                                           825.27, 2.0, 0, sid, row0, eta, prec)
    torch.cuda.synchronize()
    return Y_ref.cpu().numpy().view(np.uint32), Y.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("tiled", [False, True])
@pytest.mark.parametrize("prec", [P3, sp.SPLITEE_PREC_BF16, sp.SPLITEE_PREC_F32])
def test_noalloc_prefill_matches_workspace_call_twice(tiled, prec):
    if tiled and prec == sp.SPLITEE_PREC_F32:
        pytest.skip("tiled weights need a bfloat16 precision mode")
    # first a split-K shape (counters and partials in the scratch), then a smaller one
    for (M, N, K), seed in (((130, 3072, 3072), 3), ((37, 300, 264), 5)):
        X, W = _inputs(M, N, K, tiled, seed)
        sid = WL.stream_id(seed, 2)
        C = sp.correction(W, M, G, 825.27, 2.0, 0, sid, 7, P3 if prec != sp.SPLITEE_PREC_F32 else prec)
        ref, got = _both(X, W, C, M, N, K, prec, sid, 7)
        assert np.array_equal(ref, got), (M, N, K)


@pytest.mark.parametrize("tiled", [False, True])
def test_noalloc_decode_with_precomputed_mask_twice(tiled):
    for (M, N, K), seed in (((4, 6144, 2560), 11), ((1, 2560, 9728), 13)):
        X, W = _inputs(M, N, K, tiled, seed)
        sid = WL.stream_id(seed, 1)
        row0 = 1024
        eta = sp.noise(M, K, G, 825.27, 2.0, 0, sid, row0)
        C = sp.correction(W, M, G, 825.27, 2.0, 0, sid, row0, P3)
        ref, got = _both(X, W, C, M, N, K, P3, sid, row0, eta)
        assert np.array_equal(ref, got), (M, N, K)


def test_noalloc_refuses_shapes_beyond_its_scratch():
    M, N, K = 4096, 2560, 9728  # masked-input planes alone: 4096 x 9728 x 6 bytes = 239 MB
    assert sp.splitee_fused_workspace_bytes(M, N, K, P3) > sp.SPLITEE_NOALLOC_SCRATCH_BYTES
    lib = sp.load()
    rc = lib.splitee_masked_linear_fused_noalloc(16, K, 16, sp.SPLITEE_BF16, K, 16, N, 16, N, M, N, K, G, 1.0, 1.0, 0,
                                                 0, 0, None, P3, None)
    assert rc == sp.SPLITEE_ERR_SCRATCH
    assert b"static device buffer" in lib.splitee_status_string(rc)
