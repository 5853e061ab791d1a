"""Exactness sweep of the masked linear layer over seeded random shapes.

Every plan of the path is reached: the decode GEMVs (1-2 rows), the skinny MFMA
kernel (up to 16 rows), the streamed GEMM with the in-kernel mask (17-128 rows on
tiled W) and the two-launch path above, split and unsplit K, both weight orders,
one and three bfloat16 planes.  The inputs are small integers (|x|, |eta| <= 8,
|w| <= 4, K <= 2048), so x + eta is exact in bfloat16 and every partial sum of
X~ W^T, eta W^T and their difference stays below 2^24: whatever the summation
order, the unmasked output must equal X W^T exactly.  The same shapes go through
the fused call with a precomputed mask and through mask + GEMM + unmask.
Shapes are drawn around the plans' row boundaries, with ragged N and K.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_15039_amd as sp
import workloads as WL

pytestmark = pytest.mark.gpu

DEV = "cuda"
PREC = {"bf16": sp.SPLITEE_PREC_BF16, "bf16x3": sp.SPLITEE_PREC_BF16X3}
ROWS = [1, 2, 3, 4, 7, 16, 17, 31, 64, 65, 100, 128, 129, 200, 257, 300, 513]


def _shapes(n, seed=20260):
    g = np.random.Generator(np.random.PCG64(seed))
    out = []
    while len(out) < n:
        M = int(ROWS[len(out) % len(ROWS)])
        N = int(g.integers(1, 1300))
        K = 8 * int(g.integers(1, 257))
        if M * N * K <= 3 * 10**8:
            out.append((M, N, K))
    return out


SHAPES = _shapes(24)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def test_sweep_shapes_cover_every_row_plan():
    ms = {m for m, _, _ in SHAPES}
    assert {1, 2}.issubset(ms) and ms & set(range(3, 17)) and ms & set(range(17, 129)) and max(ms) > 128
    assert all(k % 8 == 0 and k <= 2048 for _, _, k in SHAPES)
    assert any(n % 32 for _, n, _ in SHAPES) and any(k % 64 for _, _, k in SHAPES)


@pytest.mark.parametrize("layout", ["row", "tiled"])
@pytest.mark.parametrize("prec", ["bf16", "bf16x3"])
@pytest.mark.parametrize("case", range(len(SHAPES)))
def test_shape_sweep_exact(layout, prec, case):
    M, N, K = SHAPES[case]
    print("case %d: M=%d N=%d K=%d %s %s" % (case, M, N, K, layout, prec), flush=True)
    gp = PREC[prec]
    X = WL.gen_int((M, K), -8, 8, 1000 + case)
    eta = WL.gen_int((M, K), -8, 8, 2000 + case)
    W = WL.gen_int((N, K), -4, 4, 3000 + case)
    Wd = dev(W).to(torch.bfloat16)
    Wp = sp.tile_weights(Wd) if layout == "tiled" else Wd
    # C and Y rows 16-byte aligned: a pitch of N rounded up to 4 floats
    ld = -(-N // 4) * 4
    C = torch.zeros((M, ld), dtype=torch.float32, device=DEV)[:, :N]
    C.copy_(dev(O.gemm64(eta, W).astype(np.float32)))
    want = O.gemm64(X, W)
    Y = torch.full((M, ld), float("nan"), device=DEV)[:, :N]
    sp.masked_linear_fused(dev(X), Wp, C, sp.SPLITEE_MECH_NONE, 1.0, 1.0, 0, 0, 0, gp, eta_override=dev(eta), Y=Y)
    assert np.array_equal(host(Y).astype(np.float64), want)
    Xt = sp.mask(dev(X), dev(eta), gp)
    Y2 = torch.full((M, ld), float("nan"), device=DEV)[:, :N]
    sp.masked_linear_unmask(Xt, gp, Wp, C, Y=Y2)
    assert np.array_equal(host(Y2).astype(np.float64), want)
