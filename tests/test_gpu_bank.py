"""GPU side of the noise bank: a bank created from the GPU corrections holds exactly
what splitee_correction writes for the same rows (bit for bit, block by block),
matches the oracle's eta W^T within the dot-product bound, and drives decode steps
end to end through the fused call (row0 from the bank, C rows from the bank), each
row once."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_15039_amd as sp
import workloads as WL

pytestmark = pytest.mark.gpu

DEV = "cuda"
G = sp.SPLITEE_MECH_GAUSSIAN


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


@pytest.mark.parametrize("w_dtype,prec", [("bf16", sp.SPLITEE_PREC_BF16X3), ("f32", sp.SPLITEE_PREC_F32)])
def test_bank_holds_the_corrections(tmp_path, w_dtype, prec):
    K, N, rows, row0, sid, delta, eps = 512, 640, 300, 1000, WL.stream_id(3, 2), 825.27, 2.0
    W = WL.gen_w(N, K, seed=8, dtype=w_dtype)
    Wd = torch.from_numpy(W).to(DEV)
    if w_dtype == "bf16":
        Wd = Wd.to(torch.bfloat16)
    path = str(tmp_path / "bank.spb")
    sp.bank_create(path, Wd, K, G, delta, eps, 0, sid, row0, rows, prec)
    b = sp.splitee_bank_open(path)
    info = sp.splitee_bank_info(b)
    assert (info["rows"], info["row0"], info["consumed"], info["prec"]) == (rows, row0, 0, prec)
    got = torch.full((rows, N + 4), float("nan"), device=DEV)
    firsts = []
    r = 0
    for m in (16, 240, 44):  # the second batch ends at the 256-row block boundary
        firsts.append(sp.splitee_bank_load(b, m, got[r:], N + 4, True))
        r += m
    assert firsts == [row0, row0 + 16, row0 + 256]
    with pytest.raises(sp.SpliteeError):
        sp.splitee_bank_load(b, 1, got, N + 4, True)
    sp.splitee_bank_close(b)
    got = host(got)
    assert np.all(np.isnan(got[:, N:]))
    got = got[:, :N]
    # block by block: what the correction call writes for the same rows
    ref0 = host(sp.correction(Wd, 256, G, delta, eps, 0, sid, row0, prec))
    ref1 = host(sp.correction(Wd, 44, G, delta, eps, 0, sid, row0 + 256, prec))
    assert np.array_equal(bits(got[:256]), bits(ref0))
    assert np.array_equal(bits(got[256:]), bits(ref1))
    # and the oracle's eta W^T within Higham's bound (3 products per k for the split)
    eta = O.noise(rows, K, O.MECH_GAUSSIAN, delta, eps, 0, sid, row0)
    exact = O.gemm64(eta, W)
    bound = O.dot_bound(eta, W, planes=3 if prec == sp.SPLITEE_PREC_BF16X3 else None)
    assert np.all(np.abs(got.astype(np.float64) - exact) <= bound)


def test_bank_drives_decode_steps_once_each(tmp_path):
    # Qwen3-4B QKV (2560 -> 6144): a 64-row bank from position 1024, decode steps of 1, 4 and
    # 16 tokens, each taking its C rows and row0 from the bank
    proj = WL.QWEN3_4B.projections()[0]
    K, N = proj.K, proj.N
    sid, delta, eps = WL.stream_id(5, proj.group), 2 * 2560 ** 0.75, 1.0
    W = WL.gen_w(N, K, seed=12)
    Wd = torch.from_numpy(W).to(DEV).to(torch.bfloat16)
    path = sp.splitee_bank_path(str(tmp_path), K, N, sid)
    sp.bank_create(path, Wd, K, G, delta, eps, 0, sid, 1024, 64)
    b = sp.splitee_bank_open(path)
    g = np.random.Generator(np.random.PCG64(3))
    cols = np.unique(np.concatenate([np.arange(4), np.arange(N - 4, N), g.choice(N, 40, replace=False)]))
    expect = 1024
    for step, M in enumerate((1, 4, 16, 1, 16)):
        C = torch.empty((M, N), device=DEV)
        row0 = sp.splitee_bank_load(b, M, C, N, True)
        assert row0 == expect
        expect += M
        X = WL.gen_x(M, K, seed=20 + step)
        Y = host(sp.masked_linear_fused(torch.from_numpy(X).to(DEV), Wd, C, G, delta, eps, 0, sid, row0))
        for i in range(M):
            e = O.noise(1, K, O.MECH_GAUSSIAN, delta, eps, 0, sid, row0 + i)
            bnd = O.error_bounds(X[i:i + 1], e, O.mask(X[i:i + 1], e), W[cols], O.PREC_BF16X3)
            err = np.abs(Y[i, cols].astype(np.float64) - O.gemm64(X[i:i + 1], W[cols])[0])
            assert np.all(err <= bnd["gate"][0]), (step, i)
    assert sp.splitee_bank_info(b)["consumed"] == 38
    sp.splitee_bank_close(b)
