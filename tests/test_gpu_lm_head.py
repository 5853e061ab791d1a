"""GPU parity of the vocabulary (LM-head) projection: the same entry points at the
widest N of the two models (Llama-3.2-3B 3072 -> 128256, Qwen3-4B 2560 -> 151936),
against the oracle on sampled output columns (the first and last columns of the row,
which cover the ragged tile at the end, and a random sample).  Bar as for the other
projections: the Theorem-4 gate per element (see test_gpu_parity.py).  Both weight
layouts: row-major and the tiled order (the launch configuration of the bench)."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_15039_amd as sp
import workloads as WL

pytestmark = pytest.mark.gpu

DEV = "cuda"
GAUSS = (sp.SPLITEE_MECH_GAUSSIAN, O.MECH_GAUSSIAN)
PREC = {"bf16x3": (sp.SPLITEE_PREC_BF16X3, O.PREC_BF16X3), "bf16": (sp.SPLITEE_PREC_BF16, O.PREC_BF16)}
# Theorem 1 with alpha = 1 (the input of the LM head is the final normalisation's output)
DELTA_LN = {"llama-3.2-3b": 2 * 3072 ** 0.75, "qwen3-4b": 2 * 2560 ** 0.75}


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


@pytest.fixture(scope="module", params=[("llama-3.2-3b", "row-major"), ("llama-3.2-3b", "tiled"),
                                        ("qwen3-4b", "row-major"), ("qwen3-4b", "tiled")])
def lm_head(request):
    name, layout = request.param
    model = WL.LLAMA_3B if name == "llama-3.2-3b" else WL.QWEN3_4B
    proj = model.lm_head()
    W = WL.gen_w(proj.N, proj.K, seed=5)
    Wd = torch.from_numpy(W).to(DEV).to(torch.bfloat16)
    if layout == "tiled":
        Wd = sp.tile_weights(Wd)
    yield model, proj, W, Wd
    del Wd
    torch.cuda.empty_cache()


def sample_cols(N, seed, n=48):
    g = np.random.Generator(np.random.PCG64(seed))
    return np.unique(np.concatenate([np.arange(8), np.arange(N - 8, N), g.choice(N, n, replace=False)]))


def check_rows(X, Y, W, K, sid, row0, delta, eps, op, rows, cols):
    Ws = W[cols]
    for i in rows:
        eta = O.noise(1, K, O.MECH_GAUSSIAN, delta, eps, 0, sid, row0 + int(i))
        xt = O.mask(X[i:i + 1], eta)
        b = O.error_bounds(X[i:i + 1], eta, xt, Ws, op)
        err = np.abs(Y[i, cols].astype(np.float64) - O.gemm64(X[i:i + 1], Ws)[0])
        assert np.all(err <= b["gate"][0]), (int(i), float(np.max(err / b["gate"][0])))


@pytest.mark.parametrize("M,prec", [(1, "bf16x3"), (15, "bf16x3"), (15, "bf16"), (128, "bf16x3")])
def test_lm_head_fused_sampled(lm_head, M, prec):
    model, proj, W, Wd = lm_head
    K, N = proj.K, proj.N
    gp, op = PREC[prec]
    delta, eps = DELTA_LN[model.name], 1.0
    sid = WL.stream_id(model.layers, proj.group)
    X = WL.gen_x(M, K, seed=3)
    C = sp.correction(Wd, M, GAUSS[0], delta, eps, 0, sid, 0, sp.SPLITEE_PREC_BF16X3)
    Y = host(sp.masked_linear_fused(torch.from_numpy(X).to(DEV), Wd, C, GAUSS[0], delta, eps, 0, sid, 0, gp))
    rows = sorted(set([0, M - 1] + list(np.random.Generator(np.random.PCG64(M)).choice(M, min(M, 4), replace=False))))
    check_rows(X, Y, W, K, sid, 0, delta, eps, op, rows, sample_cols(N, M))


@pytest.mark.parametrize("M", [1, 2, 15])
def test_lm_head_decode_with_bank_and_precomputed_mask(lm_head, M):
    # decode at position t: correction rows [t, t + M) of a 2048-position bank, the mask
    # drawn beforehand (as for a whole decode step) and handed to the fused call
    model, proj, W, Wd = lm_head
    K, N = proj.K, proj.N
    delta, eps = DELTA_LN[model.name], 2.0
    sid = WL.stream_id(model.layers, proj.group)
    t = 1024
    bank = torch.zeros((2048, N), dtype=torch.float32, device=DEV)
    bank[t:t + M] = sp.correction(Wd, M, GAUSS[0], delta, eps, 0, sid, t, sp.SPLITEE_PREC_BF16X3)
    eta = sp.noise(M, K, GAUSS[0], delta, eps, 0, sid, t)
    X = WL.gen_x(M, K, seed=11)
    Xd = torch.from_numpy(X).to(DEV)
    Y = host(sp.masked_linear_fused(Xd, Wd, bank[t:t + M], GAUSS[0], delta, eps, 0, sid, t,
                                    sp.SPLITEE_PREC_BF16X3, eta_override=eta))
    Y2 = host(sp.masked_linear_fused(Xd, Wd, bank[t:t + M], GAUSS[0], delta, eps, 0, sid, t,
                                     sp.SPLITEE_PREC_BF16X3))
    assert np.array_equal(Y, Y2)  # precomputed mask == mask drawn in-stream
    check_rows(X, Y, W, K, sid, t, delta, eps, O.PREC_BF16X3, range(M), sample_cols(N, 100 + M))
