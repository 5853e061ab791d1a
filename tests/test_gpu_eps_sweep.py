"""The floating-point error of the GPU path as a function of eps (the analogue of the
paper's Table 4), and full-size parity over the eps x mechanism grid of the 28-layer
Llama-3.2-3B stack at 512 tokens and the 36-layer Qwen3-4B stack at 1024 tokens.

Table 4 reports, per eps, the mean error of the masked linear operator, the mean of
Eq. fp-log-bound, their ratio and the share of elements above the bound, and shows
the error scaling as 1/eps (noise-dominated regime).  Here the same statistics are
taken on the fused bf16x3 path against the oracle, on synthetic inputs (the paper
measured real activations, so its absolute values are context only), and checked:
every element within the Theorem-4 gate, mean error below mean Eq. fp-log-bound, and
mean |error| * eps constant across the sweep to within [0.75, 1.33].

Noise scales follow Theorems 1-3 for alpha = 1, beta = 0 and N(0, 0.02^2) weights,
whose spectral norms are close to 0.02 (sqrt(rows) + sqrt(cols)):
  QKV and gate/up: Delta_LN = 2 d^(3/4)            (Theorem 1)
  O:               Delta_LN * ||W_v||_2             (Theorem 2)
  Down:            2 d^2 ||W_up||_2 ||W_gate||_2    (Theorem 3; far beyond binary32
                   cancellation, as the paper says: the gate then only bounds an
                   output that has lost X)
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_15039_amd as sp
import workloads as WL

pytestmark = pytest.mark.gpu

MECH = {"laplace": (sp.SPLITEE_MECH_LAPLACE, O.MECH_LAPLACE),
        "gaussian": (sp.SPLITEE_MECH_GAUSSIAN, O.MECH_GAUSSIAN)}
EPS = (0.5, 2.0, 8.0)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def spec_norm_estimate(rows, cols, std=0.02):
    return std * (math.sqrt(rows) + math.sqrt(cols))


def paper_delta(model, proj):
    d = model.hidden
    ln = 2.0 * d ** 0.75
    if proj.name == "o":
        return ln * spec_norm_estimate(model.kv_dim, d)
    if proj.name == "down":
        return 2.0 * d * d * spec_norm_estimate(model.ff, d) ** 2
    return ln


def _stats(err, logb, gate):
    return dict(mean_err=float(np.mean(err)), mean_logb=float(np.mean(logb)),
                ratio=float(np.mean(logb) / np.mean(err)), above=float(np.mean(err > logb)),
                max_gate=float(np.max(err / gate)))


@pytest.mark.parametrize("mech", ["gaussian", "laplace"])
def test_error_scales_as_one_over_eps(mech):
    # one Llama-shaped QKV slice: K = 3072, 64 tokens x 256 outputs, Delta of Theorem 1
    gm, om = MECH[mech]
    Mr, K, N = 64, 3072, 256
    delta = 2.0 * 3072 ** 0.75
    X = WL.gen_x(Mr, K, seed=1)
    W = WL.gen_w(N, K, seed=2)
    Wd = dev(W).to(torch.bfloat16)
    ref = O.gemm64(X, W)
    rows = {}
    for eps in EPS:
        sid = WL.stream_id(0, 0)
        C = sp.correction(Wd, Mr, gm, delta, eps, 0, sid, 0, sp.SPLITEE_PREC_BF16X3)
        Y = host(sp.masked_linear_fused(dev(X), Wd, C, gm, delta, eps, 0, sid, 0, sp.SPLITEE_PREC_BF16X3))
        eta = O.noise(Mr, K, om, delta, eps, 0, sid, 0)
        b = O.error_bounds(X, eta, O.mask(X, eta), W, O.PREC_BF16X3)
        err = np.abs(Y.astype(np.float64) - ref)
        assert np.all(err <= b["gate"]), (eps, float(np.max(err / b["gate"])))
        s = _stats(err, b["logb"], b["gate"])
        assert s["mean_err"] <= s["mean_logb"], (eps, s)
        rows[eps] = s
    print("\n%s, Delta %.2f: eps, mean err, mean Eq. fp-log-bound, ratio, share above, max err/gate" % (mech, delta))
    for eps, s in rows.items():
        print("  %4.1f  %.3e  %.3e  %6.1f  %.4f  %.3e" % (eps, s["mean_err"], s["mean_logb"], s["ratio"],
                                                        s["above"], s["max_gate"]))
    for a, b in zip(EPS, EPS[1:]):
        r = (rows[a]["mean_err"] * a) / (rows[b]["mean_err"] * b)
        assert 0.75 < r < 1.33, (a, b, r)


_W_CACHE = {}


def _weights(model, proj):
    key = (model.name, proj.name)
    if key not in _W_CACHE:
        _W_CACHE.clear()
        W = WL.gen_w(proj.N, proj.K, seed=2 + proj.group)
        _W_CACHE[key] = (W, sp.tile_weights(dev(W).to(torch.bfloat16)))
    return _W_CACHE[key]


def _grid(model, M, proj_name, nrows=8, ncols=256):
    # the bench's launch configuration: full projection shapes, tiled W, bf16x3 masked
    # input, the eps x mechanism grid; outputs checked on sampled rows and columns that
    # include the first and the last of each
    proj = next(p for p in model.projections() if p.name == proj_name)
    K, N = proj.K, proj.N
    W, T = _weights(model, proj)
    delta = paper_delta(model, proj)
    g = np.random.Generator(np.random.PCG64(97 + proj.group))
    rows = np.unique(np.concatenate([[0, M - 1], g.choice(M, size=nrows - 2, replace=False)]))
    cols = np.unique(np.concatenate([[0, N - 1], g.choice(N, size=ncols - 2, replace=False)]))
    Ws = W[cols]
    X = WL.gen_x(M, K, seed=1)
    Xd = dev(X)
    worst = 0.0
    for mech in ("laplace", "gaussian"):
        gm, om = MECH[mech]
        for eps in EPS:
            sid = WL.stream_id(1, proj.group)
            C = sp.correction(T, M, gm, delta, eps, 0, sid, 0, sp.SPLITEE_PREC_BF16X3)
            Y = host(sp.masked_linear_fused(Xd, T, C, gm, delta, eps, 0, sid, 0, sp.SPLITEE_PREC_BF16X3))
            for i in rows:
                eta = O.noise(1, K, om, delta, eps, 0, sid, int(i))
                b = O.error_bounds(X[i:i + 1], eta, O.mask(X[i:i + 1], eta), Ws, O.PREC_BF16X3)
                err = np.abs(Y[i, cols].astype(np.float64) - O.gemm64(X[i:i + 1], Ws)[0])
                assert np.all(err <= b["gate"][0]), (proj.name, mech, eps, int(i))
                worst = max(worst, float(np.max(err / b["gate"][0])))
    print("\n%s %s M=%d Delta %.4g: max err/gate %.3e" % (model.name, proj.name, M, delta, worst))


@pytest.mark.parametrize("proj", ["qkv", "o", "gate_up", "down"])
def test_llama_stack_m512_eps_mechanism_grid(proj):
    _grid(WL.LLAMA_3B, 512, proj)


@pytest.mark.parametrize("proj", ["qkv", "o", "gate_up", "down"])
def test_qwen_stack_m1024_eps_mechanism_grid(proj):
    _grid(WL.QWEN3_4B, 1024, proj)
