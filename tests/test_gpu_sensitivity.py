"""GPU parity of the noise-scale entry points (splitee_spectral_norm,
splitee_sensitivity) against the oracle in oracle/sensitivity.py.

Bars:
- first round of the power method: |sigma_gpu - sigma*| <= || gamma_L |W| |v0| ||_2 with
  L = 8 ceil(K / 2048) + 12 (the float32 roundings along one product term: the thread's
  fma chain over its 8-column chunks, the 6-level wave tree, the 3 cross-wave adds, the
  1/||g|| factor and its product, plus one for the binary64 norms), sigma* = ||W v0||
  in binary64;
- every later round: relative difference <= gamma_L sqrt(||W||_1 ||W||_inf) / sigma* from the
  binary64 oracle run from the same start: each GPU round is an exact power-method step on
  a matrix within gamma_L |W| of W elementwise, whose singular values are within
  gamma_L || |W| ||_2 <= gamma_L sqrt(||W||_1 ||W||_inf) of W's (Weyl);
- never above ||W||_2 (binary64 SVD) beyond that bound; closed forms where the
  spectrum is known (relative 1e-5);
- the sensitivity bounds: relative 1e-12 (binary64 sums of d terms).
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_15039_amd as sp
import workloads as WL
from oracle import sensitivity as S

pytestmark = pytest.mark.gpu

DEV = "cuda"


def dev_w(W, w_dtype):
    t = torch.from_numpy(np.ascontiguousarray(W)).to(DEV)
    return t.to(torch.bfloat16) if w_dtype == "bf16" else t


def start_vector(K, seed, sid):
    # the standard Gaussian row 0 of noise stream (seed, sid), as the GPU draws it
    return O.noise(1, K, O.MECH_GAUSSIAN, 1.0, 1.0, seed, sid)[0].astype(np.float64)


def rounding_terms(K):
    return 8 * math.ceil(K / 2048) + 12


def first_round_bound(W, v0):
    b = O.dot_bound((v0 / np.linalg.norm(v0))[None, :], W, k_acc=rounding_terms(W.shape[1]))[0]
    return float(np.linalg.norm(b))


def later_rounds_rtol(W, sigma):
    Wa = np.abs(np.asarray(W, dtype=np.float64))
    abs_norm = math.sqrt(Wa.sum(axis=0).max() * Wa.sum(axis=1).max())
    return O.gamma(rounding_terms(W.shape[1])) * abs_norm / sigma


SHAPES = [  # (N, K, w dtype, rounds)
    (48, 64, "f32", 20),
    (37, 200, "bf16", 25),          # ragged rows (not a multiple of 16) and columns
    (16, 8, "bf16", 5),
    (1, 4096, "f32", 3),            # a single row: every round gives ||W||_2
    (1024, 3072, "bf16", 30),       # Llama-3.2-3B W_val (8 kv heads of 128)
    (3072, 3072, "bf16", 30),       # Llama-3.2-3B W_q / W_o
    (8192, 3072, "bf16", 30),       # Llama-3.2-3B W_up / W_gate
    (3072, 8192, "bf16", 30),       # Llama-3.2-3B W_down
    (9728, 2560, "bf16", 20),       # Qwen3-4B W_up / W_gate
    (2560, 9728, "bf16", 20),       # Qwen3-4B W_down
    (700, 16384, "f32", 4),         # the widest K: eight column chunks per thread
    (5000, 12296, "bf16", 4),       # ragged chunk count (7), more row tiles than workgroups
]


@pytest.mark.parametrize("N,K,wd,iters", SHAPES)
def test_power_method_rounds_match_oracle(N, K, wd, iters):
    seed, sid = 11, WL.stream_id(27, 5)
    W = WL.gen_w(N, K, seed=100 + N % 97, dtype=wd)
    v0 = start_vector(K, seed, sid)
    sig, hist = sp.spectral_norm(dev_w(W, wd), iters, seed, sid, history=True)
    ref = S.power_iteration(W, v0, iters)
    hist = np.array(hist)
    assert sig == hist[-1]
    assert abs(hist[0] - ref[0]) <= first_round_bound(W, v0)
    np.testing.assert_allclose(hist, ref, rtol=later_rounds_rtol(W, ref[-1]), atol=0)


def test_power_method_never_exceeds_the_spectral_norm():
    N, K = 600, 264
    W = WL.gen_w(N, K, seed=8, dtype="f32")
    v0 = start_vector(K, 3, 4)
    _, hist = sp.spectral_norm(dev_w(W, "f32"), 200, 3, 4, history=True)
    s = S.spectral_norm(W)
    tol = later_rounds_rtol(W, s)
    assert max(hist) <= s * (1 + tol)
    assert hist[-1] >= hist[0]
    assert hist[-1] == pytest.approx(S.power_iteration(W, v0, 200)[-1], rel=tol)


def _orthogonal(n, seed):
    q, r = np.linalg.qr(np.random.Generator(np.random.PCG64(seed)).standard_normal((n, n)))
    return q * np.sign(np.diag(r))


def test_scaled_orthogonal_matrix_gives_its_scale_every_round():
    # every singular value is 3.25: sigma = 3.25 from the first round on
    Q = (3.25 * _orthogonal(256, 1)).astype(np.float32)
    _, hist = sp.spectral_norm(dev_w(Q, "f32"), 4, 0, 0, history=True)
    np.testing.assert_allclose(hist, 3.25, rtol=1e-5)


def test_rank_one_matrix_converges_after_one_round():
    # W = a b^T: iteration 1 gives ||a|| |b . v0| / ||v0||, every later iteration ||a|| ||b||
    g = np.random.Generator(np.random.PCG64(5))
    a, b = g.standard_normal(300), g.standard_normal(512)
    W = np.outer(a, b).astype(np.float32)
    v0 = start_vector(512, 2, 9)
    _, hist = sp.spectral_norm(dev_w(W, "f32"), 4, 2, 9, history=True)
    W64 = W.astype(np.float64)
    assert hist[0] == pytest.approx(np.linalg.norm(W64 @ (v0 / np.linalg.norm(v0))), rel=1e-5)
    np.testing.assert_allclose(hist[1:], S.spectral_norm(W64), rtol=1e-5)


def test_gapped_spectrum_reaches_the_top_singular_value():
    # singular values 2, then 1 .. 0.1: the error shrinks by (1/2)^2 per round
    m, n = 96, 160
    U, V = _orthogonal(m, 2), _orthogonal(n, 3)
    s = np.linspace(1.0, 0.1, m)
    s[0] = 2.0
    W = (U @ np.diag(s) @ V[:m]).astype(np.float32)
    sig = sp.spectral_norm(dev_w(W, "f32"), 40, 1, 1)
    assert sig == pytest.approx(S.spectral_norm(W), rel=1e-5)


def test_power_method_is_deterministic_and_reads_only_k_columns():
    N, K = 1000, 1024
    W = WL.gen_w(N, K, seed=4)
    Wd = dev_w(W, "bf16")
    a = sp.spectral_norm(Wd, 12, 7, 7, history=True)
    b = sp.spectral_norm(Wd, 12, 7, 7, history=True)
    assert a == b
    # the same matrix inside a wider allocation with NaN padding columns
    Wp = torch.full((N, K + 64), float("nan"), dtype=torch.bfloat16, device=DEV)
    Wp[:, :K] = Wd
    nbytes = sp.splitee_spectral_norm_workspace_bytes(N, K, 12)
    ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=DEV)
    ws = ws[(-ws.data_ptr()) % 256:][:nbytes]
    c = sp.splitee_spectral_norm(Wp, sp.SPLITEE_BF16, K + 64, N, K, 12, 7, 7, ws, nbytes, history=True)
    assert c == a


def test_k_beyond_the_register_tile_is_rejected():
    W = torch.zeros((4, 16392), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(sp.SpliteeError):
        sp.spectral_norm(W, 2, 0, 0)


def test_zero_matrix_gives_zero():
    _, hist = sp.spectral_norm(torch.zeros((40, 64), device=DEV), 3, 0, 0, history=True)
    assert hist == [0.0, 0.0, 0.0]


# ------------------------------------------------------------ sensitivity bounds

@pytest.mark.parametrize("d", [8, 2560, 3072, 1001])
def test_sensitivity_bounds_match_oracle(d):
    alpha, beta = WL.gen_norm(d, seed=d)
    a, b = torch.from_numpy(alpha).to(DEV), torch.from_numpy(beta).to(DEV)
    na, nb = 1.7358144427371918, 2.9090558002207105
    got_ln = sp.sensitivity(sp.SPLITEE_BOUND_LN, a)
    got_att = sp.sensitivity(sp.SPLITEE_BOUND_ATT, a, w_norm_a=na)
    got_act = sp.sensitivity(sp.SPLITEE_BOUND_ACT, a, b, na, nb)
    got_act0 = sp.sensitivity(sp.SPLITEE_BOUND_ACT, a, None, na, nb)
    a64 = alpha.astype(np.float64)
    assert got_ln == pytest.approx(S.delta_ln(d, a64), rel=1e-12)
    assert got_att == pytest.approx(S.delta_att(d, a64, na), rel=1e-12)
    assert got_act == pytest.approx(S.delta_act(d, a64, beta.astype(np.float64), na, nb), rel=1e-12)
    assert got_act0 == pytest.approx(S.delta_act(d, a64, None, na, nb), rel=1e-12)


@pytest.mark.parametrize("d", [2560, 3072])
def test_untrained_ln_bound_is_2_d_three_quarters(d):
    one = torch.ones(d, device=DEV)
    assert sp.sensitivity(sp.SPLITEE_BOUND_LN, one) == pytest.approx(2 * d ** 0.75, rel=1e-14)


def test_noise_scale_of_a_llama_layer_down_projection():
    # Theorem 3 for the Down input of a Llama-3.2-3B-shaped layer with random weights:
    # spectral norms from the power method, the bound near 1e8 (the reason the paper
    # keeps Down in the TEE)
    d, ff = 3072, 8192
    seed = 21
    w_up, w_gate = WL.gen_w(ff, d, seed=31), WL.gen_w(ff, d, seed=32)
    n_up = sp.spectral_norm(dev_w(w_up, "bf16"), 60, seed, 1)
    n_gate = sp.spectral_norm(dev_w(w_gate, "bf16"), 60, seed, 2)
    s_up = S.spectral_norm(w_up)
    assert s_up * 0.97 <= n_up <= s_up * (1 + later_rounds_rtol(w_up, s_up))
    alpha = torch.ones(d, device=DEV)
    delta = sp.sensitivity(sp.SPLITEE_BOUND_ACT, alpha, None, n_up, n_gate)
    assert delta == pytest.approx(S.delta_act(d, np.ones(d), None, n_up, n_gate), rel=1e-12)
    assert 5e7 < delta < 5e8
