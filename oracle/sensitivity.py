"""CPU oracle for the noise scale -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module; the HIP library never calls it.

The scale of the Gaussian mask is Delta f / eps (Prop. 2) with Delta f the
global l2-sensitivity of the component whose output the projection reads
(Sec. "Global Sensitivity Analysis"):

  after layer normalisation (Theorem 1)   2 sqrt(d) ||alpha||_4
  after attention           (Theorem 2)   2 sqrt(d) ||W_val||_2 ||alpha||_4
  after the SiLU activation (Theorem 3)   2 sqrt(d) (sqrt(d) ||alpha||_4 + ||beta||_2)^2 ||W_up||_2 ||W_gate||_2

||W||_2 is the spectral norm, the largest singular value (the inequality the
paper calls Eq. matrix-norm).  Everything here is binary64.

The functions the bounds are about (used by the tests to check the bounds
against sampled and constructed inputs) follow their definitions: the
normalisation of Definition "normalization", LN of Eq. ln, attention of
Eq. att-mech-normalized and the activation of Eq. activation-function.
"""
import math

import numpy as np


def norm4(v):
    """||v||_4 in binary64."""
    v = np.asarray(v, dtype=np.float64)
    return float(np.sum(v ** 4) ** 0.25)


def delta_ln(d, alpha):
    """Theorem 1: sensitivity bound of LN(x; alpha, beta)."""
    return 2.0 * math.sqrt(d) * norm4(alpha)


def delta_att(d, alpha, w_val_norm):
    """Theorem 2: sensitivity bound of the attention output."""
    return 2.0 * math.sqrt(d) * w_val_norm * norm4(alpha)


def delta_act(d, alpha, beta, w_up_norm, w_gate_norm):
    """Theorem 3: sensitivity bound of the SiLU-gated activation."""
    b2 = 0.0 if beta is None else float(np.linalg.norm(np.asarray(beta, dtype=np.float64)))
    return 2.0 * math.sqrt(d) * (math.sqrt(d) * norm4(alpha) + b2) ** 2 * w_up_norm * w_gate_norm


def spectral_norm(W):
    """||W||_2: the largest singular value (binary64 SVD of the library)."""
    return float(np.linalg.norm(np.asarray(W, dtype=np.float64), 2))


def power_iteration(W, v0, iters):
    """The power method on W^T W from the start v0, in binary64: each round
    u = W v, sigma = ||u|| (v has unit norm), z = W^T u, v = z / ||z||.
    Returns the sigma of every round (non-decreasing, bounded by ||W||_2)."""
    W = np.asarray(W, dtype=np.float64)
    v = np.asarray(v0, dtype=np.float64)
    v = v / np.linalg.norm(v)
    out = []
    for _ in range(iters):
        u = W @ v
        out.append(float(np.linalg.norm(u)))
        z = W.T @ u
        v = z / np.linalg.norm(z)
    return np.array(out)


def eps_per_token(eps_total, n):
    """Per-token eps that makes n sequential eps-GDP releases eps_total-GDP
    (Prop. "Sequential Composition": sqrt(eps_1^2 + ... + eps_n^2))."""
    return eps_total / math.sqrt(n)


# ------------------------------------------------------------ the functions

def normalize(x, gamma=0.0, rms=True):
    """Definition "normalization": z-score (rms=False) or RMS normalisation."""
    x = np.asarray(x, dtype=np.float64)
    mu = 0.0 if rms else x.mean()
    var = np.mean((x - mu) ** 2)
    return (x - mu) / math.sqrt(var + gamma)


def layer_norm(x, alpha, beta=None, gamma=0.0, rms=True):
    """Eq. ln: alpha (.) xhat + beta."""
    y = np.asarray(alpha, dtype=np.float64) * normalize(x, gamma, rms)
    return y if beta is None else y + np.asarray(beta, dtype=np.float64)


def attention(xq, xs, w_qry, w_key, w_val, alpha, beta=None, gamma=0.0):
    """Eq. att-mech-normalized: W_val beta + sum_i p_i W_val (alpha (.) xhat_i), with
    p = softmax(<q, k_i> / sqrt(d)) for q = W_qry LN(xq), k_i = W_key LN(x_i)."""
    d = len(xq)
    q = w_qry @ layer_norm(xq, alpha, beta, gamma)
    ks = [w_key @ layer_norm(x, alpha, beta, gamma) for x in xs]
    s = np.array([q @ k / math.sqrt(d) for k in ks])
    p = np.exp(s - s.max())
    p /= p.sum()
    out = np.zeros(w_val.shape[0])
    for pi, x in zip(p, xs):
        out += pi * (w_val @ (np.asarray(alpha, dtype=np.float64) * normalize(x, gamma)))
    if beta is not None:
        out += w_val @ np.asarray(beta, dtype=np.float64)
    return out


def activation(x, w_up, w_gate, alpha, beta=None, gamma=0.0):
    """Eq. activation-function: W_up LN(x) (.) W_gate LN(x) (.) sig(W_gate LN(x))."""
    h = layer_norm(x, alpha, beta, gamma)
    g = w_gate @ h
    return (w_up @ h) * g / (1.0 + np.exp(-g))
