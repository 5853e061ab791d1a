"""CPU oracle for the DP-masked linear layer -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The HIP library never calls it and shares
no code with it.

The method (Sec. "Offloading Linear Operations", Eq. add-and-then-subtract):
the trusted side adds a mask eta to the projection input x, the GPU computes
r = W (x + eta), and the trusted side subtracts the precomputed correction
W eta to get W x.  Over the reals the result is exactly W x, so every step here
is the plain definition written out:

  noise       eta      -- ``noise`` (C, binary128 transforms; see noise_ref.c)
  mask        Xt       = fl32(X + eta)                      -- ``mask``
  operand     Xhat     = Xt | bf16(Xt) | hi+mid+lo (== Xt)  -- ``gemm_operand``
  GEMM        R*       = Xhat . W^T in binary64             -- ``gemm64``
  correction  C*       = eta . W^T in binary64              -- ``gemm64``
  unmask      Y        = fl32(R - C)                        -- ``unmask``
  reference   Y*       = X . W^T in binary64                -- ``gemm64``
  bounds      Theorem 4 and Eq. fp-log-bound per element    -- ``error_bounds``
  binary64    Xt = fl64(X + eta) and its bound (Down)         -- ``mask64``, ``error_bounds_f64``

Layouts: X is M x K (tokens x in-features), W is N x K (out x in, the paper's
d' x d matrix acting on column vectors), Y = X W^T is M x N.
"""
import ctypes
import math
import os

import numpy as np

from . import build as _build

MECH_LAPLACE, MECH_GAUSSIAN, MECH_NONE = 0, 1, 2
PREC_F32, PREC_BF16, PREC_BF16X3 = 0, 1, 2
FN_LAPLACE_T, FN_GAUSS_R, FN_COS2PI, FN_SIN2PI = 0, 1, 2, 3

U32 = 2.0 ** -24  # unit round-off of binary32 (Eq. ulp with p = 24)
U64 = 2.0 ** -53  # unit round-off of binary64 (p = 53)
U_BF16 = 2.0 ** -8  # unit round-off of bfloat16 (p = 8)

_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_build.LIB):
        _build.build()
    lib = ctypes.CDLL(_build.LIB)
    P = ctypes.c_void_p
    i64, u64, u32 = ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint32
    lib.oracle_philox4x32_10.argtypes = [P, P, P]
    lib.oracle_philox4x32_10.restype = None
    lib.oracle_philox_batch.argtypes = [P, i64, u64, u64, P]
    lib.oracle_philox_batch.restype = None
    lib.oracle_transform_batch.argtypes = [ctypes.c_int, P, i64, P]
    lib.oracle_transform_batch.restype = i64
    lib.oracle_noise.argtypes = [P, i64, i64, i64, ctypes.c_int, ctypes.c_double,
                                 ctypes.c_double, u64, u64, u64]
    lib.oracle_noise.restype = ctypes.c_int
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def num_threads():
    """OpenMP threads of the oracle's C part."""
    return _load().oracle_num_threads()


# --------------------------------------------------------------------------- noise

def philox4x32_10(ctr, key):
    """One Philox4x32-10 block (Salmon et al., SC'11): 4 counter words, 2 key words."""
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    _load().oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def philox_blocks(blocks, seed, sid):
    """Philox words for block indices ``blocks`` under key=seed, counter hi = sid."""
    b = np.ascontiguousarray(blocks, dtype=np.uint64)
    out = np.zeros((b.size, 4), dtype=np.uint32)
    _load().oracle_philox_batch(_ptr(b), b.size, seed, sid, _ptr(out))
    return out


def transform(fn, words):
    """Correctly rounded binary32 transform of 32-bit words.

    fn: FN_LAPLACE_T (standard Laplace inverse CDF), FN_GAUSS_R (sqrt(-2 ln u)),
    FN_COS2PI, FN_SIN2PI, with u = (w + 1/2) 2^-32.
    """
    w = np.ascontiguousarray(words, dtype=np.uint32)
    out = np.zeros(w.size, dtype=np.float32)
    nhard = _load().oracle_transform_batch(fn, _ptr(w), w.size, _ptr(out))
    if nhard:
        raise ArithmeticError("%d words too close to a binary32 rounding boundary" % nhard)
    return out


def noise(M, K, mech, delta, eps, seed, sid, row0=0):
    """eta (M x K float32) for rows row0 .. row0+M-1 of stream (seed, sid).

    Prop. 2: eta ~ N(0, (Delta/eps)^2 I) for the Gaussian mechanism; the Laplace
    mechanism uses scale b = Delta/eps.  Generator and rounding: noise_ref.c.
    """
    eta = np.zeros((M, K), dtype=np.float32)
    rc = _load().oracle_noise(_ptr(eta), K, M, K, mech, float(delta), float(eps),
                              seed, sid, row0)
    if rc != 0:
        raise ValueError("oracle_noise failed with status %d" % rc)
    return eta


# ---------------------------------------------------------------------- mask / bf16

def bf16_rne(x):
    """Round binary32 values to the nearest bfloat16, ties to even.

    Returned as float32 arrays holding bfloat16 values.  The two bfloat16
    candidates around x are the truncation toward zero and the next value away
    from zero; the nearer one wins and a tie goes to the even significand.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    bits = x.view(np.uint32)
    down_bits = bits & np.uint32(0xFFFF0000)
    up_bits = down_bits + np.uint32(0x10000)
    down = down_bits.view(np.float32).astype(np.float64)
    up = up_bits.view(np.float32).astype(np.float64)
    xd = x.astype(np.float64)
    with np.errstate(invalid="ignore"):
        d_down = np.abs(xd - down)
        d_up = np.abs(up - xd)
    down_even = ((down_bits >> np.uint32(16)) & np.uint32(1)) == 0
    take_up = (d_up < d_down) | ((d_up == d_down) & ~down_even)
    res_bits = np.where(take_up, up_bits, down_bits)
    res_bits = np.where(np.isfinite(x), res_bits, bits)  # inf / nan pass through
    return res_bits.view(np.float32).reshape(x.shape)


def bf16_bits(x_bf16_as_f32):
    """Upper 16 bits of float32 arrays that hold bfloat16 values."""
    b = np.ascontiguousarray(x_bf16_as_f32, dtype=np.float32).view(np.uint32)
    return (b >> np.uint32(16)).astype(np.uint16)


def mask(X, eta):
    """Masked input Xt = fl32(X + eta): one IEEE binary32 addition per element."""
    return (np.asarray(X, dtype=np.float32) + np.asarray(eta, dtype=np.float32)).astype(np.float32)


def split3(xt):
    """Split binary32 Xt into three bfloat16 terms with hi + mid + lo == Xt.

    hi = bf16(Xt), mid = bf16(Xt - hi), lo = bf16(Xt - hi - mid); the two
    differences are exact in binary32 and lo equals the second residual exactly.
    """
    xt = np.asarray(xt, dtype=np.float32)
    hi = bf16_rne(xt)
    r1 = (xt - hi).astype(np.float32)
    mid = bf16_rne(r1)
    r2 = (r1 - mid).astype(np.float32)
    lo = bf16_rne(r2)
    return hi, mid, lo


def gemm_operand(xt, prec):
    """The GPU's A operand as exact binary64 values for precision mode ``prec``."""
    if prec == PREC_BF16:
        return bf16_rne(xt).astype(np.float64)
    if prec == PREC_BF16X3:
        hi, mid, lo = split3(xt)
        return hi.astype(np.float64) + mid.astype(np.float64) + lo.astype(np.float64)
    return np.asarray(xt, dtype=np.float64)


# ------------------------------------------------------------------- GEMM / unmask

def gemm64(A, W):
    """A . W^T in binary64 (A: M x K, W: N x K).

    Each product of binary32 or bfloat16 inputs is exact in binary64; the sum's
    own error is at most gamma_K(binary64) sum|a||w|, about 1e-12 relative.
    """
    return np.asarray(A, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T


def unmask(R, C):
    """Y = fl32(R - C) (Eq. add-and-then-subtract): one binary32 subtraction."""
    return (np.asarray(R, dtype=np.float32) - np.asarray(C, dtype=np.float32)).astype(np.float32)


# ------------------------------------------------------------------------- bounds

def gamma(n, u=U32):
    """gamma_n = n u / (1 - n u)  (Def. 6; requires n u < 1)."""
    nu = n * u
    if nu >= 1.0:
        raise ValueError("gamma_n undefined for n u >= 1")
    return nu / (1.0 - nu)


def mfma_bf16_coeff(K, planes):
    """c with |fl(A W^T) - A W^T| <= c sum_p sum_k |a^(p)_k| |w_k| for a length-K dot
    product that the GPU evaluates on bfloat16 matrix cores, A split into `planes`
    bfloat16 planes a^(p).

    These instructions do not round once per product sum.  Measured on the device (the
    MFMA probe test): the k depth is taken in groups of 8 consecutive k; in a group the
    products (exact) are truncated toward zero, and the running binary32 accumulator
    floored, to the grid 2^(E-24) of the group's largest product exponent E, then
    summed and rounded to nearest (Def. 6's u).  A group step is thus
        acc' = (acc + P_g + e_g)(1 + d),  |d| <= u,  |e_g| < 8 * 2^(E-24) <= 8 u max_g |p|
    (at most 7 products lose bits -- the largest, 16 significant bits at exponent E,
    never does -- plus the floor of acc).  Unrolled over n steps as in the proof of the
    dot-product bound: |error| <= gamma_n S + 8 u (1 + gamma_n) S.  n counts the steps
    a product passes: planes * ceil(K / 8) group steps plus, as an allowance for the
    binary32 additions outside the instruction chain (split-K partial sums, merged
    accumulators), one per 64-k tile.
    """
    n = planes * -(-K // 8) + -(-K // 64)
    g = gamma(n)
    return g + 8.0 * U32 * (1.0 + g)


# |hi| + |mid| + |lo| <= (1 + 2 u_bf16 + 2 u_bf16^2) |Xt| for the three-term split of Xt
SPLIT3_SUM = 1.0 + 2.0 ** -6


def acc_coeff(K, planes=None):
    """Accumulation-error coefficient that covers every kernel the GPU path may run for a
    length-K product: binary32 fused multiply-add chains (the binary32 matrix cores and
    the vector-ALU decode GEMV: K roundings, gamma_K) and, with `planes`, the bfloat16
    matrix cores on that many planes (mfma_bf16_coeff, times the planes' magnitude
    relative to |A|)."""
    c = gamma(K)
    if planes:
        c = max(c, mfma_bf16_coeff(K, planes) * (SPLIT3_SUM if planes == 3 else 1.0))
    return c


def error_bounds(X, eta, Xt, W, prec=PREC_F32):
    """Per-element error bounds for Y = fl32(fl(Xt W^T) - fl(eta W^T)) against X W^T.

    S_x = |W||x|, S_t = |W||x+eta| (with the rounded Xt), S_e = |W||eta|.
    thm4   : Theorem 4 with d = K, O(d u^2) dropped as in the paper.
    logb   : Eq. fp-log-bound, gamma_{ceil(log2 K)+1} in place of gamma_K.
    rigor  : the bound derived the same way for what the GPU computes against the
             exact reference -- it adds the rounding of x + eta, which Theorem 4
             treats as exact, keeps every second-order term, and takes the
             accumulation error of R and of the correction C from the arithmetic the
             kernels really perform (acc_coeff: c_R for R in this precision mode, c_C
             for C computed in F32 or BF16X3); for K >= 16 both equal gamma_K.
    gate   : max(thm4, rigor); thm4 whenever S_e <= (K-1) S_x (about), so the gate
             is never looser than the paper's bound where the paper's bound applies.
    For single-pass BF16 the input rounding u_bf16 * S_t is added to both.
    """
    Wa = np.abs(np.asarray(W, dtype=np.float64))
    K = Wa.shape[1]
    Sx = np.abs(np.asarray(X, dtype=np.float64)) @ Wa.T
    St = np.abs(np.asarray(Xt, dtype=np.float64)) @ Wa.T
    Se = np.abs(np.asarray(eta, dtype=np.float64)) @ Wa.T
    u = U32
    gK = gamma(K)
    glog = gamma(math.ceil(math.log2(K)) + 1)
    cR = acc_coeff(K, {PREC_BF16: 1, PREC_BF16X3: 3}.get(prec))
    cC = acc_coeff(K, 3)
    thm4 = gK * (Sx + St + Se) + u * Sx
    logb = glog * (Sx + St + Se) + u * Sx
    if prec == PREC_BF16:
        ub = U_BF16
        E = cR * (1.0 + ub) * St + ub * St + cC * Se + u * (Sx + Se)
        thm4 = thm4 + ub * St * (1.0 + gK)
        logb = logb + ub * St * (1.0 + glog)
    else:
        E = cR * St + cC * Se + u * (Sx + Se)
    rigor = (1.0 + u) * E + u * Sx
    gate = np.maximum(thm4, rigor)
    precond = Se <= (K - 1) * Sx
    return dict(Sx=Sx, St=St, Se=Se, thm4=thm4, logb=logb, rigor=rigor, gate=gate,
                precond=precond, c_R=cR, c_C=cC)


def mask64(X, eta):
    """Xt = fl64(X + eta): the mask in binary64, one addition of the binary32 operands
    (the remedy the paper names for the Down projection, Sec. "The Case Against the
    Down Linear Projection": binary64 instead of binary32)."""
    return np.asarray(X, dtype=np.float32).astype(np.float64) + np.asarray(eta, dtype=np.float32).astype(np.float64)


def error_bounds_f64(X, eta, W):
    """Per-element bound for Y = fl32(fl64(fl64(Xt W^T) - fl64(eta W^T))) against X W^T,
    Xt = fl64(X + eta): the derivation of Theorem 4 with the unit roundoff of binary64
    for the mask and both products, then one binary64 subtraction and one rounding to
    binary32.  With u = 2^-53, S_x, S_t (|Xt|) and S_e as in error_bounds:

      E     = gamma_K(u) (S_t + S_e) + 2 u S_t      products (any order) and the mask
      bound = E + (u32 + 2 u)(S_x + E)              subtraction, rounding to binary32
      thm4  = gamma_K(u) (S_x + S_t + S_e) + u S_x  Theorem 4 itself at u = 2^-53
    """
    Wa = np.abs(np.asarray(W, dtype=np.float64))
    K = Wa.shape[1]
    Sx = np.abs(np.asarray(X, dtype=np.float64)) @ Wa.T
    St = np.abs(mask64(X, eta)) @ Wa.T
    Se = np.abs(np.asarray(eta, dtype=np.float64)) @ Wa.T
    g = gamma(K, U64)
    E = g * (St + Se) + 2.0 * U64 * St
    bound = E + (U32 + 2.0 * U64) * (Sx + E)
    thm4 = g * (Sx + St + Se) + U64 * Sx
    return dict(Sx=Sx, St=St, Se=Se, E=E, bound=bound, thm4=thm4)


def dot_bound(A, W, k_acc=None, planes=None):
    """Higham's dot-product bound gamma_n sum|a||w| (used for R and C alone), n = k_acc
    (default K) roundings; with `planes`, at least the bound of the bfloat16 matrix
    cores on that many planes of A (acc_coeff), so that it covers every kernel."""
    Wa = np.abs(np.asarray(W, dtype=np.float64))
    K = Wa.shape[1]
    c = gamma(K if k_acc is None else k_acc)
    if planes:
        c = max(c, acc_coeff(K, planes))
    return c * (np.abs(np.asarray(A, dtype=np.float64)) @ Wa.T)


# ------------------------------------------------------------------- full pipeline

def masked_linear(X, W, mech, delta, eps, seed, sid, row0=0, prec=PREC_F32, eta=None):
    """The whole path for one projection, every step the plain definition.

    Returns a dict with eta, Xt, the exact R* and C*, the fp32 unmask of the
    rounded R*, C* (``Y``), the exact reference Y* = X W^T, and the bounds.
    """
    X = np.asarray(X, dtype=np.float32)
    M, K = X.shape
    if eta is None:
        eta = noise(M, K, mech, delta, eps, seed, sid, row0)
    Xt = mask(X, eta)
    R = gemm64(gemm_operand(Xt, prec), W)
    C = gemm64(eta, W)
    Y = unmask(R.astype(np.float32), C.astype(np.float32))
    Yref = gemm64(X, W)
    return dict(eta=eta, Xt=Xt, R=R, C=C, Y=Y, Yref=Yref,
                bounds=error_bounds(X, eta, Xt, W, prec))


# --------------------------------------------------------------- noise statistics

def laplace_cdf(x, b):
    x = np.asarray(x, dtype=np.float64)
    return np.where(x < 0, 0.5 * np.exp(x / b), 1.0 - 0.5 * np.exp(-x / b))


def gauss_cdf(x, sigma):
    x = np.asarray(x, dtype=np.float64)
    from scipy.special import erfc
    return 0.5 * erfc(-x / (sigma * math.sqrt(2.0)))


def ks_statistic(samples, cdf):
    """Kolmogorov-Smirnov distance of the empirical CDF from ``cdf``."""
    s = np.sort(np.asarray(samples, dtype=np.float64).ravel())
    n = s.size
    F = cdf(s)
    i = np.arange(1, n + 1, dtype=np.float64)
    return float(max(np.max(i / n - F), np.max(F - (i - 1) / n)))
