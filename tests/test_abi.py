"""The C-ABI library on the host: it loads, exports every declared entry point,
and rejects invalid arguments synchronously without touching a device.

The pointers passed here are never dereferenced: every call fails validation
before any launch (16 is a non-null, 16-byte aligned stand-in address).
"""
import ctypes
import math
import os
import re

import pytest

import paper_2609_15039_amd as sp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR = os.path.join(ROOT, "include", "splitee.h")
PROBE_HDR = os.path.join(ROOT, "include", "splitee_probe.h")
OK, ARG, SHAPE, DTYPE, ALIGN, UNSUP, HIP, WS = 0, -1, -2, -3, -4, -5, -6, -7
P = 16  # aligned stand-in pointer
L, G, NONE = 0, 1, 2
F32, BF16, TILED = 0, 1, 2
PF, PB, PX = 0, 1, 2


def declared_functions(hdr=HDR):
    text = open(hdr).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(splitee_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    return sp.load()


def test_library_exports_every_declared_function(lib):
    decl = declared_functions()
    assert set(decl) == set(sp.EXPORTED)
    probe = declared_functions(PROBE_HDR)
    assert set(probe) == set(sp.EXPORTED_PROBE)
    for name in decl + probe:
        assert hasattr(lib, name), name


def test_version_and_status_strings(lib):
    assert lib.splitee_abi_version() == 2
    for code in (OK, ARG, SHAPE, DTYPE, ALIGN, UNSUP, HIP, WS):
        assert lib.splitee_status_string(code)
    assert lib.splitee_status_string(12345) == b"unknown status"


def noise(lib, eta=P, ld=8, M=2, K=8, mech=L, d=1.0, e=1.0):
    return lib.splitee_noise_gen(eta, ld, M, K, mech, d, e, 0, 0, 0, None)


@pytest.mark.parametrize("kw,code", [
    (dict(e=0.0), ARG), (dict(e=-1.0), ARG), (dict(e=math.nan), ARG), (dict(e=math.inf), ARG),
    (dict(d=-1.0), ARG), (dict(d=math.nan), ARG), (dict(d=math.inf), ARG), (dict(mech=3), ARG),
    (dict(K=6, ld=8), SHAPE), (dict(ld=4), SHAPE), (dict(M=-1), SHAPE),
    (dict(eta=8), ALIGN), (dict(ld=10, K=8), ALIGN), (dict(eta=None), ARG),
    (dict(M=0), OK), (dict(K=0, ld=0), OK)])
def test_noise_gen_validation(lib, kw, code):
    assert noise(lib, **kw) == code


def noise_multi(lib, etas=(P, P), lds=(8, 16), ks=(8, 16), sids=(0, 1), count=None, reps=2,
                rep_strides=(64, 64), rep_sid_step=256, M=2, mech=G, d=1.0, e=1.0, null_arrays=False):
    n = len(etas)
    arr = lambda t, v: (t * max(n, 1))(*v)
    a = [arr(ctypes.c_void_p, etas), arr(ctypes.c_int64, lds), arr(ctypes.c_int64, ks),
         arr(ctypes.c_uint64, sids)]
    a = [None if null_arrays else ctypes.cast(x, ctypes.c_void_p) for x in a]
    st = None if rep_strides is None else ctypes.cast(arr(ctypes.c_int64, rep_strides), ctypes.c_void_p)
    return lib.splitee_noise_gen_multi(*a, n if count is None else count, reps, st, rep_sid_step, M,
                                       mech, d, e, 0, 0, None)


@pytest.mark.parametrize("kw,code", [
    (dict(e=0.0), ARG), (dict(d=math.inf), ARG), (dict(mech=5), ARG),
    (dict(count=9), ARG), (dict(count=-1), ARG), (dict(null_arrays=True), ARG),
    (dict(reps=-1), ARG), (dict(reps=65536), ARG), (dict(rep_strides=None), ARG),
    (dict(rep_strides=(64, -4)), SHAPE), (dict(rep_strides=(6, 64)), ALIGN),
    (dict(ks=(8, 6)), SHAPE), (dict(lds=(8, 12)), SHAPE), (dict(M=-3), SHAPE),
    (dict(etas=(P, 8)), ALIGN), (dict(lds=(8, 18)), ALIGN), (dict(etas=(P, None)), ARG),
    (dict(count=0, null_arrays=True), OK), (dict(reps=0, null_arrays=True), OK), (dict(M=0), OK),
    (dict(reps=1, rep_strides=None, M=0), OK),
    (dict(etas=(None, None), ks=(0, 0), lds=(0, 0)), OK)])
def test_noise_gen_multi_validation(lib, kw, code):
    assert noise_multi(lib, **kw) == code


def test_mask_validation(lib):
    f = lib.splitee_mask
    assert f(P, 8, P, 8, P, 7, 8, 2, 8, None) == UNSUP
    assert f(P, 8, P, 8, P, PF, 8, 2, 6, None) == SHAPE
    assert f(P, 4, P, 8, P, PF, 8, 2, 8, None) == SHAPE
    assert f(P, 8, None, 8, P, PF, 8, 2, 8, None) == ARG
    assert f(P, 8, P, 8, 8, PF, 8, 2, 8, None) == ALIGN
    assert f(P, 8, P, 8, P, PB, 12, 2, 8, None) == ALIGN  # 24-byte bf16 row pitch
    assert f(P, 8, P, 8, P, PB, 8, 0, 8, None) == OK


def test_masked_linear_validation(lib):
    f = lib.splitee_masked_linear
    assert f(P, PX, 8, P, F32, 8, P, 8, 2, 8, 8, None) == UNSUP  # BF16X3 needs bf16 W
    assert f(P, PB, 8, P, F32, 8, P, 8, 2, 8, 8, None) == UNSUP
    assert f(P, PF, 8, P, 5, 8, P, 8, 2, 8, 8, None) == DTYPE
    assert f(P, PF, 4, P, F32, 4, P, 4, 2, 4, 4, None) == SHAPE  # K % 8
    assert f(P, PF, 8, P, F32, 8, P, 4, 2, 8, 8, None) == SHAPE  # ldr < N
    assert f(P, PF, 8, 4, F32, 8, P, 8, 2, 8, 8, None) == ALIGN
    assert f(P, PF, 8, P, F32, 8, P, 8, 0, 8, 8, None) == OK


def test_unmask_validation(lib):
    f = lib.splitee_unmask
    assert f(P, 4, P, 8, P, 8, 2, 8, None) == SHAPE
    assert f(P, 8, P, 8, 4, 8, 2, 8, None) == ALIGN
    assert f(P, 8, None, 8, P, 8, 2, 8, None) == ARG
    assert f(P, 8, P, 8, P, 8, 2, 0, None) == OK


def fused(lib, X=P, W=P, wt=BF16, C=P, Y=P, M=2, N=8, K=8, mech=G, d=1.0, e=1.0, prec=PX,
          ws=256, wsb=1 << 20, eta=None):
    return lib.splitee_masked_linear_fused(X, K, W, wt, K, C, N, Y, N, M, N, K, mech, d, e, 0, 0, 0,
                                           eta, prec, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(e=0.0), ARG), (dict(d=-2.0), ARG), (dict(mech=9), ARG), (dict(prec=3), UNSUP),
    (dict(wt=F32), UNSUP), (dict(wt=F32, prec=PB), UNSUP), (dict(wt=4, prec=PF), DTYPE),
    (dict(K=4), SHAPE), (dict(C=None), ARG), (dict(X=None), ARG), (dict(Y=8), ALIGN),
    (dict(eta=8), ALIGN), (dict(wsb=0), WS), (dict(ws=None), WS), (dict(ws=16), ALIGN),
    (dict(M=0), OK), (dict(N=0), OK)])
def test_fused_validation(lib, kw, code):
    assert fused(lib, **kw) == code


def test_correction_validation(lib):
    f = lib.splitee_correction
    assert f(P, 8, P, BF16, 8, 2, 8, 8, G, 1.0, 1.0, 0, 0, 0, PB, 256, 1 << 20, None) == UNSUP
    assert f(P, 8, P, BF16, 8, 2, 8, 8, G, 1.0, 0.0, 0, 0, 0, PX, 256, 1 << 20, None) == ARG
    assert f(P, 8, P, BF16, 8, 2, 8, 8, G, 1.0, 1.0, 0, 0, 0, PX, 256, 0, None) == WS
    assert f(P, 8, P, BF16, 8, 0, 8, 8, G, 1.0, 1.0, 0, 0, 0, PX, 256, 0, None) == OK


def test_workspace_sizes(lib):
    q = lib.splitee_fused_workspace_bytes
    assert q(2, 8, 6, PX) == 0  # K % 8
    assert q(2, 8, 8, 7) == 0
    # the masked-input planes alone: 3 x M x K bfloat16, 256-byte rounded
    assert q(128, 5120, 3072, PX) >= 3 * 128 * 3072 * 2
    assert q(128, 5120, 3072, PF) >= 128 * 3072 * 4
    assert q(1, 6144, 2560, PX) % 256 == 0


def test_mfma_probe_validation(lib):
    for op, n in ((-1, 1), (4, 1), (0, 0), (0, 65), (3, -2)):
        assert lib.splitee_mfma_probe(op, n, P, P, 0.0, P, None) == ARG
    assert lib.splitee_mfma_probe(0, 1, None, P, 0.0, P, None) == ARG
    assert lib.splitee_mfma_probe(0, 1, P, P, 0.0, None, None) == ARG


def test_transform_probe_validation(lib):
    assert lib.splitee_transform_probe(P, 4, 4, 0, P, None) == ARG
    assert lib.splitee_transform_probe(P, 0, 0, 0, P, None) == OK


def spectral(lib, W=P, wt=BF16, ldw=8, N=4, K=8, iters=3, sigma=True, hist=None, ws=256, wsb=1 << 20):
    s = ctypes.c_double(-1.0)
    rc = lib.splitee_spectral_norm(W, wt, ldw, N, K, iters, 0, 0, ctypes.byref(s) if sigma else None, hist, ws,
                                   wsb, None)
    return rc, s.value


@pytest.mark.parametrize("kw,code", [
    (dict(wt=7), DTYPE), (dict(iters=0), ARG), (dict(iters=(1 << 20) + 1), ARG), (dict(sigma=False), ARG),
    (dict(K=12, ldw=16), SHAPE), (dict(ldw=4), SHAPE), (dict(N=-1), SHAPE), (dict(K=-8), SHAPE),
    (dict(W=None), ARG), (dict(W=8), ALIGN), (dict(ldw=12), ALIGN), (dict(wt=F32, ldw=10, K=8), ALIGN),
    (dict(ws=None), WS), (dict(wsb=16), WS), (dict(ws=16), ALIGN)])
def test_spectral_norm_validation(lib, kw, code):
    assert spectral(lib, **kw)[0] == code


def test_spectral_norm_of_empty_matrix_is_zero(lib):
    hist = (ctypes.c_double * 3)(7.0, 7.0, 7.0)
    for N, K in ((0, 8), (4, 0)):
        rc, s = spectral(lib, N=N, K=K, hist=ctypes.cast(hist, ctypes.c_void_p), ws=None, wsb=0)
        assert (rc, s, list(hist)) == (OK, 0.0, [0.0, 0.0, 0.0])


def test_spectral_norm_workspace_size(lib):
    q = lib.splitee_spectral_norm_workspace_bytes
    assert q(8, 8, 0) == 0 and q(-1, 8, 1) == 0
    # partial rows (one per 16 rows of W) dominate: float32 per column
    assert q(3072, 3072, 50) >= (3072 // 16) * 3072 * 4
    assert q(3072, 3072, 50) % 256 == 0
    assert q(3073, 3072, 50) > q(3072, 3072, 50)


def sens(lib, bound=0, d=8, alpha=P, beta=None, a=1.0, b=1.0, delta=True, ws=256, wsb=256):
    out = ctypes.c_double(-1.0)
    return lib.splitee_sensitivity(bound, d, alpha, beta, a, b, ctypes.byref(out) if delta else None, ws, wsb,
                                   None)


@pytest.mark.parametrize("kw,code", [
    (dict(bound=3), ARG), (dict(bound=-1), ARG), (dict(d=0), SHAPE), (dict(alpha=None), ARG),
    (dict(delta=False), ARG), (dict(bound=1, a=-1.0), ARG), (dict(bound=1, a=math.inf), ARG),
    (dict(bound=2, b=math.nan), ARG), (dict(ws=None), WS), (dict(wsb=8), WS), (dict(ws=16), ALIGN)])
def test_sensitivity_validation(lib, kw, code):
    assert sens(lib, **kw) == code


def test_sensitivity_ignores_norms_it_does_not_use(lib):
    # LN reads neither matrix norm and ATT not the second: invalid values there pass validation
    # (workspace too small keeps the call from launching)
    assert sens(lib, bound=0, a=math.nan, b=-1.0, wsb=8) == WS
    assert sens(lib, bound=1, b=math.nan, wsb=8) == WS


@pytest.mark.parametrize("eps,n", [(1.0, 1), (1.0, 128), (4.0, 512), (0.25, 10 ** 9)])
def test_eps_per_token_matches_the_oracle(lib, eps, n):
    from oracle import sensitivity as S
    assert sp.splitee_eps_per_token(eps, n) == S.eps_per_token(eps, n)


@pytest.mark.parametrize("eps,n", [(0.0, 4), (-1.0, 4), (math.inf, 4), (math.nan, 4), (1.0, 0), (1.0, -3)])
def test_eps_per_token_validation(lib, eps, n):
    out = ctypes.c_double()
    assert lib.splitee_eps_per_token(eps, n, ctypes.byref(out)) == ARG
    assert lib.splitee_eps_per_token(1.0, 4, None) == ARG


def f64_fused(lib, X=P, ldx=8, W=P, wt=BF16, ldw=8, C=P, ldc=8, Y=P, ldy=8, M=2, N=8, K=8, mech=G, d=1.0, e=1.0,
              ws=256, wsb=1 << 20):
    return lib.splitee_masked_linear_fused_f64(X, ldx, W, wt, ldw, C, ldc, Y, ldy, M, N, K, mech, d, e, 0, 0, 0, ws,
                                               wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(e=0.0), ARG), (dict(mech=3), ARG), (dict(K=12, ldx=12, ldw=16), SHAPE), (dict(ldc=4), SHAPE),
    (dict(ldy=4), SHAPE), (dict(ldx=4), SHAPE), (dict(wt=7), DTYPE), (dict(ldw=4), SHAPE), (dict(W=8), ALIGN),
    (dict(X=None), ARG), (dict(C=None), ARG), (dict(Y=None), ARG), (dict(C=8), ALIGN), (dict(X=8), ALIGN),
    (dict(ws=None, wsb=0), WS), (dict(wsb=64), WS), (dict(ws=16), ALIGN), (dict(M=0), OK), (dict(N=0), OK)])
def test_fused_f64_validation(lib, kw, code):
    assert f64_fused(lib, **kw) == code


def test_correction_f64_validation_and_workspace(lib):
    f = lib.splitee_correction_f64
    assert f(P, 4, P, BF16, 8, 2, 8, 8, G, 1.0, 1.0, 0, 0, 0, 256, 1 << 20, None) == SHAPE
    assert f(None, 8, P, BF16, 8, 2, 8, 8, G, 1.0, 1.0, 0, 0, 0, 256, 1 << 20, None) == ARG
    assert f(P, 8, P, BF16, 8, 2, 8, 8, G, -1.0, 1.0, 0, 0, 0, 256, 1 << 20, None) == ARG
    assert f(P, 8, P, BF16, 8, 2, 8, 8, G, 1.0, 1.0, 0, 0, 0, None, 0, None) == WS
    q = lib.splitee_f64_workspace_bytes
    assert q(2, 8, 6) == 0
    assert q(128, 3072, 8192) >= 128 * 8192 * 8  # the binary64 masked input
    assert q(128, 3072, 8192) % 256 == 0


# ------------------------------------------------------------ tiled weight order

@pytest.mark.parametrize("N,K", [(1, 8), (32, 64), (33, 64), (200, 264), (5120, 3072), (128256, 3072)])
def test_tiled_weights_bytes(lib, N, K):
    # 32-row blocks of 64-k tiles, 4 KB each
    assert lib.splitee_tiled_weights_bytes(N, K) == -(-N // 32) * -(-K // 64) * 4096
    assert lib.splitee_tiled_weights_bytes(N, K) >= N * K * 2


def test_tiled_weights_bytes_invalid(lib):
    assert lib.splitee_tiled_weights_bytes(8, 12) == 0
    assert lib.splitee_tiled_weights_bytes(-1, 8) == 0
    assert lib.splitee_tiled_weights_bytes(0, 8) == 0


def test_tile_weights_validation(lib):
    f = lib.splitee_tile_weights
    big = 1 << 20
    assert f(P, 8, 4, 12, big, None) == SHAPE    # K % 8
    assert f(P, 4, 4, 8, big, None) == SHAPE     # ldw < K
    assert f(None, 8, 4, 8, big, None) == ARG
    assert f(P, 8, 4, 8, None, None) == ARG
    assert f(8, 8, 4, 8, big, None) == ALIGN
    assert f(P, 12, 4, 8, big, None) == ALIGN    # 24-byte row pitch
    assert f(P, 8, 4, 8, big + 8, None) == ALIGN
    assert f(big, 8, 4, 8, big + 32, None) == ARG  # Wt overlaps the 64 bytes of W
    assert f(P, 8, 0, 8, big, None) == OK


def test_tiled_weights_are_rejected_where_unsupported(lib):
    assert lib.splitee_masked_linear(P, PF, 8, P, TILED, 8, P, 8, 2, 8, 8, None) == UNSUP
    assert lib.splitee_masked_linear(P, PX, 8, 8, TILED, 8, P, 8, 2, 8, 8, None) == ALIGN
    assert lib.splitee_masked_linear(P, PX, 8, P, TILED, 0, P, 8, 0, 8, 8, None) == OK  # ldw unused
    assert fused(lib, wt=TILED, prec=PF) == UNSUP
    assert fused(lib, wt=TILED, W=8) == ALIGN
    assert fused(lib, wt=TILED, M=0) == OK
    assert lib.splitee_correction(P, 8, P, TILED, 8, 2, 8, 8, G, 1.0, 1.0, 0, 0, 0, PF, 256, 1 << 20,
                                  None) == UNSUP
    assert f64_fused(lib, wt=TILED) == UNSUP
    assert spectral(lib, wt=TILED)[0] == UNSUP


@pytest.mark.parametrize("M,N,K", [(128, 16384, 3072), (128, 5120, 3072), (512, 16384, 3072), (64, 19456, 2560),
                                   (1, 151936, 2560)])
def test_workspace_queries_cover_both_layouts(lib, M, N, K):
    # the largest split-K partial set of either plan fits: tiles x splits x tile floats
    gq, fq = lib.splitee_gemm_workspace_bytes, lib.splitee_fused_workspace_bytes
    for prec in (PB, PX):
        assert fq(M, N, K, prec) >= gq(M, N, K, prec)
        assert gq(M, N, K, prec) % 4 == 0


def test_noalloc_validation(lib):
    # the fused call's checks, then the static scratch limit, all before any device call
    G3 = PX
    fn = lib.splitee_masked_linear_fused_noalloc
    args = dict(X=P, ldx=264, W=P, wt=BF16, ldw=264, C=P, ldc=96, Y=P, ldy=96, M=37, N=96, K=264, mech=G, d=1.0,
                e=1.0, eta=None, prec=G3)

    def call(**kw):
        a = dict(args, **kw)
        return fn(a["X"], a["ldx"], a["W"], a["wt"], a["ldw"], a["C"], a["ldc"], a["Y"], a["ldy"], a["M"], a["N"],
                  a["K"], a["mech"], a["d"], a["e"], 0, 0, 0, a["eta"], a["prec"], None)

    assert call(e=0.0) == ARG
    assert call(K=260, ldx=264, ldw=264) == SHAPE
    assert call(X=8) == ALIGN
    assert call(X=None) == ARG
    assert call(prec=7) == UNSUP
    assert call(M=0) == OK
    assert call(M=4096, N=2560, K=9728, ldx=9728, ldw=9728, ldc=2560, ldy=2560) == sp.SPLITEE_ERR_SCRATCH
