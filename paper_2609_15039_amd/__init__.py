"""Python binding of libsplitee.so, the MI355X DP-masked linear layer.

Argument marshalling only: every function below forwards to the C entry point
of the same name (declared in include/splitee.h) with device pointers taken
from torch tensors and the current torch stream.  All arithmetic runs in the
HIP kernels; there is no fallback.  If the library is not built the import
still works but every call raises.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsplitee.so")

SPLITEE_OK = 0
SPLITEE_MECH_LAPLACE, SPLITEE_MECH_GAUSSIAN, SPLITEE_MECH_NONE = 0, 1, 2
SPLITEE_F32, SPLITEE_BF16, SPLITEE_BF16_TILED = 0, 1, 2
SPLITEE_PREC_F32, SPLITEE_PREC_BF16, SPLITEE_PREC_BF16X3 = 0, 1, 2
MECHS = {"laplace": SPLITEE_MECH_LAPLACE, "gaussian": SPLITEE_MECH_GAUSSIAN, "none": SPLITEE_MECH_NONE}
PRECS = {"f32": SPLITEE_PREC_F32, "bf16": SPLITEE_PREC_BF16, "bf16x3": SPLITEE_PREC_BF16X3}
SPLITEE_BOUND_LN, SPLITEE_BOUND_ATT, SPLITEE_BOUND_ACT = 0, 1, 2

EXPORTED = [
    "splitee_abi_version", "splitee_status_string", "splitee_noise_gen", "splitee_mask",
    "splitee_masked_linear", "splitee_unmask", "splitee_fused_workspace_bytes",
    "splitee_masked_linear_fused", "splitee_correction",
    "splitee_noise_mask", "splitee_gemm_workspace_bytes", "splitee_masked_linear_unmask",
    "splitee_noise_gen_multi", "splitee_spectral_norm_workspace_bytes", "splitee_spectral_norm",
    "splitee_sensitivity_workspace_bytes", "splitee_sensitivity", "splitee_eps_per_token",
    "splitee_bank_path", "splitee_bank_workspace_bytes", "splitee_bank_create", "splitee_bank_open",
    "splitee_bank_info", "splitee_bank_load", "splitee_bank_close",
    "splitee_f64_workspace_bytes", "splitee_masked_linear_fused_f64", "splitee_correction_f64",
    "splitee_tiled_weights_bytes", "splitee_tile_weights", "splitee_masked_linear_fused_noalloc",
]
# test hooks (include/splitee_probe.h)
EXPORTED_PROBE = ["splitee_transform_probe", "splitee_mfma_probe"]
SPLITEE_PREC_F64 = 3
SPLITEE_ERR_IO, SPLITEE_ERR_EXHAUSTED, SPLITEE_ERR_FORMAT, SPLITEE_ERR_BUSY = -8, -9, -10, -11
SPLITEE_ERR_SCRATCH = -12
SPLITEE_NOALLOC_SCRATCH_BYTES = 64 << 20


class BankInfo(ctypes.Structure):
    """splitee_bank_info_t"""
    _fields_ = [("K", ctypes.c_int64), ("N", ctypes.c_int64), ("seed", ctypes.c_uint64),
                ("stream_id", ctypes.c_uint64), ("mech", ctypes.c_int32), ("prec", ctypes.c_int32),
                ("sensitivity", ctypes.c_double), ("epsilon", ctypes.c_double), ("row0", ctypes.c_int64),
                ("rows", ctypes.c_int64), ("consumed", ctypes.c_int64), ("bytes_stored", ctypes.c_int64),
                ("bytes_with_masks", ctypes.c_int64)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class SpliteeError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (fn, _status_text(status), status))


_lib = None


def load():
    """Load libsplitee.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libsplitee.so is not built (run __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    P, I, I64, U64, D, SZ = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_uint64,
                             ctypes.c_double, ctypes.c_size_t)
    sig = {
        "splitee_abi_version": (I, []),
        "splitee_status_string": (ctypes.c_char_p, [I]),
        "splitee_noise_gen": (I, [P, I64, I64, I64, I, D, D, U64, U64, U64, P]),
        "splitee_mask": (I, [P, I64, P, I64, P, I, I64, I64, I64, P]),
        "splitee_masked_linear": (I, [P, I, I64, P, I, I64, P, I64, I64, I64, I64, P]),
        "splitee_unmask": (I, [P, I64, P, I64, P, I64, I64, I64, P]),
        "splitee_fused_workspace_bytes": (SZ, [I64, I64, I64, I]),
        "splitee_masked_linear_fused": (I, [P, I64, P, I, I64, P, I64, P, I64, I64, I64, I64, I, D, D,
                                            U64, U64, U64, P, I, P, SZ, P]),
        "splitee_correction": (I, [P, I64, P, I, I64, I64, I64, I64, I, D, D, U64, U64, U64, I, P, SZ,
                                   P]),
        "splitee_transform_probe": (I, [P, I64, I, I, P, P]),
        "splitee_noise_mask": (I, [P, I64, P, I, I64, I64, I64, I, D, D, U64, U64, U64, P]),
        "splitee_gemm_workspace_bytes": (SZ, [I64, I64, I64, I]),
        "splitee_masked_linear_unmask": (I, [P, I, I64, P, I, I64, P, I64, P, I64, I64, I64, I64, P,
                                             SZ, P]),
        "splitee_noise_gen_multi": (I, [P, P, P, P, I, I, P, U64, I64, I, D, D, U64, U64, P]),
        "splitee_spectral_norm_workspace_bytes": (SZ, [I64, I64, I]),
        "splitee_spectral_norm": (I, [P, I, I64, I64, I64, I, U64, U64, P, P, P, SZ, P]),
        "splitee_sensitivity_workspace_bytes": (SZ, []),
        "splitee_sensitivity": (I, [I, I64, P, P, D, D, P, P, SZ, P]),
        "splitee_eps_per_token": (I, [D, I64, P]),
        "splitee_bank_path": (I, [ctypes.c_char_p, I64, I64, U64, ctypes.c_char_p, SZ]),
        "splitee_bank_workspace_bytes": (SZ, [I64, I64, I]),
        "splitee_bank_create": (I, [ctypes.c_char_p, P, I, I64, I64, I64, I, D, D, U64, U64, U64, I64, I, P, SZ,
                                    P]),
        "splitee_bank_open": (I, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_void_p)]),
        "splitee_bank_info": (I, [P, ctypes.POINTER(BankInfo)]),
        "splitee_bank_load": (I, [P, I64, P, I64, I, ctypes.POINTER(ctypes.c_int64), P]),
        "splitee_bank_close": (I, [P]),
        "splitee_f64_workspace_bytes": (SZ, [I64, I64, I64]),
        "splitee_masked_linear_fused_f64": (I, [P, I64, P, I, I64, P, I64, P, I64, I64, I64, I64, I, D, D, U64,
                                                U64, U64, P, SZ, P]),
        "splitee_correction_f64": (I, [P, I64, P, I, I64, I64, I64, I64, I, D, D, U64, U64, U64, P, SZ, P]),
        "splitee_tiled_weights_bytes": (SZ, [I64, I64]),
        "splitee_tile_weights": (I, [P, I64, I64, I64, P, P]),
        "splitee_mfma_probe": (I, [I, I, P, P, D, P, P]),
        "splitee_masked_linear_fused_noalloc": (I, [P, I64, P, I, I64, P, I64, P, I64, I64, I64, I64, I, D, D,
                                                    U64, U64, U64, P, I, P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _status_text(status):
    try:
        return load().splitee_status_string(status).decode()
    except Exception:  # library missing
        return "status"


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return stream


def _check(fn, status):
    if status != SPLITEE_OK:
        raise SpliteeError(fn, status)


class TiledWeights:
    """A bfloat16 N x K weight matrix stored in the tiled order of
    splitee_tile_weights (`data`, a flat device tensor).  Passed wherever a W tensor
    is taken; shape, dtype, stride and data_ptr describe the logical matrix."""

    dtype = torch.bfloat16

    def __init__(self, data, N, K):
        self.data, self.N, self.K = data, N, K

    @property
    def shape(self):
        return (self.N, self.K)

    @property
    def device(self):
        return self.data.device

    @property
    def is_cuda(self):
        return self.data.is_cuda

    def stride(self, dim):
        return (self.K, 1)[dim]

    def data_ptr(self):
        return self.data.data_ptr()


def _wtype(W):
    if isinstance(W, TiledWeights):
        return SPLITEE_BF16_TILED
    return SPLITEE_BF16 if W.dtype == torch.bfloat16 else SPLITEE_F32


# ------------------------------------------------------------ C entry points

def splitee_abi_version():
    return load().splitee_abi_version()


def splitee_status_string(status):
    return load().splitee_status_string(status).decode()


def splitee_tiled_weights_bytes(N, K):
    return load().splitee_tiled_weights_bytes(N, K)


def splitee_tile_weights(W, ldw, N, K, Wt, stream=None):
    _check("splitee_tile_weights", load().splitee_tile_weights(_ptr(W), ldw, N, K, _ptr(Wt), _stream(stream)))


def splitee_noise_gen(eta, ld_eta, M, K, mech, sensitivity, epsilon, seed, stream_id, row0=0,
                      stream=None):
    _check("splitee_noise_gen", load().splitee_noise_gen(
        _ptr(eta), ld_eta, M, K, mech, sensitivity, epsilon, seed, stream_id, row0, _stream(stream)))


def splitee_noise_gen_multi(etas, ld_etas, Ks, stream_ids, M, mech, sensitivity, epsilon, seed,
                            row0=0, reps=1, rep_strides=None, rep_sid_step=0, stream=None):
    """etas, ld_etas, Ks, stream_ids (and rep_strides when reps > 1): sequences of
    equal length, one entry per noise block."""
    n = len(etas)
    if not (len(ld_etas) == len(Ks) == len(stream_ids) == n):
        raise ValueError("splitee_noise_gen_multi: per-block sequences differ in length")
    ptrs = (ctypes.c_void_p * max(n, 1))(*[_ptr(e) for e in etas])
    lds = (ctypes.c_int64 * max(n, 1))(*ld_etas)
    ks = (ctypes.c_int64 * max(n, 1))(*Ks)
    sids = (ctypes.c_uint64 * max(n, 1))(*stream_ids)
    strides = None
    if rep_strides is not None:
        if len(rep_strides) != n:
            raise ValueError("splitee_noise_gen_multi: rep_strides differs in length")
        strides = ctypes.cast((ctypes.c_int64 * max(n, 1))(*rep_strides), ctypes.c_void_p)
    _check("splitee_noise_gen_multi", load().splitee_noise_gen_multi(
        ctypes.cast(ptrs, ctypes.c_void_p), ctypes.cast(lds, ctypes.c_void_p), ctypes.cast(ks, ctypes.c_void_p),
        ctypes.cast(sids, ctypes.c_void_p), n, reps, strides, rep_sid_step, M, mech, sensitivity, epsilon,
        seed, row0, _stream(stream)))


def splitee_mask(X, ldx, eta, ld_eta, Xt, out_prec, ldxt, M, K, stream=None):
    _check("splitee_mask", load().splitee_mask(
        _ptr(X), ldx, _ptr(eta), ld_eta, _ptr(Xt), out_prec, ldxt, M, K, _stream(stream)))


def splitee_masked_linear(Xt, in_prec, ldxt, W, w_type, ldw, R, ldr, M, N, K, stream=None):
    _check("splitee_masked_linear", load().splitee_masked_linear(
        _ptr(Xt), in_prec, ldxt, _ptr(W), w_type, ldw, _ptr(R), ldr, M, N, K, _stream(stream)))


def splitee_unmask(R, ldr, C, ldc, Y, ldy, M, N, stream=None):
    _check("splitee_unmask", load().splitee_unmask(
        _ptr(R), ldr, _ptr(C), ldc, _ptr(Y), ldy, M, N, _stream(stream)))


def splitee_fused_workspace_bytes(M, N, K, prec):
    return load().splitee_fused_workspace_bytes(M, N, K, prec)


def splitee_masked_linear_fused(X, ldx, W, w_type, ldw, C, ldc, Y, ldy, M, N, K, mech, sensitivity,
                                epsilon, seed, stream_id, row0, eta_override, prec, workspace,
                                workspace_bytes, stream=None):
    _check("splitee_masked_linear_fused", load().splitee_masked_linear_fused(
        _ptr(X), ldx, _ptr(W), w_type, ldw, _ptr(C), ldc, _ptr(Y), ldy, M, N, K, mech, sensitivity,
        epsilon, seed, stream_id, row0, _ptr(eta_override), prec, _ptr(workspace), workspace_bytes,
        _stream(stream)))


def splitee_masked_linear_fused_noalloc(X, ldx, W, w_type, ldw, C, ldc, Y, ldy, M, N, K, mech, sensitivity,
                                        epsilon, seed, stream_id, row0, eta_override, prec, stream=None):
    _check("splitee_masked_linear_fused_noalloc", load().splitee_masked_linear_fused_noalloc(
        _ptr(X), ldx, _ptr(W), w_type, ldw, _ptr(C), ldc, _ptr(Y), ldy, M, N, K, mech, sensitivity, epsilon, seed,
        stream_id, row0, _ptr(eta_override), prec, _stream(stream)))


def splitee_correction(C, ldc, W, w_type, ldw, M, N, K, mech, sensitivity, epsilon, seed,
                       stream_id, row0, prec, workspace, workspace_bytes, stream=None):
    _check("splitee_correction", load().splitee_correction(
        _ptr(C), ldc, _ptr(W), w_type, ldw, M, N, K, mech, sensitivity, epsilon, seed, stream_id,
        row0, prec, _ptr(workspace), workspace_bytes, _stream(stream)))


def splitee_transform_probe(words, n, fn, force_slow, out, stream=None):
    _check("splitee_transform_probe", load().splitee_transform_probe(
        _ptr(words), n, fn, force_slow, _ptr(out), _stream(stream)))


def splitee_mfma_probe(op, n, a, b, c, d, stream=None):
    _check("splitee_mfma_probe", load().splitee_mfma_probe(op, n, _ptr(a), _ptr(b), float(c), _ptr(d),
                                                           _stream(stream)))


def splitee_noise_mask(X, ldx, Xt, out_prec, ldxt, M, K, mech, sensitivity, epsilon, seed,
                       stream_id, row0=0, stream=None):
    _check("splitee_noise_mask", load().splitee_noise_mask(
        _ptr(X), ldx, _ptr(Xt), out_prec, ldxt, M, K, mech, sensitivity, epsilon, seed, stream_id,
        row0, _stream(stream)))


def splitee_gemm_workspace_bytes(M, N, K, prec):
    return load().splitee_gemm_workspace_bytes(M, N, K, prec)


def splitee_masked_linear_unmask(Xt, in_prec, ldxt, W, w_type, ldw, C, ldc, Y, ldy, M, N, K,
                                 workspace, workspace_bytes, stream=None):
    _check("splitee_masked_linear_unmask", load().splitee_masked_linear_unmask(
        _ptr(Xt), in_prec, ldxt, _ptr(W), w_type, ldw, _ptr(C), ldc, _ptr(Y), ldy, M, N, K,
        _ptr(workspace), workspace_bytes, _stream(stream)))


def splitee_spectral_norm_workspace_bytes(N, K, iters):
    return load().splitee_spectral_norm_workspace_bytes(N, K, iters)


def splitee_spectral_norm(W, w_type, ldw, N, K, iters, seed, stream_id, workspace, workspace_bytes,
                          history=False, stream=None):
    """Returns sigma of the last round, or (sigma, [sigma of every round]) with history."""
    sigma = ctypes.c_double()
    hist = (ctypes.c_double * iters)() if history and iters > 0 else None
    _check("splitee_spectral_norm", load().splitee_spectral_norm(
        _ptr(W), w_type, ldw, N, K, iters, seed, stream_id, ctypes.byref(sigma),
        ctypes.cast(hist, ctypes.c_void_p) if hist is not None else None, _ptr(workspace), workspace_bytes,
        _stream(stream)))
    return (sigma.value, list(hist) if hist is not None else []) if history else sigma.value


def splitee_sensitivity_workspace_bytes():
    return load().splitee_sensitivity_workspace_bytes()


def splitee_sensitivity(bound, d, alpha, beta, w_norm_a, w_norm_b, workspace, workspace_bytes, stream=None):
    """Returns the bound Delta f."""
    delta = ctypes.c_double()
    _check("splitee_sensitivity", load().splitee_sensitivity(
        bound, d, _ptr(alpha), _ptr(beta), w_norm_a, w_norm_b, ctypes.byref(delta), _ptr(workspace),
        workspace_bytes, _stream(stream)))
    return delta.value


def splitee_eps_per_token(eps_total, n):
    eps = ctypes.c_double()
    _check("splitee_eps_per_token", load().splitee_eps_per_token(eps_total, n, ctypes.byref(eps)))
    return eps.value


def splitee_f64_workspace_bytes(M, N, K):
    return load().splitee_f64_workspace_bytes(M, N, K)


def splitee_masked_linear_fused_f64(X, ldx, W, w_type, ldw, C, ldc, Y, ldy, M, N, K, mech, sensitivity, epsilon,
                                    seed, stream_id, row0, workspace, workspace_bytes, stream=None):
    _check("splitee_masked_linear_fused_f64", load().splitee_masked_linear_fused_f64(
        _ptr(X), ldx, _ptr(W), w_type, ldw, _ptr(C), ldc, _ptr(Y), ldy, M, N, K, mech, sensitivity, epsilon, seed,
        stream_id, row0, _ptr(workspace), workspace_bytes, _stream(stream)))


def splitee_correction_f64(C, ldc, W, w_type, ldw, M, N, K, mech, sensitivity, epsilon, seed, stream_id, row0,
                           workspace, workspace_bytes, stream=None):
    _check("splitee_correction_f64", load().splitee_correction_f64(
        _ptr(C), ldc, _ptr(W), w_type, ldw, M, N, K, mech, sensitivity, epsilon, seed, stream_id, row0,
        _ptr(workspace), workspace_bytes, _stream(stream)))


def splitee_bank_path(directory, K, N, stream_id):
    buf = ctypes.create_string_buffer(4096)
    _check("splitee_bank_path", load().splitee_bank_path(os.fsencode(directory), K, N, stream_id, buf, 4096))
    return os.fsdecode(buf.value)


def splitee_bank_workspace_bytes(K, N, prec):
    return load().splitee_bank_workspace_bytes(K, N, prec)


def splitee_bank_create(path, W, w_type, ldw, K, N, mech, sensitivity, epsilon, seed, stream_id, row0, rows, prec,
                        workspace, workspace_bytes, stream=None):
    _check("splitee_bank_create", load().splitee_bank_create(
        os.fsencode(path), _ptr(W), w_type, ldw, K, N, mech, sensitivity, epsilon, seed, stream_id, row0, rows,
        prec, _ptr(workspace), workspace_bytes, _stream(stream)))


def splitee_bank_open(path):
    """Returns the bank handle (an integer address)."""
    h = ctypes.c_void_p()
    _check("splitee_bank_open", load().splitee_bank_open(os.fsencode(path), ctypes.byref(h)))
    return h.value


def splitee_bank_info(bank):
    info = BankInfo()
    _check("splitee_bank_info", load().splitee_bank_info(bank, ctypes.byref(info)))
    return info.as_dict()


def splitee_bank_load(bank, rows, C, ldc, dst_device, stream=None):
    """C: a device tensor (dst_device true) or a host address / contiguous CPU tensor;
    returns the first stream row of the loaded rows."""
    row0 = ctypes.c_int64()
    if dst_device:
        ptr = _ptr(C)
    else:
        ptr = C if isinstance(C, int) or C is None else C.data_ptr()
    _check("splitee_bank_load", load().splitee_bank_load(bank, rows, ptr, ldc, 1 if dst_device else 0,
                                                         ctypes.byref(row0), _stream(stream) if dst_device else None))
    return row0.value


def splitee_bank_close(bank):
    _check("splitee_bank_close", load().splitee_bank_close(bank))


# ------------------------------------------------- tensor-level conveniences

def _aligned_bytes(nbytes, device):
    buf = torch.empty(max(nbytes, 1) + 256, dtype=torch.uint8, device=device)
    off = (-buf.data_ptr()) % 256
    return buf[off:off + max(nbytes, 1)]


def spectral_norm(W, iters, seed, stream_id, history=False, ws=None):
    """||W||_2 of a row-major N x K tensor by the power method (see splitee_spectral_norm)."""
    N, K = W.shape
    nbytes = splitee_spectral_norm_workspace_bytes(N, K, iters)
    if ws is None:
        ws = _aligned_bytes(nbytes, W.device)
    return splitee_spectral_norm(W, _wtype(W), W.stride(0), N, K, iters, seed, stream_id, ws, nbytes,
                                 history=history)


def workspace_f64(M, N, K, device="cuda"):
    """A 256-byte aligned workspace for the binary64 calls; returns (tensor, bytes)."""
    nbytes = splitee_f64_workspace_bytes(M, N, K)
    return _aligned_bytes(nbytes, device), nbytes


def correction_f64(W, M, mech, sensitivity, epsilon, seed, stream_id, row0=0, ws=None):
    N, K = W.shape
    C = torch.empty((M, N), dtype=torch.float64, device=W.device)
    if ws is None:
        ws = workspace_f64(M, N, K, W.device)
    splitee_correction_f64(C, N, W, _wtype(W), W.stride(0), M, N, K, mech, sensitivity, epsilon, seed, stream_id,
                           row0, ws[0], ws[1])
    return C


def masked_linear_fused_f64(X, W, C, mech, sensitivity, epsilon, seed, stream_id, row0=0, ws=None, Y=None):
    M, K = X.shape
    N = W.shape[0]
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float32, device=X.device)
    if ws is None:
        ws = workspace_f64(M, N, K, X.device)
    splitee_masked_linear_fused_f64(X, X.stride(0), W, _wtype(W), W.stride(0), C, C.stride(0), Y, Y.stride(0), M,
                                    N, K, mech, sensitivity, epsilon, seed, stream_id, row0, ws[0], ws[1])
    return Y


def bank_create(path, W, K, mech, sensitivity, epsilon, seed, stream_id, row0, rows, prec=SPLITEE_PREC_BF16X3):
    """Precompute and store the corrections of W (N x K) for `rows` stream rows."""
    N = W.shape[0]
    nbytes = splitee_bank_workspace_bytes(K, N, prec)
    ws = torch.zeros(nbytes + 256, dtype=torch.uint8, device=W.device)
    ws = ws[(-ws.data_ptr()) % 256:][:nbytes]
    splitee_bank_create(path, W, _wtype(W), W.stride(0), K, N, mech, sensitivity, epsilon, seed, stream_id, row0,
                        rows, prec, ws, nbytes)


def sensitivity(bound, alpha, beta=None, w_norm_a=0.0, w_norm_b=0.0):
    """Delta f of Theorem 1 (LN), 2 (ATT) or 3 (ACT) for float32 device vectors."""
    nbytes = splitee_sensitivity_workspace_bytes()
    ws = _aligned_bytes(nbytes, alpha.device)
    return splitee_sensitivity(bound, alpha.numel(), alpha, beta, w_norm_a, w_norm_b, ws, nbytes)


def workspace(M, N, K, prec, device="cuda", gemm_only=False):
    """A zeroed, 256-byte aligned workspace for the fused call / correction (or, with
    gemm_only, for splitee_masked_linear_unmask); returns (tensor, bytes)."""
    nbytes = (splitee_gemm_workspace_bytes if gemm_only else splitee_fused_workspace_bytes)(M, N, K, prec)
    ws = torch.zeros(max(nbytes, 1) + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws[off:off + max(nbytes, 1)], nbytes


def tile_weights(W):
    """W (N x K bfloat16, row-major) in the tiled order, as TiledWeights."""
    N, K = W.shape
    data = torch.empty(splitee_tiled_weights_bytes(N, K) // 2, dtype=torch.bfloat16, device=W.device)
    splitee_tile_weights(W, W.stride(0), N, K, data)
    return TiledWeights(data, N, K)


def noise(M, K, mech, sensitivity, epsilon, seed, stream_id, row0=0, device="cuda"):
    eta = torch.empty((M, K), dtype=torch.float32, device=device)
    splitee_noise_gen(eta, K, M, K, mech, sensitivity, epsilon, seed, stream_id, row0)
    return eta


def mask(X, eta, prec):
    M, K = X.shape
    planes = 3 if prec == SPLITEE_PREC_BF16X3 else 1
    dt = torch.float32 if prec == SPLITEE_PREC_F32 else torch.int16
    Xt = torch.empty((planes, M, K), dtype=dt, device=X.device)
    splitee_mask(X, X.stride(0), eta, eta.stride(0), Xt, prec, K, M, K)
    return Xt


def masked_linear(Xt, prec, W):
    M, K = Xt.shape[-2:]
    N = W.shape[0]
    R = torch.empty((M, N), dtype=torch.float32, device=W.device)
    splitee_masked_linear(Xt, prec, K, W, _wtype(W), W.stride(0), R, N, M, N, K)
    return R


def noise_mask(X, prec, mech, sensitivity, epsilon, seed, stream_id, row0=0):
    M, K = X.shape
    planes = 3 if prec == SPLITEE_PREC_BF16X3 else 1
    dt = {SPLITEE_PREC_F32: torch.float32, SPLITEE_PREC_F64: torch.float64}.get(prec, torch.int16)
    Xt = torch.empty((planes, M, K), dtype=dt, device=X.device)
    splitee_noise_mask(X, X.stride(0), Xt, prec, K, M, K, mech, sensitivity, epsilon, seed,
                       stream_id, row0)
    return Xt


def masked_linear_unmask(Xt, prec, W, C, ws=None, Y=None):
    M, K = Xt.shape[-2:]
    N = W.shape[0]
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float32, device=W.device)
    if ws is None:
        ws = workspace(M, N, K, prec, W.device, gemm_only=True)
    splitee_masked_linear_unmask(Xt, prec, K, W, _wtype(W), W.stride(0), C,
                                 C.stride(0) if C is not None else 0, Y, Y.stride(0), M, N, K,
                                 ws[0], ws[1])
    return Y


def unmask(R, C):
    M, N = R.shape
    Y = torch.empty((M, N), dtype=torch.float32, device=R.device)
    splitee_unmask(R, R.stride(0), C, C.stride(0), Y, N, M, N)
    return Y


def correction(W, M, mech, sensitivity, epsilon, seed, stream_id, row0=0, prec=SPLITEE_PREC_BF16X3,
               ws=None):
    N, K = W.shape
    C = torch.empty((M, N), dtype=torch.float32, device=W.device)
    if ws is None:
        ws = workspace(M, N, K, prec, W.device)
    splitee_correction(C, N, W, _wtype(W), W.stride(0), M, N, K, mech, sensitivity, epsilon, seed,
                       stream_id, row0, prec, ws[0], ws[1])
    return C


def masked_linear_fused(X, W, C, mech, sensitivity, epsilon, seed, stream_id, row0=0,
                        prec=SPLITEE_PREC_BF16X3, eta_override=None, ws=None, Y=None):
    M, K = X.shape
    N = W.shape[0]
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float32, device=X.device)
    if ws is None:
        ws = workspace(M, N, K, prec, X.device)
    splitee_masked_linear_fused(X, X.stride(0), W, _wtype(W), W.stride(0), C, C.stride(0), Y,
                                Y.stride(0), M, N, K, mech, sensitivity, epsilon, seed, stream_id,
                                row0, eta_override, prec, ws[0], ws[1])
    return Y
