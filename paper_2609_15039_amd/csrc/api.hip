// C ABI of the DP-masked linear layer: argument validation and kernel launches.
// Semantics of every entry point are documented in include/splitee.h.
#include <math.h>

#include <mutex>

#include "common.hpp"
#include "splitee_probe.h"

namespace splitee_host {
size_t gemm_counter_bytes(int64_t M, int64_t N, int64_t K, int prec, int w_type);
size_t skinny_counter_bytes(int64_t M, int64_t N, int64_t K, int prec, int w_type);
}

namespace {

constexpr int64_t MAX_DIM = int64_t(1) << 30;
constexpr int MAX_POWER_ITERS = 1 << 20;

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline size_t align256(size_t b) { return (b + 255) / 256 * 256; }
inline bool pitch16(int64_t ld, int64_t elsize) { return (ld * elsize) % 16 == 0; }
inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

inline bool valid_mech(int mech)
{
    return mech == SPLITEE_MECH_LAPLACE || mech == SPLITEE_MECH_GAUSSIAN || mech == SPLITEE_MECH_NONE;
}

inline int check_noise_args(int mech, double sensitivity, double epsilon)
{
    if (!valid_mech(mech)) return SPLITEE_ERR_ARG;
    if (!(epsilon > 0.0) || !isfinite(epsilon)) return SPLITEE_ERR_ARG;
    if (!(sensitivity >= 0.0) || !isfinite(sensitivity)) return SPLITEE_ERR_ARG;
    return SPLITEE_OK;
}

inline bool dims_ok(int64_t M, int64_t N, int64_t K)
{
    return M >= 0 && N >= 0 && K >= 0 && M <= MAX_DIM && N <= MAX_DIM && K <= MAX_DIM;
}

inline int64_t prec_elsize(int prec) { return prec == SPLITEE_PREC_F64 ? 8 : prec == SPLITEE_PREC_F32 ? 4 : 2; }
inline int64_t prec_planes(int prec) { return prec == SPLITEE_PREC_BF16X3 ? 3 : 1; }
inline bool valid_prec(int prec)
{
    return prec == SPLITEE_PREC_F32 || prec == SPLITEE_PREC_BF16 || prec == SPLITEE_PREC_BF16X3;
}
inline bool valid_dtype(int t) { return t == SPLITEE_F32 || t == SPLITEE_BF16 || t == SPLITEE_BF16_TILED; }

// Skinny kernel for decode-sized M with bfloat16 operands, tiled kernel otherwise.
inline bool use_skinny(int64_t M, int prec) { return M <= 16 && prec != SPLITEE_PREC_F32; }

size_t gemm_ws(int64_t M, int64_t N, int64_t K, int prec, int w_type)
{
    return use_skinny(M, prec) ? splitee_host::skinny_workspace_bytes(M, N, K, prec, w_type)
                               : splitee_host::gemm_workspace_bytes(M, N, K, prec, w_type);
}
// Workspace queries take no weight layout: the larger of the row-major and the
// tiled plan (the float32 MFMA path reads row-major W only).
size_t gemm_ws_any(int64_t M, int64_t N, int64_t K, int prec)
{
    const size_t a = gemm_ws(M, N, K, prec, SPLITEE_BF16);
    const size_t b = prec == SPLITEE_PREC_F32 ? 0 : gemm_ws(M, N, K, prec, SPLITEE_BF16_TILED);
    return a > b ? a : b;
}
size_t gemm_counters(int64_t M, int64_t N, int64_t K, int prec, int w_type)
{
    return use_skinny(M, prec) ? splitee_host::skinny_counter_bytes(M, N, K, prec, w_type)
                               : splitee_host::gemm_counter_bytes(M, N, K, prec, w_type);
}

// GEMM operand checks shared by the GEMM entry points.
int check_w(const void* W, int w_type, int64_t ldw, int64_t K, int prec)
{
    if (!valid_dtype(w_type)) return SPLITEE_ERR_DTYPE;
    if (w_type == SPLITEE_BF16_TILED) { // ldw is not used: the layout is fixed by N and K
        if (prec == SPLITEE_PREC_F32) return SPLITEE_ERR_UNSUPPORTED;
        return aligned16(W) ? SPLITEE_OK : SPLITEE_ERR_ALIGN;
    }
    if (prec != SPLITEE_PREC_F32 && w_type != SPLITEE_BF16) return SPLITEE_ERR_UNSUPPORTED;
    const int64_t wes = w_type == SPLITEE_F32 ? 4 : 2;
    if (ldw < K) return SPLITEE_ERR_SHAPE;
    if (!aligned16(W) || !pitch16(ldw, wes)) return SPLITEE_ERR_ALIGN;
    return SPLITEE_OK;
}

// GEMM (+ unmask) on a masked input already in memory.
int run_gemm(const void* Xt, int prec, int64_t ldxt, const void* W, int w_type, int64_t ldw,
             const float* C, int64_t ldc, float* Y, int64_t ldy, int64_t M, int64_t N, int64_t K,
             void* ws, size_t ws_bytes, hipStream_t s)
{
    if (use_skinny(M, prec))
        return splitee_host::launch_skinny(Xt, prec, ldxt, M * ldxt, W, w_type, ldw, C, ldc, Y, ldy, M, N, K, ws,
                                           ws_bytes, s);
    return splitee_host::launch_gemm(Xt, prec, ldxt, M * ldxt, W, w_type, ldw, C, ldc, Y, ldy, M, N, K,
                                     ws, ws_bytes, s);
}

// Noise + mask into the workspace, then the GEMM with the unmask epilogue.
// X == nullptr computes the correction (A = eta, no C).
int run_masked(const float* X, int64_t ldx, const void* W, int w_type, int64_t ldw, const float* C,
               int64_t ldc, float* Y, int64_t ldy, int64_t M, int64_t N, int64_t K, int mech,
               double sensitivity, double epsilon, uint64_t seed, uint64_t sid, uint64_t row0,
               const float* eta_override, int prec, void* ws, size_t ws_bytes, hipStream_t s)
{
    const size_t gws = align256(gemm_ws(M, N, K, prec, w_type));
    const size_t need = gws + align256((size_t)(prec_planes(prec) * M * K * prec_elsize(prec)));
    if (ws_bytes < need || (need > 0 && ws == nullptr)) return SPLITEE_ERR_WORKSPACE;
    if (ws && (reinterpret_cast<uintptr_t>(ws) & 255u)) return SPLITEE_ERR_ALIGN;
    if (M == 0 || N == 0) return SPLITEE_OK;
    char* base = reinterpret_cast<char*>(ws);
    if (eta_override && use_skinny(M, prec))
        // decode with a precomputed mask: the GEMM forms fl32(X + eta) itself
        return splitee_host::launch_skinny_masked(X, ldx, eta_override, K, prec, W, w_type, ldw, C, ldc, Y, ldy, M, N,
                                                  K, base, gws, s);
    if (eta_override) {
        // prefill-sized M with a precomputed mask: the streamed GEMM forms fl32(X + eta)
        // itself where its plan allows (64-row tiles), else the two launches below
        const int rc = splitee_host::launch_gemm_masked(X, ldx, eta_override, K, prec, W, w_type, C, ldc, Y, ldy, M, N,
                                                        K, base, gws, s);
        if (rc != SPLITEE_ERR_UNSUPPORTED) return rc;
    }
    void* Xt = base + gws;
    unsigned* counters = reinterpret_cast<unsigned*>(base);
    const int64_t ncounters = (int64_t)(gemm_counters(M, N, K, prec, w_type) / 4);
    const double scale = sensitivity / epsilon;
    int rc = splitee_host::launch_mask(X, ldx, eta_override, K, mech, scale, seed, sid, row0, Xt, prec,
                                       K, M * K, M, K, counters, ncounters, s);
    if (rc != SPLITEE_OK) return rc;
    return run_gemm(Xt, prec, K, W, w_type, ldw, C, ldc, Y, ldy, M, N, K, base, gws, s);
}

// Binary64 path: the mask fl64(X + eta) (or eta alone for the correction) into the
// workspace, then the binary64 GEMM with the unmask epilogue.
size_t f64_ws(int64_t M, int64_t N, int64_t K)
{
    return align256((size_t)M * K * 8) + align256(splitee_host::f64_gemm_workspace_bytes(M, N, K));
}

int run_f64(const float* X, int64_t ldx, const void* W, int w_type, int64_t ldw, const double* C, int64_t ldc,
            void* Out, bool out64, int64_t ldo, int64_t M, int64_t N, int64_t K, int mech, double sensitivity,
            double epsilon, uint64_t seed, uint64_t sid, uint64_t row0, void* ws, size_t ws_bytes, hipStream_t s)
{
    const size_t need = f64_ws(M, N, K);
    if (ws_bytes < need || (need > 0 && ws == nullptr)) return SPLITEE_ERR_WORKSPACE;
    if (ws && (reinterpret_cast<uintptr_t>(ws) & 255u)) return SPLITEE_ERR_ALIGN;
    if (M == 0 || N == 0) return SPLITEE_OK;
    char* base = reinterpret_cast<char*>(ws);
    double* Xt = reinterpret_cast<double*>(base);
    const size_t xt_bytes = align256((size_t)M * K * 8);
    int rc = splitee_host::launch_mask(X, ldx, nullptr, 0, mech, sensitivity / epsilon, seed, sid, row0, Xt,
                                       SPLITEE_PREC_F64, K, 0, M, K, nullptr, 0, s);
    if (rc != SPLITEE_OK) return rc;
    return splitee_host::launch_gemm_f64(Xt, K, W, w_type, ldw, C, ldc, Out, out64, ldo, M, N, K, base + xt_bytes,
                                         ws_bytes - xt_bytes, s);
}

int check_w_f64(const void* W, int w_type, int64_t ldw, int64_t K)
{
    if (!valid_dtype(w_type)) return SPLITEE_ERR_DTYPE;
    if (w_type == SPLITEE_BF16_TILED) return SPLITEE_ERR_UNSUPPORTED;
    if (ldw < K) return SPLITEE_ERR_SHAPE;
    if (!aligned16(W) || !pitch16(ldw, w_type == SPLITEE_F32 ? 4 : 2)) return SPLITEE_ERR_ALIGN;
    return SPLITEE_OK;
}

// ------------------------------------------------------ no-allocation entry point
// The scratch space of splitee_masked_linear_fused_noalloc: a file-scope device array
// (one copy per GPU, held until the process ends).  Host code never passes the
// array's name to a kernel -- on the host it is only a stand-in symbol -- but the
// device address hipGetSymbolAddress returns for the current device, looked up once
// per device and kept.
static __device__ __align__(256) unsigned char scratch[SPLITEE_NOALLOC_SCRATCH_BYTES];

constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex scratch_mutex;
void* scratch_ptr[SCRATCH_MAX_DEVICES] = {};

// The current device's copy of `scratch`, or nullptr if it cannot be resolved.
void* scratch_for_current_device()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= SCRATCH_MAX_DEVICES) return nullptr;
    std::lock_guard<std::mutex> lock(scratch_mutex);
    if (!scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return nullptr;
        scratch_ptr[dev] = p;
    }
    return scratch_ptr[dev];
}

// Zero-fills n words: the split-K tile counters must read zero when a call starts.
__global__ void __launch_bounds__(256) zero_words_kernel(unsigned* __restrict__ p, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = 0u;
}

}  // namespace

extern "C" {

int splitee_abi_version(void) { return SPLITEE_ABI_VERSION; }

size_t splitee_tiled_weights_bytes(int64_t N, int64_t K)
{
    if (!dims_ok(0, N, K) || K % 8 != 0) return 0;
    return splitee::tiled_weights_bytes(N, K);
}

int splitee_tile_weights(const void* W, int64_t ldw, int64_t N, int64_t K, void* Wt, void* stream)
{
    if (!dims_ok(0, N, K) || K % 8 != 0 || ldw < K) return SPLITEE_ERR_SHAPE;
    if (N == 0 || K == 0) return SPLITEE_OK;
    if (!W || !Wt) return SPLITEE_ERR_ARG;
    if (!aligned16(W) || !pitch16(ldw, 2) || !aligned16(Wt)) return SPLITEE_ERR_ALIGN;
    const char* a = reinterpret_cast<const char*>(W);
    const char* b = reinterpret_cast<const char*>(Wt);
    const size_t in_bytes = (size_t)((N - 1) * ldw + K) * 2, out_bytes = splitee::tiled_weights_bytes(N, K);
    if (a < b + out_bytes && b < a + in_bytes) return SPLITEE_ERR_ARG; // in place is not supported
    return splitee_host::launch_tile_weights(reinterpret_cast<const uint16_t*>(W), ldw, N, K,
                                             reinterpret_cast<uint16_t*>(Wt), as_stream(stream));
}

const char* splitee_status_string(int status)
{
    switch (status) {
    case SPLITEE_OK: return "ok";
    case SPLITEE_ERR_ARG: return "invalid argument (mechanism, sensitivity, epsilon or null pointer)";
    case SPLITEE_ERR_SHAPE: return "invalid shape or leading dimension";
    case SPLITEE_ERR_DTYPE: return "invalid data type";
    case SPLITEE_ERR_ALIGN: return "pointer or row pitch not 16-byte aligned";
    case SPLITEE_ERR_UNSUPPORTED: return "unsupported precision / data type combination";
    case SPLITEE_ERR_HIP: return "HIP launch failed";
    case SPLITEE_ERR_WORKSPACE: return "workspace missing or too small";
    case SPLITEE_ERR_IO: return "bank file could not be created, opened, read or written";
    case SPLITEE_ERR_EXHAUSTED: return "noise bank has fewer unused rows than requested";
    case SPLITEE_ERR_FORMAT: return "bank file header or size is invalid";
    case SPLITEE_ERR_BUSY: return "bank file is open in another handle";
    case SPLITEE_ERR_SCRATCH:
        return "shape needs more scratch than the no-allocation entry point's static device buffer "
               "(SPLITEE_NOALLOC_SCRATCH_BYTES) holds";
    default: return "unknown status";
    }
}

int splitee_noise_gen(float* eta, int64_t ld_eta, int64_t M, int64_t K, int mech,
                      double sensitivity, double epsilon, uint64_t seed, uint64_t stream_id,
                      uint64_t row0, void* stream)
{
    int rc = check_noise_args(mech, sensitivity, epsilon);
    if (rc) return rc;
    if (!dims_ok(M, 0, K) || K % 4 != 0 || ld_eta < K) return SPLITEE_ERR_SHAPE;
    if (M == 0 || K == 0) return SPLITEE_OK;
    if (!eta) return SPLITEE_ERR_ARG;
    if (!aligned16(eta) || !pitch16(ld_eta, 4)) return SPLITEE_ERR_ALIGN;
    return splitee_host::launch_noise(eta, ld_eta, M, K, mech, sensitivity / epsilon, seed, stream_id,
                                      row0, as_stream(stream));
}

int splitee_noise_gen_multi(float* const* eta, const int64_t* ld_eta, const int64_t* K,
                            const uint64_t* stream_id, int count, int reps, const int64_t* rep_stride,
                            uint64_t rep_sid_step, int64_t M, int mech, double sensitivity, double epsilon,
                            uint64_t seed, uint64_t row0, void* stream)
{
    int rc = check_noise_args(mech, sensitivity, epsilon);
    if (rc) return rc;
    if (count < 0 || count > splitee::NOISE_MULTI_MAX || reps < 0 || reps > 65535) return SPLITEE_ERR_ARG;
    if (count == 0 || reps == 0) return SPLITEE_OK;
    if (!eta || !ld_eta || !K || !stream_id) return SPLITEE_ERR_ARG;
    if (reps > 1 && !rep_stride) return SPLITEE_ERR_ARG;
    if (!dims_ok(M, 0, 0)) return SPLITEE_ERR_SHAPE;
    for (int q = 0; q < count; ++q) {
        if (!dims_ok(M, 0, K[q]) || K[q] % 4 != 0 || ld_eta[q] < K[q]) return SPLITEE_ERR_SHAPE;
        if (reps > 1 && rep_stride[q] < 0) return SPLITEE_ERR_SHAPE;
        if (reps > 1 && rep_stride[q] % 4 != 0) return SPLITEE_ERR_ALIGN;
        if (M > 0 && K[q] > 0 && !eta[q]) return SPLITEE_ERR_ARG;
        if (eta[q] && (!aligned16(eta[q]) || !pitch16(ld_eta[q], 4))) return SPLITEE_ERR_ALIGN;
    }
    if (M == 0) return SPLITEE_OK;
    return splitee_host::launch_noise_multi(eta, ld_eta, K, stream_id, count, reps, rep_stride, rep_sid_step, M,
                                            mech, sensitivity / epsilon, seed, row0, as_stream(stream));
}

int splitee_mask(const float* X, int64_t ldx, const float* eta, int64_t ld_eta, void* Xt,
                 int out_prec, int64_t ldxt, int64_t M, int64_t K, void* stream)
{
    if (!valid_prec(out_prec) && out_prec != SPLITEE_PREC_F64) return SPLITEE_ERR_UNSUPPORTED;
    if (!dims_ok(M, 0, K) || K % 4 != 0 || ld_eta < K || ldxt < K || (X && ldx < K))
        return SPLITEE_ERR_SHAPE;
    if (M == 0 || K == 0) return SPLITEE_OK;
    if (!eta || !Xt) return SPLITEE_ERR_ARG;
    if (!aligned16(eta) || !pitch16(ld_eta, 4) || !aligned16(Xt) ||
        !pitch16(ldxt, prec_elsize(out_prec)) || (X && (!aligned16(X) || !pitch16(ldx, 4))))
        return SPLITEE_ERR_ALIGN;
    // bfloat16 rows are written 4 elements (8 bytes) at a time; the 16-byte row
    // pitch keeps every store aligned.
    return splitee_host::launch_mask(X, ldx, eta, ld_eta, SPLITEE_MECH_NONE, 0.0, 0, 0, 0, Xt, out_prec,
                                     ldxt, M * ldxt, M, K, nullptr, 0, as_stream(stream));
}

int splitee_noise_mask(const float* X, int64_t ldx, void* Xt, int out_prec, int64_t ldxt, int64_t M,
                       int64_t K, int mech, double sensitivity, double epsilon, uint64_t seed,
                       uint64_t stream_id, uint64_t row0, void* stream)
{
    int rc = check_noise_args(mech, sensitivity, epsilon);
    if (rc) return rc;
    if (!valid_prec(out_prec) && out_prec != SPLITEE_PREC_F64) return SPLITEE_ERR_UNSUPPORTED;
    if (!dims_ok(M, 0, K) || K % 4 != 0 || ldxt < K || (X && ldx < K)) return SPLITEE_ERR_SHAPE;
    if (M == 0 || K == 0) return SPLITEE_OK;
    if (!Xt) return SPLITEE_ERR_ARG;
    if (!aligned16(Xt) || !pitch16(ldxt, prec_elsize(out_prec)) || (X && (!aligned16(X) || !pitch16(ldx, 4))))
        return SPLITEE_ERR_ALIGN;
    return splitee_host::launch_mask(X, ldx, nullptr, 0, mech, sensitivity / epsilon, seed, stream_id,
                                     row0, Xt, out_prec, ldxt, M * ldxt, M, K, nullptr, 0,
                                     as_stream(stream));
}

int splitee_masked_linear(const void* Xt, int in_prec, int64_t ldxt, const void* W, int w_type,
                          int64_t ldw, float* R, int64_t ldr, int64_t M, int64_t N, int64_t K,
                          void* stream)
{
    if (!valid_prec(in_prec)) return SPLITEE_ERR_UNSUPPORTED;
    if (!dims_ok(M, N, K) || K % 8 != 0 || ldxt < K || ldr < N) return SPLITEE_ERR_SHAPE;
    int rc = check_w(W, w_type, ldw, K, in_prec);
    if (rc) return rc;
    if (M == 0 || N == 0) return SPLITEE_OK;
    if (!Xt || !W || !R) return SPLITEE_ERR_ARG;
    if (!aligned16(Xt) || !pitch16(ldxt, prec_elsize(in_prec)) || !aligned16(R) || !pitch16(ldr, 4))
        return SPLITEE_ERR_ALIGN;
    return splitee_host::launch_gemm(Xt, in_prec, ldxt, M * ldxt, W, w_type, ldw, nullptr, 0, R, ldr, M,
                                     N, K, nullptr, 0, as_stream(stream));
}

int splitee_unmask(const float* R, int64_t ldr, const float* C, int64_t ldc, float* Y, int64_t ldy,
                   int64_t M, int64_t N, void* stream)
{
    if (!dims_ok(M, N, 0) || ldr < N || ldc < N || ldy < N) return SPLITEE_ERR_SHAPE;
    if (M == 0 || N == 0) return SPLITEE_OK;
    if (!R || !C || !Y) return SPLITEE_ERR_ARG;
    if (!aligned16(R) || !aligned16(C) || !aligned16(Y) || !pitch16(ldr, 4) || !pitch16(ldc, 4) ||
        !pitch16(ldy, 4))
        return SPLITEE_ERR_ALIGN;
    return splitee_host::launch_unmask(R, ldr, C, ldc, Y, ldy, M, N, as_stream(stream));
}

size_t splitee_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int prec)
{
    if (!valid_prec(prec) || !dims_ok(M, N, K) || K % 8 != 0) return 0;
    return gemm_ws_any(M, N, K, prec);
}

int splitee_masked_linear_unmask(const void* Xt, int in_prec, int64_t ldxt, const void* W,
                                 int w_type, int64_t ldw, const float* C, int64_t ldc, float* Y,
                                 int64_t ldy, int64_t M, int64_t N, int64_t K, void* workspace,
                                 size_t workspace_bytes, void* stream)
{
    if (!valid_prec(in_prec)) return SPLITEE_ERR_UNSUPPORTED;
    if (!dims_ok(M, N, K) || K % 8 != 0 || ldxt < K || ldy < N || (C && ldc < N)) return SPLITEE_ERR_SHAPE;
    int rc = check_w(W, w_type, ldw, K, in_prec);
    if (rc) return rc;
    const size_t need = gemm_ws(M, N, K, in_prec, w_type);
    if (workspace_bytes < need || (need > 0 && workspace == nullptr)) return SPLITEE_ERR_WORKSPACE;
    if (workspace && (reinterpret_cast<uintptr_t>(workspace) & 255u)) return SPLITEE_ERR_ALIGN;
    if (M == 0 || N == 0) return SPLITEE_OK;
    if (!Xt || !W || !Y) return SPLITEE_ERR_ARG;
    if (!aligned16(Xt) || !pitch16(ldxt, prec_elsize(in_prec)) || !aligned16(Y) || !pitch16(ldy, 4) ||
        (C && (!aligned16(C) || !pitch16(ldc, 4))))
        return SPLITEE_ERR_ALIGN;
    return run_gemm(Xt, in_prec, ldxt, W, w_type, ldw, C, ldc, Y, ldy, M, N, K, workspace,
                    workspace_bytes, as_stream(stream));
}

size_t splitee_fused_workspace_bytes(int64_t M, int64_t N, int64_t K, int prec)
{
    if (!valid_prec(prec) || !dims_ok(M, N, K) || K % 8 != 0) return 0;
    return align256(gemm_ws_any(M, N, K, prec)) +
           align256((size_t)(prec_planes(prec) * M * K * prec_elsize(prec)));
}

int splitee_masked_linear_fused(const float* X, int64_t ldx, const void* W, int w_type, int64_t ldw,
                                const float* C, int64_t ldc, float* Y, int64_t ldy, int64_t M,
                                int64_t N, int64_t K, int mech, double sensitivity, double epsilon,
                                uint64_t seed, uint64_t stream_id, uint64_t row0,
                                const float* eta_override, int prec, void* workspace,
                                size_t workspace_bytes, void* stream)
{
    int rc = check_noise_args(mech, sensitivity, epsilon);
    if (rc) return rc;
    if (!valid_prec(prec)) return SPLITEE_ERR_UNSUPPORTED;
    if (!dims_ok(M, N, K) || K % 8 != 0 || ldx < K || ldc < N || ldy < N) return SPLITEE_ERR_SHAPE;
    rc = check_w(W, w_type, ldw, K, prec);
    if (rc) return rc;
    if (M == 0 || N == 0) return SPLITEE_OK;
    if (!X || !W || !C || !Y) return SPLITEE_ERR_ARG;
    if (!aligned16(X) || !pitch16(ldx, 4) || !aligned16(C) || !pitch16(ldc, 4) || !aligned16(Y) ||
        !pitch16(ldy, 4) || (eta_override && !aligned16(eta_override)))
        return SPLITEE_ERR_ALIGN;
    // an injected mask is M x K with leading dimension K
    return run_masked(X, ldx, W, w_type, ldw, C, ldc, Y, ldy, M, N, K, mech, sensitivity, epsilon,
                      seed, stream_id, row0, eta_override, prec, workspace, workspace_bytes,
                      as_stream(stream));
}

int splitee_masked_linear_fused_noalloc(const float* X, int64_t ldx, const void* W, int w_type, int64_t ldw,
                                        const float* C, int64_t ldc, float* Y, int64_t ldy, int64_t M, int64_t N,
                                        int64_t K, int mech, double sensitivity, double epsilon, uint64_t seed,
                                        uint64_t stream_id, uint64_t row0, const float* eta_override, int prec,
                                        void* stream)
{
    // the checks of splitee_masked_linear_fused, then the scratch size against the static buffer
    int rc = check_noise_args(mech, sensitivity, epsilon);
    if (rc) return rc;
    if (!valid_prec(prec)) return SPLITEE_ERR_UNSUPPORTED;
    if (!dims_ok(M, N, K) || K % 8 != 0 || ldx < K || ldc < N || ldy < N) return SPLITEE_ERR_SHAPE;
    rc = check_w(W, w_type, ldw, K, prec);
    if (rc) return rc;
    if (M == 0 || N == 0) return SPLITEE_OK;
    if (!X || !W || !C || !Y) return SPLITEE_ERR_ARG;
    if (!aligned16(X) || !pitch16(ldx, 4) || !aligned16(C) || !pitch16(ldc, 4) || !aligned16(Y) ||
        !pitch16(ldy, 4) || (eta_override && !aligned16(eta_override)))
        return SPLITEE_ERR_ALIGN;
    const size_t need = align256(gemm_ws(M, N, K, prec, w_type)) +
                        align256((size_t)(prec_planes(prec) * M * K * prec_elsize(prec)));
    if (need > (size_t)SPLITEE_NOALLOC_SCRATCH_BYTES) return SPLITEE_ERR_SCRATCH;
    void* ws = scratch_for_current_device();
    if (!ws) return SPLITEE_ERR_HIP;
    hipStream_t s = as_stream(stream);
    // the previous call on this device left the counters zeroed; clear them anyway, so that
    // the call does not depend on that (the mask kernel of the two-launch path clears them
    // too, the decode path with a precomputed mask has no such launch)
    const int64_t nc = (int64_t)(gemm_counters(M, N, K, prec, w_type) / 4);
    if (nc > 0) {
        const int64_t blocks = (nc + 255) / 256 < 1024 ? (nc + 255) / 256 : 1024;
        hipLaunchKernelGGL(zero_words_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                           reinterpret_cast<unsigned*>(ws), nc);
        if (hipGetLastError() != hipSuccess) return SPLITEE_ERR_HIP;
    }
    return run_masked(X, ldx, W, w_type, ldw, C, ldc, Y, ldy, M, N, K, mech, sensitivity, epsilon, seed, stream_id,
                      row0, eta_override, prec, ws, (size_t)SPLITEE_NOALLOC_SCRATCH_BYTES, s);
}

int splitee_correction(float* C, int64_t ldc, const void* W, int w_type, int64_t ldw, int64_t M,
                       int64_t N, int64_t K, int mech, double sensitivity, double epsilon,
                       uint64_t seed, uint64_t stream_id, uint64_t row0, int prec, void* workspace,
                       size_t workspace_bytes, void* stream)
{
    int rc = check_noise_args(mech, sensitivity, epsilon);
    if (rc) return rc;
    if (prec == SPLITEE_PREC_BF16 || !valid_prec(prec)) return SPLITEE_ERR_UNSUPPORTED;
    if (!dims_ok(M, N, K) || K % 8 != 0 || ldc < N) return SPLITEE_ERR_SHAPE;
    rc = check_w(W, w_type, ldw, K, prec);
    if (rc) return rc;
    if (M == 0 || N == 0) return SPLITEE_OK;
    if (!W || !C) return SPLITEE_ERR_ARG;
    if (!aligned16(C) || !pitch16(ldc, 4)) return SPLITEE_ERR_ALIGN;
    return run_masked(nullptr, K, W, w_type, ldw, nullptr, 0, C, ldc, M, N, K, mech, sensitivity,
                      epsilon, seed, stream_id, row0, nullptr, prec, workspace, workspace_bytes,
                      as_stream(stream));
}

int splitee_transform_probe(const uint32_t* words, int64_t n, int fn, int force_slow, float* out,
                            void* stream)
{
    if (fn < 0 || fn > 3 || n < 0) return SPLITEE_ERR_ARG;
    if (n == 0) return SPLITEE_OK;
    if (!words || !out) return SPLITEE_ERR_ARG;
    return splitee_host::launch_transform_probe(words, n, fn, force_slow, out, as_stream(stream));
}

size_t splitee_f64_workspace_bytes(int64_t M, int64_t N, int64_t K)
{
    if (!dims_ok(M, N, K) || K % 8 != 0) return 0;
    return f64_ws(M, N, K);
}

int splitee_masked_linear_fused_f64(const float* X, int64_t ldx, const void* W, int w_type, int64_t ldw,
                                    const double* C, int64_t ldc, float* Y, int64_t ldy, int64_t M, int64_t N,
                                    int64_t K, int mech, double sensitivity, double epsilon, uint64_t seed,
                                    uint64_t stream_id, uint64_t row0, void* workspace, size_t workspace_bytes,
                                    void* stream)
{
    int rc = check_noise_args(mech, sensitivity, epsilon);
    if (rc) return rc;
    if (!dims_ok(M, N, K) || K % 8 != 0 || ldx < K || ldc < N || ldy < N) return SPLITEE_ERR_SHAPE;
    rc = check_w_f64(W, w_type, ldw, K);
    if (rc) return rc;
    if (M == 0 || N == 0) return SPLITEE_OK;
    if (!X || !W || !C || !Y) return SPLITEE_ERR_ARG;
    if (!aligned16(X) || !pitch16(ldx, 4) || !aligned16(C) || !aligned16(Y)) return SPLITEE_ERR_ALIGN;
    return run_f64(X, ldx, W, w_type, ldw, C, ldc, Y, false, ldy, M, N, K, mech, sensitivity, epsilon, seed,
                   stream_id, row0, workspace, workspace_bytes, as_stream(stream));
}

int splitee_correction_f64(double* C, int64_t ldc, const void* W, int w_type, int64_t ldw, int64_t M, int64_t N,
                           int64_t K, int mech, double sensitivity, double epsilon, uint64_t seed,
                           uint64_t stream_id, uint64_t row0, void* workspace, size_t workspace_bytes, void* stream)
{
    int rc = check_noise_args(mech, sensitivity, epsilon);
    if (rc) return rc;
    if (!dims_ok(M, N, K) || K % 8 != 0 || ldc < N) return SPLITEE_ERR_SHAPE;
    rc = check_w_f64(W, w_type, ldw, K);
    if (rc) return rc;
    if (M == 0 || N == 0) return SPLITEE_OK;
    if (!W || !C) return SPLITEE_ERR_ARG;
    if (!aligned16(C)) return SPLITEE_ERR_ALIGN;
    return run_f64(nullptr, K, W, w_type, ldw, nullptr, 0, C, true, ldc, M, N, K, mech, sensitivity, epsilon,
                   seed, stream_id, row0, workspace, workspace_bytes, as_stream(stream));
}

size_t splitee_spectral_norm_workspace_bytes(int64_t N, int64_t K, int iters)
{
    if (!dims_ok(0, N, K) || iters < 1 || iters > MAX_POWER_ITERS || K > splitee_host::spectral_max_k()) return 0;
    return splitee_host::spectral_workspace_bytes(N, K, iters);
}

int splitee_spectral_norm(const void* W, int w_type, int64_t ldw, int64_t N, int64_t K, int iters,
                          uint64_t seed, uint64_t stream_id, double* sigma, double* history,
                          void* workspace, size_t workspace_bytes, void* stream)
{
    if (!valid_dtype(w_type)) return SPLITEE_ERR_DTYPE;
    if (w_type == SPLITEE_BF16_TILED) return SPLITEE_ERR_UNSUPPORTED;
    if (iters < 1 || iters > MAX_POWER_ITERS || !sigma) return SPLITEE_ERR_ARG;
    if (!dims_ok(0, N, K) || K % 8 != 0 || ldw < K) return SPLITEE_ERR_SHAPE;
    if (K > splitee_host::spectral_max_k()) return SPLITEE_ERR_UNSUPPORTED;
    if (N == 0 || K == 0) {
        *sigma = 0.0;
        if (history)
            for (int i = 0; i < iters; ++i) history[i] = 0.0;
        return SPLITEE_OK;
    }
    if (!W) return SPLITEE_ERR_ARG;
    if (!aligned16(W) || !pitch16(ldw, w_type == SPLITEE_F32 ? 4 : 2)) return SPLITEE_ERR_ALIGN;
    if (!workspace || workspace_bytes < splitee_host::spectral_workspace_bytes(N, K, iters))
        return SPLITEE_ERR_WORKSPACE;
    if (reinterpret_cast<uintptr_t>(workspace) & 255u) return SPLITEE_ERR_ALIGN;
    return splitee_host::launch_spectral_norm(W, w_type, ldw, N, K, iters, seed, stream_id, sigma, history,
                                              workspace, as_stream(stream));
}

size_t splitee_sensitivity_workspace_bytes(void) { return 256; }

int splitee_sensitivity(int bound, int64_t d, const float* alpha, const float* beta, double w_norm_a,
                        double w_norm_b, double* delta, void* workspace, size_t workspace_bytes,
                        void* stream)
{
    if (bound != SPLITEE_BOUND_LN && bound != SPLITEE_BOUND_ATT && bound != SPLITEE_BOUND_ACT)
        return SPLITEE_ERR_ARG;
    if (d < 1 || d > MAX_DIM) return SPLITEE_ERR_SHAPE;
    if (!alpha || !delta) return SPLITEE_ERR_ARG;
    const bool uses_a = bound != SPLITEE_BOUND_LN, uses_b = bound == SPLITEE_BOUND_ACT;
    if (uses_a && !(w_norm_a >= 0.0 && isfinite(w_norm_a))) return SPLITEE_ERR_ARG;
    if (uses_b && !(w_norm_b >= 0.0 && isfinite(w_norm_b))) return SPLITEE_ERR_ARG;
    if (!workspace || workspace_bytes < splitee_sensitivity_workspace_bytes()) return SPLITEE_ERR_WORKSPACE;
    if (reinterpret_cast<uintptr_t>(workspace) & 255u) return SPLITEE_ERR_ALIGN;
    double sums[2];
    const int rc = splitee_host::launch_vec_norms(alpha, uses_b ? beta : nullptr, d,
                                                  reinterpret_cast<double*>(workspace), sums, as_stream(stream));
    if (rc) return rc;
    const double n4 = pow(sums[0], 0.25), b2 = sqrt(sums[1]), sd = sqrt((double)d);
    if (bound == SPLITEE_BOUND_LN)
        *delta = 2.0 * sd * n4;  // Theorem 1
    else if (bound == SPLITEE_BOUND_ATT)
        *delta = 2.0 * sd * w_norm_a * n4;  // Theorem 2
    else {
        const double t = sd * n4 + b2;  // Theorem 3
        *delta = 2.0 * sd * (t * t) * w_norm_a * w_norm_b;
    }
    return SPLITEE_OK;
}

int splitee_eps_per_token(double eps_total, int64_t n, double* eps)
{
    if (!(eps_total > 0.0) || !isfinite(eps_total) || n < 1 || !eps) return SPLITEE_ERR_ARG;
    *eps = eps_total / sqrt((double)n);
    return SPLITEE_OK;
}

}  // extern "C"
