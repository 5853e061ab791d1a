/*
 * splitee.h -- C ABI of the MI355X (gfx950) DP-masked linear layer.
 *
 * The method (SpliTEE, Sec. "Offloading Linear Operations", Eq.
 * add-and-then-subtract): to offload y = W x, the trusted side draws a mask eta,
 * sends x + eta, the GPU returns r = W (x + eta), and the trusted side recovers
 * W x = r - W eta with the correction W eta computed in advance (Sec.
 * "Precomputing the Mask and Noise Correction").  The mask is differentially
 * private noise of scale Delta/eps (Prop. 2; Sec. "Making the Process
 * Differentially Private"); Delta is the global l2-sensitivity of the function
 * producing x (Def. 2, Thms 1-3).
 *
 * Row-major conventions for every entry point (all sizes in elements):
 *   X    M x K float32, leading dimension ldx  -- tokens x in-features
 *   eta  M x K float32 (same shape as X)
 *   W    N x K, float32 or bfloat16, ldw       -- out x in (the paper's d' x d
 *                                                 matrix acting on column vectors),
 *        or bfloat16 in the tiled order below (SPLITEE_BF16_TILED; ldw unused)
 *   R, C, Y  M x N float32                     -- Y = X W^T
 *
 * Ownership: every pointer is a device pointer owned by the caller; the library
 * allocates no device memory.  Scratch space is passed in as `workspace`, sized by
 * the matching *_workspace_bytes query.
 *
 * Asynchrony: work is enqueued on `stream` (a hipStream_t; NULL = the default
 * stream) and the call returns after the launch.  SPLITEE_ERR_HIP reports a
 * failed launch; faults during execution surface at the caller's synchronize.
 *
 * Validation (synchronous; nothing is launched on error):
 *   eps finite and > 0, Delta finite and >= 0, mechanism known  -> SPLITEE_ERR_ARG
 *   M, N, K >= 0, ld >= row width, K % 4 == 0 (noise, mask) or
 *   K % 8 == 0 (GEMM entry points)                                -> SPLITEE_ERR_SHAPE
 *   16-byte aligned base pointers and 16-byte row pitches        -> SPLITEE_ERR_ALIGN
 *   unsupported dtype / precision pair                            -> SPLITEE_ERR_UNSUPPORTED
 *   null pointer where data is required                           -> SPLITEE_ERR_ARG
 *   workspace too small                                           -> SPLITEE_ERR_WORKSPACE
 * M == 0 or N == 0 is a valid empty call that launches nothing.
 *
 * Noise stream (the paper fixes the law but names no generator; this is the
 * library's definition, a pure function of its arguments, with no hidden state):
 *   element (i, k), absolute index e = (row0 + i) K + k, block b = e / 4,
 *   lane = e % 4; (w0..w3) = Philox4x32-10(counter = (b_lo, b_hi, sid_lo, sid_hi),
 *   key = (seed_lo, seed_hi)) [Salmon et al., SC'11]; u(w) = (w + 1/2) 2^-32;
 *   s = fl64(Delta / eps);
 *   LAPLACE:  eta = RN32(fl64(s * RN32(F^-1(u(w_lane))))), F^-1(u) = ln 2u (u < 1/2),
 *             -ln(2 - 2u) (u >= 1/2);
 *   GAUSSIAN: pairs (w0,w1) -> lanes 0,1 and (w2,w3) -> lanes 2,3 (Box-Muller):
 *             r = RN32(sqrt(-2 ln u(w_a))), c = RN32(cos 2 pi u(w_b)), sn = RN32(sin 2 pi u(w_b)),
 *             eta = RN32(fl64(s * (r * c))) on even lanes, RN32(fl64(s * (r * sn))) on odd;
 *   NONE:     eta = 0 (the split without noise).
 * RN32 is the correctly rounded binary32 value.  Single use of a mask
 * (Sec. "Precomputing the Mask and Noise Correction") is the caller's duty: never
 * reissue the same (seed, stream_id, row).
 *
 * Precision modes of the GEMM operand built from Xt = fl32(X + eta):
 *   SPLITEE_PREC_F32    Xt as float32, binary32 MFMA (bfloat16 W widened exactly).
 *   SPLITEE_PREC_BF16   Xt rounded once to bfloat16 (single pass; adds u_bf16 * sum|w||Xt|).
 *   SPLITEE_PREC_BF16X3 Xt = hi + mid + lo as three bfloat16 terms (exact), three
 *                       bfloat16 MFMA passes into one float32 accumulator; needs bf16 W.
 * BF16 and BF16X3 planes are stored one after another, plane p at
 * Xt + p * M * ldxt elements.
 *
 * Thread safety: the functions are stateless and reentrant.  Calls that share a
 * workspace must not overlap in time.
 *
 * Trust note: the fused call and splitee_correction place eta on the GPU.  That is
 * the one-GPU benchmark arrangement; in the paper's deployment only the GEMM of
 * the masked input (splitee_masked_linear) runs on the untrusted device and the
 * correction is computed inside the TEE.
 */
#ifndef SPLITEE_H
#define SPLITEE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPLITEE_ABI_VERSION 2

typedef enum {
    SPLITEE_OK = 0,
    SPLITEE_ERR_ARG = -1,
    SPLITEE_ERR_SHAPE = -2,
    SPLITEE_ERR_DTYPE = -3,
    SPLITEE_ERR_ALIGN = -4,
    SPLITEE_ERR_UNSUPPORTED = -5,
    SPLITEE_ERR_HIP = -6,
    SPLITEE_ERR_WORKSPACE = -7,
    SPLITEE_ERR_IO = -8,
    SPLITEE_ERR_EXHAUSTED = -9,
    SPLITEE_ERR_FORMAT = -10,
    SPLITEE_ERR_BUSY = -11,
    SPLITEE_ERR_SCRATCH = -12
} splitee_status;

typedef enum { SPLITEE_MECH_LAPLACE = 0, SPLITEE_MECH_GAUSSIAN = 1, SPLITEE_MECH_NONE = 2 } splitee_mech;
typedef enum { SPLITEE_F32 = 0, SPLITEE_BF16 = 1, SPLITEE_BF16_TILED = 2 } splitee_dtype;
typedef enum {
    SPLITEE_PREC_F32 = 0,
    SPLITEE_PREC_BF16 = 1,
    SPLITEE_PREC_BF16X3 = 2,
    SPLITEE_PREC_F64 = 3 /* binary64 mask, GEMM and correction: only the *_f64 entry points */
} splitee_prec;

/* Version of this ABI (SPLITEE_ABI_VERSION). */
int splitee_abi_version(void);

/* Static text for a status code. */
const char* splitee_status_string(int status);

/*
 * Noise eta (the mask; Prop. 2, Sec. "Making the Process Differentially Private").
 *   eta       out, M x K float32, leading dimension ld_eta (>= K, multiple of 4)
 *   mech      splitee_mech; sensitivity = Delta >= 0; epsilon > 0
 *   seed, stream_id, row0   select the counter block (see "Noise stream" above)
 * Requires K % 4 == 0.
 */
int splitee_noise_gen(float* eta, int64_t ld_eta, int64_t M, int64_t K, int mech,
                      double sensitivity, double epsilon, uint64_t seed, uint64_t stream_id,
                      uint64_t row0, void* stream);

/*
 * Several noise blocks in one launch: block (q, r), q < count, r < reps, is what
 * splitee_noise_gen(eta[q] + r * rep_stride[q], ld_eta[q], M, K[q], mech, sensitivity,
 * epsilon, seed, stream_id[q] + r * rep_sid_step, row0, stream) writes, element for
 * element.  The blocks share M, the mechanism, seed and row0; each q has its own K,
 * leading dimension, stream id and repetition stride, and repetition r steps
 * block q's output by rep_stride[q] elements and its stream id by rep_sid_step.  This is the
 * precomputation of the masks (Sec. "Precomputing the Mask and Noise Correction"):
 * one launch draws the masks of all projections of a layer, or of all layers
 * (r = layer) for one decode step.
 *   eta, ld_eta, K, stream_id   host arrays of `count` entries (0 <= count <= 8);
 *                               eta[q] a device pointer, 16-byte aligned, ld_eta[q]
 *                               >= K[q], a multiple of 4
 *   reps                        0 <= reps <= 65535 (count or reps 0: nothing to do)
 *   rep_stride                  host array of `count` strides in elements, >= 0 and a
 *                               multiple of 4 (may be NULL when reps <= 1)
 * Requires K[q] % 4 == 0.  The host arrays are read during the call only.  Blocks
 * must not overlap in memory.
 */
int splitee_noise_gen_multi(float* const* eta, const int64_t* ld_eta, const int64_t* K,
                            const uint64_t* stream_id, int count, int reps, const int64_t* rep_stride,
                            uint64_t rep_sid_step, int64_t M, int mech, double sensitivity,
                            double epsilon, uint64_t seed, uint64_t row0, void* stream);

/*
 * Mask: Xt = fl32(X + eta) (the vector addition of Sec. "Offloading Linear
 * Operations"), written in precision out_prec:
 *   F32: float32 M x K (ldxt); BF16: one bfloat16 plane; BF16X3: three bfloat16
 *   planes hi, mid, lo (plane p at Xt + p * M * ldxt); F64: binary64 M x K holding
 *   fl64(X + eta) instead (the operand of the *_f64 entry points).
 *   X may be NULL, meaning X = 0 (used to split eta for the correction).
 * Requires K % 4 == 0; ldxt a multiple of 8 for bfloat16 output, of 4 for float32,
 * of 2 for binary64.
 */
int splitee_mask(const float* X, int64_t ldx, const float* eta, int64_t ld_eta, void* Xt,
                 int out_prec, int64_t ldxt, int64_t M, int64_t K, void* stream);

/*
 * Noise and mask in one pass: Xt = fl32(X + eta) with eta generated in-kernel from
 * (mech, Delta, eps, seed, stream_id, row0) exactly as splitee_noise_gen would
 * produce it; eta itself is never stored.  Output layout as in splitee_mask.
 * X may be NULL (Xt = eta, as needed for the correction).  Requires K % 4 == 0.
 * This is the first half of splitee_masked_linear_fused.
 */
int splitee_noise_mask(const float* X, int64_t ldx, void* Xt, int out_prec, int64_t ldxt, int64_t M,
                       int64_t K, int mech, double sensitivity, double epsilon, uint64_t seed,
                       uint64_t stream_id, uint64_t row0, void* stream);

/*
 * Tiled weight order (SPLITEE_BF16_TILED).  The projection weights are fixed for
 * the life of a model, so they can be stored once in the order the MFMA kernels
 * load them: every 16-byte load of a wavefront then covers whole 128-byte cache
 * lines (row-major W gives 32 rows x 32 bytes per load, a quarter of the vector L1
 * bandwidth).  With N32 = ceil(N / 32) 32-row blocks and KT = ceil(K / 64) 64-wide k
 * tiles, bfloat16 element W[n][k] sits at element index
 *     ((((n / 32) KT + k / 64) 4 + (k % 64) / 16) 64 + ((k % 16) / 8) 32 + n % 32) 8 + k % 8
 * of an N32 x KT x 4096-byte buffer; rows n >= N and columns k >= K are zeros.
 * Accepted by splitee_masked_linear, splitee_masked_linear_unmask,
 * splitee_masked_linear_fused and splitee_correction with BF16 / BF16X3 precision
 * (SPLITEE_ERR_UNSUPPORTED with F32, in the binary64 calls and splitee_spectral_norm);
 * the result equals the row-major call's within the same error bounds (the kernels
 * and their K splits differ, so the summation order may too).
 */
size_t splitee_tiled_weights_bytes(int64_t N, int64_t K); /* 0 on invalid N, K (K % 8 != 0) */

/*
 * Writes W (N x K bfloat16, row-major, ldw >= K, 16-byte aligned rows) into Wt in
 * the tiled order, splitee_tiled_weights_bytes(N, K) bytes (caller-owned, 16-byte
 * aligned, must not overlap W: SPLITEE_ERR_ARG).  Requires K % 8 == 0.  A copy:
 * every byte of W reaches Wt unchanged.
 */
int splitee_tile_weights(const void* W, int64_t ldw, int64_t N, int64_t K, void* Wt, void* stream);

/*
 * The GPU's part of the method: R = Xt W^T (r = W (x + eta), Sec. "Offloading
 * Linear Operations"), with float32 accumulation.
 *   Xt     in_prec operand as written by splitee_mask (ldxt)
 *   W      N x K, w_type float32, bfloat16 (ldw) or tiled bfloat16; BF16 / BF16X3 need
 *          bfloat16 W, F32 takes row-major W
 *   R      out, M x N float32 (ldr)
 * Requires K % 8 == 0.  Needs no workspace (single-pass K reduction per tile).
 */
int splitee_masked_linear(const void* Xt, int in_prec, int64_t ldxt, const void* W, int w_type,
                          int64_t ldw, float* R, int64_t ldr, int64_t M, int64_t N, int64_t K,
                          void* stream);

/*
 * Unmask: Y = fl32(R - C) (Eq. add-and-then-subtract), C the correction eta W^T.
 * Requires 16-byte aligned rows.
 */
int splitee_unmask(const float* R, int64_t ldr, const float* C, int64_t ldc, float* Y, int64_t ldy,
                   int64_t M, int64_t N, void* stream);

/* Workspace bytes needed by splitee_masked_linear_unmask for this shape and
 * precision (split-K counters and partial tiles), enough for either weight
 * layout; 0 when none is needed. */
size_t splitee_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int prec);

/*
 * GEMM with the unmask epilogue: Y = fl32(fl(Xt W^T) - C) (C NULL: Y = R), the
 * second half of splitee_masked_linear_fused.  Xt as written by splitee_mask or
 * splitee_noise_mask (ldxt, planes M * ldxt apart).  Small tile counts are split
 * over K; the partial tiles are summed in split order (by a second kernel, or by
 * the last workgroup of each tile), so results are deterministic.  workspace: >=
 * splitee_gemm_workspace_bytes bytes, 256-byte aligned, zero-filled before its
 * first use (calls leave it zeroed).  Requires K % 8 == 0.
 */
int splitee_masked_linear_unmask(const void* Xt, int in_prec, int64_t ldxt, const void* W,
                                 int w_type, int64_t ldw, const float* C, int64_t ldc, float* Y,
                                 int64_t ldy, int64_t M, int64_t N, int64_t K, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* Workspace bytes needed by splitee_masked_linear_fused (and splitee_correction)
 * for this shape and precision, enough for either weight layout; 0 on invalid
 * arguments. */
size_t splitee_fused_workspace_bytes(int64_t M, int64_t N, int64_t K, int prec);

/*
 * Fused mask -> GEMM -> unmask for one projection: Y = fl32(fl(Xt W^T) - C) with
 * Xt = fl32(X + eta), eta generated in-stream from (mech, Delta, eps, seed,
 * stream_id, row0) -- or taken from eta_override when it is not NULL: a precomputed
 * mask (splitee_noise_gen / splitee_noise_gen_multi, Sec. "Precomputing the Mask
 * and Noise Correction"), M x K float32, leading dimension K, 16-byte aligned; the
 * noise arguments are then only validated.  C (M x N, ldc) must be the correction
 * of the same mask, e.g. from splitee_correction with the same noise arguments; for
 * a decode step at positions [t, t+M) pass row0 = t and C = bank + t * ldc.
 * M <= 16 with BF16 or BF16X3 takes the bandwidth-bound decode kernels (M <= 2: a
 * vector-ALU GEMV, on whole rows of row-major W or 32-row blocks of tiled W; else
 * the skinny MFMA kernel); given eta_override they form fl32(X + eta) and its
 * bfloat16 planes themselves (one launch, bit-identical to the two-launch path).  Otherwise the tiled
 * or W-streamed MFMA kernel runs, split over K when the tile count is small; for
 * 17 <= M <= 128 on tiled W given eta_override, the streamed kernel too forms the masked
 * input itself (bit-identical to the mask launch followed by the GEMM).
 * workspace: >= splitee_fused_workspace_bytes(M, N, K, prec) bytes, 256-byte
 * aligned; it must hold zeros before its first use and calls leave it that way.
 */
int splitee_masked_linear_fused(const float* X, int64_t ldx, const void* W, int w_type, int64_t ldw,
                                const float* C, int64_t ldc, float* Y, int64_t ldy, int64_t M,
                                int64_t N, int64_t K, int mech, double sensitivity, double epsilon,
                                uint64_t seed, uint64_t stream_id, uint64_t row0,
                                const float* eta_override, int prec, void* workspace,
                                size_t workspace_bytes, void* stream);

/*
 * splitee_masked_linear_fused without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation.  Arguments, results and validation are those of
 * splitee_masked_linear_fused (the same kernels run, so Y is bit-identical to that
 * call's); its scratch space (split-K counters and partial tiles, the masked-input
 * planes) is instead a static device buffer of SPLITEE_NOALLOC_SCRATCH_BYTES that the
 * library holds on each GPU it runs on until the process ends.  The call allocates
 * nothing: on its first use on a device it looks up that device's copy of the buffer,
 * and it clears the split-K counters on `stream` itself.
 *   SPLITEE_ERR_SCRATCH   the shape needs more scratch than the buffer holds (the
 *                         workspace splitee_fused_workspace_bytes would ask for, roughly
 *                         M K 6 bytes for BF16X3 plus the split-K partials): use
 *                         splitee_masked_linear_fused with a caller-owned workspace
 *   SPLITEE_ERR_HIP       the buffer could not be resolved on the current device
 * Every call on one GPU uses the same buffer: calls that overlap in time on one GPU
 * (different streams, or host threads) race and give wrong results; serialise them.
 */
#define SPLITEE_NOALLOC_SCRATCH_BYTES (64u << 20)
int splitee_masked_linear_fused_noalloc(const float* X, int64_t ldx, const void* W, int w_type, int64_t ldw,
                                        const float* C, int64_t ldc, float* Y, int64_t ldy, int64_t M, int64_t N,
                                        int64_t K, int mech, double sensitivity, double epsilon, uint64_t seed,
                                        uint64_t stream_id, uint64_t row0, const float* eta_override, int prec,
                                        void* stream);

/*
 * Correction C = eta W^T (Sec. "Precomputing the Mask and Noise Correction"),
 * computed in F32 or BF16X3 (single-pass BF16 would round eta and break the
 * cancellation: SPLITEE_ERR_UNSUPPORTED).  Noise arguments as in the fused call.
 * In the paper this runs offline inside the TEE.
 */
int splitee_correction(float* C, int64_t ldc, const void* W, int w_type, int64_t ldw, int64_t M,
                       int64_t N, int64_t K, int mech, double sensitivity, double epsilon,
                       uint64_t seed, uint64_t stream_id, uint64_t row0, int prec, void* workspace,
                       size_t workspace_bytes, void* stream);

/*
 * Binary64 variant of the fused call and the correction (SPLITEE_PREC_F64): for a
 * projection whose noise scale is too large for binary32 cancellation, as for the Down
 * projection under Theorem 3 (Sec. "The Case Against the Down Linear Projection": with
 * the unit roundoff of binary64 the error bound of Theorem 4 shrinks by about 2^29).
 *   Xt = fl64(X + eta) with eta the binary32 noise of splitee_noise_gen (the sum is exact
 *   while |X| and |eta| are within a factor 2^29); R = Xt W^T accumulated in binary64
 *   (W bfloat16 or float32, exact in binary64); Y = fl32(R - C).
 *   C          M x N binary64 correction from splitee_correction_f64 with the same noise
 *              arguments, leading dimension ldc >= N, 16-byte aligned
 *   X, Y       as in splitee_masked_linear_fused (float32)
 *   workspace  >= splitee_f64_workspace_bytes(M, N, K) bytes, 256-byte aligned, no
 *              initial contents needed (the binary64 Xt and, for small tile counts, the
 *              split-K partials)
 * Requires K % 8 == 0.
 */
size_t splitee_f64_workspace_bytes(int64_t M, int64_t N, int64_t K);
int splitee_masked_linear_fused_f64(const float* X, int64_t ldx, const void* W, int w_type, int64_t ldw,
                                    const double* C, int64_t ldc, float* Y, int64_t ldy, int64_t M, int64_t N,
                                    int64_t K, int mech, double sensitivity, double epsilon, uint64_t seed,
                                    uint64_t stream_id, uint64_t row0, void* workspace, size_t workspace_bytes,
                                    void* stream);

/* C = eta W^T in binary64 (M x N, leading dimension ldc >= N, 16-byte aligned); noise
 * and W arguments as for splitee_masked_linear_fused_f64. */
int splitee_correction_f64(double* C, int64_t ldc, const void* W, int w_type, int64_t ldw, int64_t M, int64_t N,
                           int64_t K, int mech, double sensitivity, double epsilon, uint64_t seed,
                           uint64_t stream_id, uint64_t row0, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Noise scale (Prop. 2: the Gaussian mask has standard deviation Delta f / eps per
 * coordinate) from the global sensitivity bounds of Sec. "Global Sensitivity
 * Analysis".  d is the model width; alpha, beta the scale and shift of the layer
 * normalisation that precedes the bounded component.
 *   SPLITEE_BOUND_LN   Theorem 1: 2 sqrt(d) ||alpha||_4
 *                      (inputs of QKV, Gate / Up and the LM head)
 *   SPLITEE_BOUND_ATT  Theorem 2: 2 sqrt(d) ||W_val||_2 ||alpha||_4       (input of O)
 *   SPLITEE_BOUND_ACT  Theorem 3: 2 sqrt(d) (sqrt(d) ||alpha||_4 + ||beta||_2)^2
 *                      ||W_up||_2 ||W_gate||_2                          (input of Down)
 */
typedef enum { SPLITEE_BOUND_LN = 0, SPLITEE_BOUND_ATT = 1, SPLITEE_BOUND_ACT = 2 } splitee_bound;

/* Workspace bytes needed by splitee_spectral_norm for an N x K matrix and `iters`
 * rounds; 0 on invalid arguments. */
size_t splitee_spectral_norm_workspace_bytes(int64_t N, int64_t K, int iters);

/*
 * Spectral norm ||W||_2, the largest singular value (the matrix norm whose
 * consistency, Eq. matrix-norm, the proofs of Theorems 2 and 3 use), by the power
 * method on W^T W: from v_0 = g / ||g||, each round forms u = W v, sigma = ||u||,
 * z = W^T u and v = z / ||z||.  g is the standard Gaussian row 0 of noise stream
 * (seed, stream_id), i.e. what splitee_noise_gen(g, K, 1, K, SPLITEE_MECH_GAUSSIAN,
 * 1, 1, seed, stream_id, 0, stream) writes.  sigma never exceeds ||W||_2 in exact
 * arithmetic and rises towards it at a rate set by the gap between the two largest
 * singular values; the caller chooses iters.
 *   W          N x K, w_type (splitee_dtype), leading dimension ldw >= K, row-major,
 *              16-byte aligned with a 16-byte row pitch; read only
 *   N, K       N >= 0, 0 <= K <= 16384, K % 8 == 0 (K above 16384:
 *              SPLITEE_ERR_UNSUPPORTED); N == 0 or K == 0 gives sigma = 0 and launches
 *              nothing
 *   iters      1 <= iters <= 1048576
 *   sigma      host, receives sigma of the last round
 *   history    host array of iters entries or NULL; receives sigma of every round
 *   workspace  device, >= splitee_spectral_norm_workspace_bytes(N, K, iters) bytes,
 *              256-byte aligned; no initial contents needed
 * Products accumulate in float32, squared norms in binary64.  The call
 * synchronises `stream` before it returns.
 */
int splitee_spectral_norm(const void* W, int w_type, int64_t ldw, int64_t N, int64_t K, int iters,
                          uint64_t seed, uint64_t stream_id, double* sigma, double* history,
                          void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes needed by splitee_sensitivity. */
size_t splitee_sensitivity_workspace_bytes(void);

/*
 * Sensitivity bound Delta f of one component (splitee_bound above).
 *   d          model width, >= 1
 *   alpha      device, d float32 (the normalisation scale); required
 *   beta       device, d float32 (the normalisation shift) or NULL for beta = 0; read
 *              only by SPLITEE_BOUND_ACT
 *   w_norm_a   ||W_val||_2 (ATT) or ||W_up||_2 (ACT); unused for LN; finite, >= 0
 *   w_norm_b   ||W_gate||_2 (ACT); unused otherwise; finite, >= 0
 *   delta      host, receives the bound
 *   workspace  device, >= splitee_sensitivity_workspace_bytes() bytes, 256-byte aligned
 * The vector norms are reduced on the GPU in binary64 (sum of alpha^4, sum of beta^2);
 * the bound is assembled from them in binary64.  The call synchronises `stream`.
 */
int splitee_sensitivity(int bound, int64_t d, const float* alpha, const float* beta, double w_norm_a,
                        double w_norm_b, double* delta, void* workspace, size_t workspace_bytes,
                        void* stream);

/*
 * Per-token privacy budget: n releases that are each eps-GDP compose to
 * sqrt(n) eps-GDP (Prop. "Sequential Composition"), so a prompt of n tokens within a
 * total budget eps_total takes eps = eps_total / sqrt(n) per token (the EPN
 * configuration of the experiments).  eps_total > 0 and finite, n >= 1; *eps is written on
 * success.  Host only.
 */
int splitee_eps_per_token(double eps_total, int64_t n, double* eps);

/*
 * Noise bank (Sec. "Precomputing the Mask and Noise Correction"): the corrections
 * C = eta W^T of one projection group, precomputed for rows row0 .. row0 + rows - 1 of
 * one noise stream, stored in a file, loaded per batch and handed out exactly once.
 * The paper keeps a separate bank per offloaded component (QKV, O, Gate/Up, LM head)
 * and indexes it by the input shape; here a bank is one (stream_id, K, N) and
 * splitee_bank_path names its file in a bank directory.  The masks are not stored:
 * the fused call regenerates eta from (seed, stream_id, row), so a bank takes
 * rows x N x 4 bytes instead of rows x (K + N) x 4.
 *
 * A bank file has a 128-byte header (see csrc/bank.cpp) and rows x N float32.  Its
 * single-use watermark `consumed` is written to the file and synced before the
 * rows it covers are read; a row is never handed out twice, also across processes
 * (one open handle per file at a time: a second open gets SPLITEE_ERR_BUSY).  Rows
 * taken by a load that then fails are lost, not reissued.  Handles are not
 * thread-safe.
 */
typedef struct splitee_bank splitee_bank;

typedef struct {
    int64_t K, N;                 /* mask width, correction width */
    uint64_t seed, stream_id;     /* the noise stream */
    int32_t mech, prec;           /* splitee_mech; splitee_prec the corrections were computed in */
    double sensitivity, epsilon;  /* noise scale Delta / eps */
    int64_t row0, rows;           /* stream rows row0 .. row0 + rows - 1 are stored */
    int64_t consumed;             /* rows row0 .. row0 + consumed - 1 have been handed out */
    int64_t bytes_stored;         /* file size: header + rows x N float32 */
    int64_t bytes_with_masks;     /* the same bank storing the masks too: + rows x K float32 */
} splitee_bank_info_t;

/* Canonical file of the bank of (stream_id, K, N) in directory dir (the shape index):
 * "<dir>/bank-s<stream_id, 16 hex digits>-k<K>-n<N>.spb", written to out (out_len
 * bytes, NUL-terminated); SPLITEE_ERR_ARG if it does not fit. */
int splitee_bank_path(const char* dir, int64_t K, int64_t N, uint64_t stream_id, char* out, size_t out_len);

/* Device workspace bytes splitee_bank_create needs: the fused call's workspace for 256
 * rows plus a 256 x N float32 staging block; 0 on invalid arguments. */
size_t splitee_bank_workspace_bytes(int64_t K, int64_t N, int prec);

/*
 * Precompute and store a bank: C rows for stream rows row0 .. row0 + rows - 1, in
 * blocks of 256 rows, each exactly what splitee_correction(C, N, W, ..., block rows,
 * N, K, mech, sensitivity, epsilon, seed, stream_id, block row0, prec, ...) writes.
 *   path        new file; an existing file is never overwritten (SPLITEE_ERR_IO)
 *   W, w_type, ldw, K, N, mech, sensitivity, epsilon, seed, stream_id, prec
 *               as for splitee_correction (prec F32 or BF16X3); N % 4 == 0
 *   rows        >= 0 (0 writes an empty bank)
 *   workspace   device, >= splitee_bank_workspace_bytes(K, N, prec) bytes, 256-byte
 *               aligned, zeros at first use (left that way), as for the fused call
 * The header is written last; a failed call removes the file.  Synchronises `stream`.
 */
int splitee_bank_create(const char* path, const void* W, int w_type, int64_t ldw, int64_t K, int64_t N, int mech,
                        double sensitivity, double epsilon, uint64_t seed, uint64_t stream_id, uint64_t row0,
                        int64_t rows, int prec, void* workspace, size_t workspace_bytes, void* stream);

/* Open a bank file: SPLITEE_ERR_IO if it cannot be opened, SPLITEE_ERR_BUSY if another
 * handle holds it, SPLITEE_ERR_FORMAT if its header or size is inconsistent. */
int splitee_bank_open(const char* path, splitee_bank** bank);

/* The bank's parameters, watermark and storage accounting. Host only. */
int splitee_bank_info(const splitee_bank* bank, splitee_bank_info_t* info);

/*
 * Load the next `rows` rows not yet handed out into C (rows x N float32, leading
 * dimension ldc >= N; device memory if dst_device != 0, else host memory) and take
 * them: *row0 receives their first stream row, to be passed as row0 to the fused call
 * together with these C rows.  SPLITEE_ERR_EXHAUSTED if fewer rows remain (nothing
 * taken).  rows == 0 only reports the next row.  Synchronises `stream` for a device
 * destination, which goes through pinned host memory that the handle keeps (up to 256
 * rows) until it is closed.  Every load syncs the watermark to the file, so loading a
 * batch's rows at once costs far less than one load per decode step.
 */
int splitee_bank_load(splitee_bank* bank, int64_t rows, float* C, int64_t ldc, int dst_device, int64_t* row0,
                      void* stream);

/* Close the handle and free its pinned staging memory (the file and its watermark stay). */
int splitee_bank_close(splitee_bank* bank);

#ifdef __cplusplus
}
#endif

#endif /* SPLITEE_H */
