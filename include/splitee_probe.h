/*
 * splitee_probe.h -- test hooks of libsplitee.so (not part of the masked-linear path).
 *
 * These two entry points let the tests look at the arithmetic the kernels are built
 * on: the correctly rounded noise transforms, and the rounding of the matrix-core
 * (MFMA) instructions the GEMM kernels issue.  The error bounds that the tests
 * apply to the GEMM (the dot-product bound gamma_n of Def. 6 and Theorem 4) assume
 * that each floating-point operation rounds to nearest with unit roundoff u; the
 * MFMA probe lets a test check that assumption for each instruction on the device.
 * Conventions as in splitee.h: device pointers owned by the caller, work enqueued
 * on `stream`, synchronous argument checks.
 */
#ifndef SPLITEE_PROBE_H
#define SPLITEE_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Evaluates one correctly rounded noise transform on n words
 * (fn 0: Laplace inverse CDF, 1: sqrt(-2 ln u), 2: cos 2 pi u, 3: sin 2 pi u,
 * u = (w + 1/2) 2^-32; the definitions of splitee.h's noise stream).
 *   words   device, n uint32
 *   out     device, n float32
 * force_slow = 1 takes the double-double path for every word instead of only
 * for words whose binary64 value lies near a binary32 rounding boundary.
 * fn outside 0..3 or n < 0: SPLITEE_ERR_ARG; n == 0 launches nothing.
 */
int splitee_transform_probe(const uint32_t* words, int64_t n, int fn, int force_slow, float* out,
                            void* stream);

/*
 * Matrix-core rounding probe: one wavefront runs a chain of n instructions of one
 * MFMA kind, D_i = A_i B_i + D_{i-1} with D_0 = c in every element, where every row
 * of the A operand of instruction i holds a[i kb .. i kb + kb) and every column of
 * its B operand holds b[i kb .. i kb + kb) (kb = the instruction's k depth), so that
 * every element of the output tile receives the same value
 *     c + sum_i sum_k a[i kb + k] b[i kb + k]
 * rounded the way the hardware rounds it.
 *   op   0: v_mfma_f32_32x32x16_bf16 (kb 16, 32 x 32 tile; the W-streamed GEMM)
 *        1: v_mfma_f32_16x16x32_bf16 (kb 32, 16 x 16 tile; the skinny decode GEMM)
 *        2: v_mfma_f32_16x16x4_f32   (kb 4,  16 x 16 tile; the binary32 GEMM)
 *        3: v_mfma_f64_16x16x4_f64   (kb 4,  16 x 16 tile; the binary64 GEMM)
 *   n    1 <= n <= 64 instructions
 *   a, b device, n kb binary64 values each; they are converted to the instruction's
 *        operand type (bfloat16 or binary32 by round to nearest even, binary64 as is),
 *        so pass values that the operand type holds exactly
 *   c    the initial accumulator (rounded to binary32 for ops 0-2)
 *   d    device, receives every accumulator element of the final tile as binary64:
 *        lane l's element e at d[l * R + e], R = 16 (op 0) or 4 (ops 1-3), so 1024 or
 *        256 values
 * op outside 0..3, n outside 1..64 or a null pointer: SPLITEE_ERR_ARG.
 */
int splitee_mfma_probe(int op, int n, const double* a, const double* b, double c, double* d, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SPLITEE_PROBE_H */
