// Shared device/host helpers of the HIP library (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "splitee.h"

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

namespace splitee {

// most noise blocks one splitee_noise_gen_multi call generates
constexpr int NOISE_MULTI_MAX = 8;

// Bytes of a bfloat16 N x K weight matrix in the tiled order: 32-row blocks of
// 64-k tiles, 4 KB each, N padded to a multiple of 32 and K to a multiple of 64.
inline size_t tiled_weights_bytes(int64_t N, int64_t K)
{
    return (size_t)((N + 31) / 32) * (size_t)((K + 63) / 64) * 4096u;
}

// binary32 -> bfloat16 bits, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t bf16_bits_rne(float x)
{
    uint32_t b = __float_as_uint(x);
    if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu)) return (b >> 16) | 0x40u;
    return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// Split binary32 x into hi + mid + lo bfloat16 terms that sum to x exactly.
__device__ __forceinline__ void split3_bf16(float x, uint32_t& hi, uint32_t& mid, uint32_t& lo)
{
    hi = bf16_bits_rne(x);
    float r1 = x - bf16_bits_to_f32(hi);   // exact in binary32
    mid = bf16_bits_rne(r1);
    float r2 = r1 - bf16_bits_to_f32(mid); // exact in binary32
    lo = bf16_bits_rne(r2);                // exact: r2 has at most 8 significant bits
}

// RN bfloat16 bits of a (low half) and b (high half) by the hardware conversion
// (one v_cvt_pk_bf16_f32: round to nearest even, binary32 denormals kept); the same
// bits as bf16_bits_rne on every binary32 input, NaNs included (checked on all 2^32).
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16x2_rne(float a, float b)
{
    const f32x2_t v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// split3_bf16 of a pair: the hi, mid and lo terms of a in the low halves, of b in the
// high halves.
__device__ __forceinline__ void split3_bf16x2(float a, float b, uint32_t& hi, uint32_t& mid, uint32_t& lo)
{
    hi = bf16x2_rne(a, b);
    const float ra = a - __uint_as_float(hi << 16), rb = b - __uint_as_float(hi & 0xFFFF0000u);
    mid = bf16x2_rne(ra, rb);
    lo = bf16x2_rne(ra - __uint_as_float(mid << 16), rb - __uint_as_float(mid & 0xFFFF0000u));
}

// Workgroup-id remap so that consecutive logical tiles land on the same XCD.
// The dispatcher places workgroup b on XCD (b mod 8); tiles that share operands
// are given consecutive logical ids and thus share that XCD's L2.
__device__ __forceinline__ uint32_t xcd_logical_block(uint32_t b, uint32_t nblocks)
{
    const uint32_t nx = 8;
    uint32_t per = nblocks / nx;
    uint32_t full = per * nx;
    if (b >= full) return b;
    return (b % nx) * per + b / nx;
}

}  // namespace splitee

// host-side launch helpers implemented in the kernel translation units
namespace splitee_host {
int launch_noise(float* eta, int64_t ld_eta, int64_t M, int64_t K, int mech, double scale,
                 uint64_t seed, uint64_t sid, uint64_t row0, hipStream_t s);
int launch_noise_multi(float* const* eta, const int64_t* ld, const int64_t* K, const uint64_t* sid, int count,
                       int reps, const int64_t* rep_stride, uint64_t rep_sid_step, int64_t M, int mech,
                       double scale, uint64_t seed, uint64_t row0, hipStream_t s);
int launch_mask(const float* X, int64_t ldx, const float* eta, int64_t ld_eta, int gen_mech,
                double scale, uint64_t seed, uint64_t sid, uint64_t row0, void* Xt, int prec,
                int64_t ldxt, int64_t plane_stride, int64_t M, int64_t K,
                unsigned* zero_ptr, int64_t zero_count, hipStream_t s);
int launch_unmask(const float* R, int64_t ldr, const float* C, int64_t ldc, float* Y, int64_t ldy,
                  int64_t M, int64_t N, hipStream_t s);
int launch_transform_probe(const uint32_t* w, int64_t n, int fn, int force_slow, float* out,
                           hipStream_t s);
// Tiled MFMA GEMM: Out = A . W^T (- C if C != nullptr), A given as prec planes.
size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int prec, int w_type);
int launch_gemm(const void* A, int prec, int64_t lda, int64_t plane_stride, const void* W,
                int w_type, int64_t ldw, const float* C, int64_t ldc, float* Out, int64_t ldo,
                int64_t M, int64_t N, int64_t K, void* ws, size_t ws_bytes, hipStream_t s);
// Decode GEMM whose masked input fl32(X + eta) is formed in-kernel from X and a
// given mask eta (both M x K float32).
int launch_skinny_masked(const float* X, int64_t ldx, const float* eta, int64_t ld_eta, int prec,
                         const void* W, int w_type, int64_t ldw, const float* C, int64_t ldc, float* Out,
                         int64_t ldo, int64_t M, int64_t N, int64_t K, void* ws, size_t ws_bytes, hipStream_t s);
// The streamed GEMM with its masked input formed in-kernel the same way (64-row tiles on
// tiled W, M <= 128); SPLITEE_ERR_UNSUPPORTED where the plan has no such variant.
int launch_gemm_masked(const float* X, int64_t ldx, const float* eta, int64_t ld_eta, int prec, const void* W,
                       int w_type, const float* C, int64_t ldc, float* Out, int64_t ldo, int64_t M, int64_t N,
                       int64_t K, void* ws, size_t ws_bytes, hipStream_t s);
size_t skinny_workspace_bytes(int64_t M, int64_t N, int64_t K, int prec, int w_type);
int launch_skinny(const void* A, int prec, int64_t lda, int64_t plane_stride, const void* W, int w_type,
                  int64_t ldw, const float* C, int64_t ldc, float* Out, int64_t ldo, int64_t M,
                  int64_t N, int64_t K, void* ws, size_t ws_bytes, hipStream_t s);
// bfloat16 W (N x K, row-major) -> the tiled order (splitee_tile_weights).
int launch_tile_weights(const uint16_t* W, int64_t ldw, int64_t N, int64_t K, uint16_t* Wt, hipStream_t s);
// Binary64 GEMM Out = A W^T (- C), A binary64, W bf16 / f32, Out binary64 or rounded to binary32.
size_t f64_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);
int launch_gemm_f64(const double* A, int64_t lda, const void* W, int w_type, int64_t ldw, const double* C,
                    int64_t ldc, void* Out, bool out64, int64_t ldo, int64_t M, int64_t N, int64_t K, void* ws,
                    size_t ws_bytes, hipStream_t s);
// Power method for ||W||_2 and the vector norms of the sensitivity bounds.
size_t spectral_workspace_bytes(int64_t N, int64_t K, int iters);
int spectral_max_k();
int launch_spectral_norm(const void* W, int w_type, int64_t ldw, int64_t N, int64_t K, int iters, uint64_t seed,
                         uint64_t sid, double* sigma, double* history, void* ws, hipStream_t s);
int launch_vec_norms(const float* alpha, const float* beta, int64_t d, double* out_dev, double* out_host,
                     hipStream_t s);
}  // namespace splitee_host
