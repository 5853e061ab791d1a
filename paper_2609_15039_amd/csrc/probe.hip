// Matrix-core rounding probe (test hook, include/splitee_probe.h): one wavefront
// runs a chain of MFMA instructions of the kinds the GEMM kernels issue, on
// operands whose rows (A) and columns (B) are all equal, so that every element of
// the output tile holds the same rounded sum.  The operand lane layouts are those
// the GEMM kernels use:
//   v_mfma_f32_32x32x16_bf16  lane l: row / column l % 32, k = 8 (l / 32) + j, j < 8
//   v_mfma_f32_16x16x32_bf16  lane l: row / column l % 16, k = 8 (l / 16) + j, j < 8
//   v_mfma_f32_16x16x4_f32    lane l: row / column l % 16, k = l / 16
//   v_mfma_f64_16x16x4_f64    lane l: row / column l % 16, k = l / 16
#include "common.hpp"
#include "splitee_probe.h"

typedef double f64x4_t __attribute__((ext_vector_type(4)));

namespace {

constexpr int PROBE_MAX_N = 64;

template <int OP>
__global__ void __launch_bounds__(64) mfma_probe_kernel(const double* __restrict__ a, const double* __restrict__ b,
                                                        double c, int n, double* __restrict__ d)
{
    const int l = threadIdx.x;
    if constexpr (OP == 0) {
        f32x16_t acc;
        for (int e = 0; e < 16; ++e) acc[e] = (float)c;
        for (int i = 0; i < n; ++i) {
            bf16x8_t av, bv;
            for (int j = 0; j < 8; ++j) {
                const int k = 8 * (l / 32) + j;
                av[j] = (__bf16)(float)a[i * 16 + k];
                bv[j] = (__bf16)(float)b[i * 16 + k];
            }
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc, 0, 0, 0);
        }
        for (int e = 0; e < 16; ++e) d[l * 16 + e] = (double)acc[e];
    } else if constexpr (OP == 1) {
        f32x4_t acc;
        for (int e = 0; e < 4; ++e) acc[e] = (float)c;
        for (int i = 0; i < n; ++i) {
            bf16x8_t av, bv;
            for (int j = 0; j < 8; ++j) {
                const int k = 8 * (l / 16) + j;
                av[j] = (__bf16)(float)a[i * 32 + k];
                bv[j] = (__bf16)(float)b[i * 32 + k];
            }
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc, 0, 0, 0);
        }
        for (int e = 0; e < 4; ++e) d[l * 4 + e] = (double)acc[e];
    } else if constexpr (OP == 2) {
        f32x4_t acc;
        for (int e = 0; e < 4; ++e) acc[e] = (float)c;
        for (int i = 0; i < n; ++i) {
            const int k = l / 16;
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32((float)a[i * 4 + k], (float)b[i * 4 + k], acc, 0, 0, 0);
        }
        for (int e = 0; e < 4; ++e) d[l * 4 + e] = (double)acc[e];
    } else {
        f64x4_t acc;
        for (int e = 0; e < 4; ++e) acc[e] = c;
        for (int i = 0; i < n; ++i) {
            const int k = l / 16;
            acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i * 4 + k], b[i * 4 + k], acc, 0, 0, 0);
        }
        for (int e = 0; e < 4; ++e) d[l * 4 + e] = acc[e];
    }
}

}  // namespace

extern "C" int splitee_mfma_probe(int op, int n, const double* a, const double* b, double c, double* d,
                                  void* stream)
{
    if (op < 0 || op > 3 || n < 1 || n > PROBE_MAX_N || !a || !b || !d) return SPLITEE_ERR_ARG;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    switch (op) {
    case 0: hipLaunchKernelGGL(mfma_probe_kernel<0>, dim3(1), dim3(64), 0, s, a, b, c, n, d); break;
    case 1: hipLaunchKernelGGL(mfma_probe_kernel<1>, dim3(1), dim3(64), 0, s, a, b, c, n, d); break;
    case 2: hipLaunchKernelGGL(mfma_probe_kernel<2>, dim3(1), dim3(64), 0, s, a, b, c, n, d); break;
    default: hipLaunchKernelGGL(mfma_probe_kernel<3>, dim3(1), dim3(64), 0, s, a, b, c, n, d); break;
    }
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}
