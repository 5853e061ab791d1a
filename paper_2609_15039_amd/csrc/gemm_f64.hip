// Binary64 GEMM for the masked projection whose noise is too large for binary32
// cancellation (the Down projection at the sensitivity of Theorem 3): Out = A W^T (- C)
// with A (the binary64 masked input, or the mask itself for the correction) M x K,
// W N x K bfloat16 or float32 converted exactly to binary64, C M x N binary64.
// v_mfma_f64_16x16x4_f64 on 64 x 64 output tiles: 4 waves of 32 x 32 (2 x 2 MFMA
// tiles), 16-deep K tiles double-buffered in LDS.  Split over K when the tile count is
// small; the splits' binary64 partials are summed in split order by a second kernel,
// which also subtracts C and rounds the output.
#include "common.hpp"

namespace {

typedef double f64x4 __attribute__((ext_vector_type(4)));

constexpr int F64_BM = 64, F64_BN = 64, F64_BK = 16;
constexpr int F64_NT = 256;
constexpr int F64_LDS_LD = F64_BK + 1;   // padded row: fragment reads of 16 rows hit distinct banks
constexpr int F64_TARGET_WGS = 512;      // two workgroups per CU
constexpr int F64_MIN_KT = 8;            // K tiles per split at least

// One K tile of A and W into registers: thread t takes row t / 4, k = 4 (t % 4) .. + 3 of
// both (zeros outside the matrices; K % 4 == 0 keeps each quad whole).
template <bool WBF16>
struct F64Stage {
    double a[4];
    double w[4];

    __device__ __forceinline__ void load(const double* __restrict__ A, int64_t lda, const void* __restrict__ W,
                                         int64_t ldw, int M, int N, int K, int m0, int n0, int k0, int tid)
    {
        const int r = tid >> 2, kq = k0 + 4 * (tid & 3);
        const bool kin = kq < K;
        if (kin && m0 + r < M) {
            const double* p = A + (int64_t)(m0 + r) * lda + kq;
            const double2 u = *reinterpret_cast<const double2*>(p);
            const double2 v = *reinterpret_cast<const double2*>(p + 2);
            a[0] = u.x; a[1] = u.y; a[2] = v.x; a[3] = v.y;
        } else {
            a[0] = a[1] = a[2] = a[3] = 0.0;
        }
        if (kin && n0 + r < N) {
            if (WBF16) {
                const uint2 q = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(W) +
                                                                (int64_t)(n0 + r) * ldw + kq);
                w[0] = (double)__uint_as_float(q.x << 16);
                w[1] = (double)__uint_as_float(q.x & 0xFFFF0000u);
                w[2] = (double)__uint_as_float(q.y << 16);
                w[3] = (double)__uint_as_float(q.y & 0xFFFF0000u);
            } else {
                const float4 q = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(W) +
                                                                  (int64_t)(n0 + r) * ldw + kq);
                w[0] = q.x; w[1] = q.y; w[2] = q.z; w[3] = q.w;
            }
        } else {
            w[0] = w[1] = w[2] = w[3] = 0.0;
        }
    }

    __device__ __forceinline__ void store(double (*As)[F64_LDS_LD], double (*Ws)[F64_LDS_LD], int tid) const
    {
        const int r = tid >> 2, kq = 4 * (tid & 3);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            As[r][kq + e] = a[e];
            Ws[r][kq + e] = w[e];
        }
    }
};

// Tile (blockIdx.x % tiles) over K tiles [split * ktps, ..) with split = blockIdx.x / tiles.
// ksplit == 1: Out = acc - C (C may be null), as binary64 (OUT64) or rounded to binary32.
// ksplit > 1: part[split][row][col] = acc (binary64), summed by f64_sum_kernel.
template <bool WBF16, bool OUT64>
__global__ void __launch_bounds__(F64_NT) gemm_f64_kernel(const double* __restrict__ A, int64_t lda,
                                                          const void* __restrict__ W, int64_t ldw,
                                                          const double* __restrict__ C, int64_t ldc,
                                                          void* __restrict__ Out, int64_t ldo,
                                                          double* __restrict__ part, int M, int N, int K,
                                                          int ntiles, int tiles, int ktps)
{
    __shared__ double As[2][F64_BM][F64_LDS_LD];
    __shared__ double Ws[2][F64_BN][F64_LDS_LD];
    const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
    const int wm = wave >> 1, wn = wave & 1;
    const int tile = blockIdx.x % tiles, split = blockIdx.x / tiles;
    const int m0 = (tile / ntiles) * F64_BM, n0 = (tile % ntiles) * F64_BN;
    const int ktiles = (K + F64_BK - 1) / F64_BK;
    const int kt0 = split * ktps, kt1 = min(ktiles, kt0 + ktps);

    f64x4 acc[2][2];
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int t = 0; t < 2; ++t) acc[s][t] = f64x4{0.0, 0.0, 0.0, 0.0};

    F64Stage<WBF16> st;
    if (kt0 < kt1) {
        st.load(A, lda, W, ldw, M, N, K, m0, n0, kt0 * F64_BK, tid);
        st.store(As[0], Ws[0], tid);
    }
    __syncthreads();
    const int fr = lane % 16, fk = lane / 16;
    for (int kt = kt0; kt < kt1; ++kt) {
        const int buf = (kt - kt0) & 1;
        const bool more = kt + 1 < kt1;
        if (more) st.load(A, lda, W, ldw, M, N, K, m0, n0, (kt + 1) * F64_BK, tid);
#pragma unroll
        for (int kk = 0; kk < F64_BK; kk += 4) {
            double a[2], b[2];
#pragma unroll
            for (int s = 0; s < 2; ++s) a[s] = As[buf][wm * 32 + s * 16 + fr][kk + fk];
#pragma unroll
            for (int t = 0; t < 2; ++t) b[t] = Ws[buf][wn * 32 + t * 16 + fr][kk + fk];
#pragma unroll
            for (int s = 0; s < 2; ++s)
#pragma unroll
                for (int t = 0; t < 2; ++t)
                    acc[s][t] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[s], b[t], acc[s][t], 0, 0, 0);
        }
        if (more) st.store(As[buf ^ 1], Ws[buf ^ 1], tid);
        __syncthreads();
    }

    // accumulator element e of lane l: row l / 16 + 4 e, column l % 16 of its 16 x 16 tile
    // (v_mfma_f64_16x16x4_f64 on gfx950, checked against a binary64 reference)
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int row = m0 + wm * 32 + s * 16 + fk + 4 * e;
                const int col = n0 + wn * 32 + t * 16 + fr;
                if (row >= M || col >= N) continue;
                const double v = acc[s][t][e];
                if (part) {
                    part[((int64_t)split * M + row) * N + col] = v;
                } else {
                    const double y = C ? v - C[(int64_t)row * ldc + col] : v;
                    if (OUT64)
                        reinterpret_cast<double*>(Out)[(int64_t)row * ldo + col] = y;
                    else
                        reinterpret_cast<float*>(Out)[(int64_t)row * ldo + col] = (float)y;
                }
            }
}

// Out[i][j] = sum over the splits in order of part[s][i][j], minus C[i][j] when C is given.
template <bool OUT64>
__global__ void __launch_bounds__(256) f64_sum_kernel(const double* __restrict__ part, int ksplit,
                                                      const double* __restrict__ C, int64_t ldc,
                                                      void* __restrict__ Out, int64_t ldo, int M, int N)
{
    const int64_t total = (int64_t)M * N;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = t / N, j = t - i * N;
        double v = part[t];
        for (int s = 1; s < ksplit; ++s) v += part[(int64_t)s * total + t];
        if (C) v -= C[i * ldc + j];
        if (OUT64)
            reinterpret_cast<double*>(Out)[i * ldo + j] = v;
        else
            reinterpret_cast<float*>(Out)[i * ldo + j] = (float)v;
    }
}

struct F64Plan {
    int ntiles, tiles, ksplit, ktps;
    size_t part_bytes;
};

F64Plan plan_f64(int64_t M, int64_t N, int64_t K)
{
    F64Plan p{};
    const int mtiles = (int)((M + F64_BM - 1) / F64_BM);
    p.ntiles = (int)((N + F64_BN - 1) / F64_BN);
    p.tiles = mtiles * p.ntiles;
    const int ktiles = (int)((K + F64_BK - 1) / F64_BK);
    int ks = p.tiles > 0 ? (F64_TARGET_WGS + p.tiles - 1) / p.tiles : 1;
    ks = std::max(1, std::min(ks, ktiles / F64_MIN_KT));
    p.ktps = ktiles > 0 ? (ktiles + ks - 1) / ks : 1;
    p.ksplit = ktiles > 0 ? (ktiles + p.ktps - 1) / p.ktps : 1;
    p.part_bytes = p.ksplit > 1 ? (size_t)p.ksplit * M * N * 8 : 0;
    return p;
}

}  // namespace

namespace splitee_host {

size_t f64_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) { return plan_f64(M, N, K).part_bytes; }

int launch_gemm_f64(const double* A, int64_t lda, const void* W, int w_type, int64_t ldw, const double* C,
                    int64_t ldc, void* Out, bool out64, int64_t ldo, int64_t M, int64_t N, int64_t K, void* ws,
                    size_t ws_bytes, hipStream_t s)
{
    if (M == 0 || N == 0) return SPLITEE_OK;
    const F64Plan p = plan_f64(M, N, K);
    if (ws_bytes < p.part_bytes || (p.part_bytes && !ws)) return SPLITEE_ERR_WORKSPACE;
    double* part = p.ksplit > 1 ? reinterpret_cast<double*>(ws) : nullptr;
    const dim3 grid((unsigned)(p.tiles * p.ksplit));
    const bool bf16 = w_type == SPLITEE_BF16;
#define F64_LAUNCH(WB, O64)                                                                                   \
    hipLaunchKernelGGL((gemm_f64_kernel<WB, O64>), grid, dim3(F64_NT), 0, s, A, lda, W, ldw, C, ldc, Out, ldo, \
                       part, (int)M, (int)N, (int)K, p.ntiles, p.tiles, p.ktps)
    if (bf16) { if (out64) F64_LAUNCH(true, true); else F64_LAUNCH(true, false); }
    else { if (out64) F64_LAUNCH(false, true); else F64_LAUNCH(false, false); }
#undef F64_LAUNCH
    if (p.ksplit > 1) {
        const int64_t total = M * N;
        const unsigned g = (unsigned)std::min<int64_t>((total + 255) / 256, 4096);
        if (out64)
            hipLaunchKernelGGL((f64_sum_kernel<true>), dim3(g), dim3(256), 0, s, part, p.ksplit, C, ldc, Out, ldo,
                               (int)M, (int)N);
        else
            hipLaunchKernelGGL((f64_sum_kernel<false>), dim3(g), dim3(256), 0, s, part, p.ksplit, C, ldc, Out,
                               ldo, (int)M, (int)N);
    }
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

}  // namespace splitee_host
