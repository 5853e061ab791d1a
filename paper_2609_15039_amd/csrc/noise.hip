// Noise, mask and unmask kernels (gfx950).  The noise stream and its correctly
// rounded transforms are in noise_dev.hpp; the transforms' fast and slow paths
// are checked against each other on all 2^32 words and against a binary128
// reference on samples.
#include "noise_dev.hpp"

#pragma clang fp contract(off)

namespace {

// ------------------------------------------------------------------ kernels

// Launch shape of the noise and mask kernels: blockIdx.y walks the rows, the x
// dimension the row's units (no 64-bit divide per thread).  A unit is one Philox
// block (four consecutive elements of a row, 16-byte accesses) or, when the launch
// has fewer than two waves per SIMD of whole blocks (PAIR), half of one: two lanes
// then take the two Box-Muller pairs (or Laplace word pairs) of a block, halving the
// serial chain of binary64 transforms per lane where there are too few waves to
// hide it.  The values are the same either way.
constexpr int64_t PAIR_BELOW = 256 * 4 * 64 * 2; // Philox blocks: 256 CUs x 4 SIMDs x 64 lanes x 2 waves

template <bool PAIR>
__global__ void __launch_bounds__(256) noise_kernel(float* __restrict__ eta, int64_t ld, int64_t M,
                                                    int64_t K, int mech, double scale, uint64_t seed,
                                                    uint64_t sid, uint64_t row0)
{
    constexpr int EPT = PAIR ? 2 : 4; // elements per thread
    const int64_t bpr = K >> 2;       // Philox blocks per row
    const int64_t upr = K / EPT;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int64_t i = blockIdx.y; i < M; i += gridDim.y)
        for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < upr;
             u += (int64_t)gridDim.x * blockDim.x) {
            const uint64_t b = (row0 + (uint64_t)i) * (uint64_t)bpr + (uint64_t)(PAIR ? u >> 1 : u);
            float* o = eta + i * ld + EPT * u;
            if (PAIR)
                *reinterpret_cast<float2*>(o) =
                    noise_half(mech, scale, b, (int)(u & 1), (uint32_t)sid, (uint32_t)(sid >> 32), k0, k1);
            else
                *reinterpret_cast<float4*>(o) = noise_block(mech, scale, b, (uint32_t)sid, (uint32_t)(sid >> 32), k0, k1);
        }
}

// Several noise blocks (same M, row0, mechanism and scale; own K, stream_id and
// output) in one launch, each repeated `reps` times: repetition r of block q
// writes at eta[q] + r * rep_stride[q] with stream id sid[q] + r * rep_sid_step.
// blockIdx.y is the repetition; thread t of it handles Philox block t of the
// concatenation of the noise blocks' M x K / 4 Philox blocks.
struct NoiseBlocks {
    float* eta[splitee::NOISE_MULTI_MAX];
    int64_t ld[splitee::NOISE_MULTI_MAX];
    int64_t K[splitee::NOISE_MULTI_MAX];
    uint64_t sid[splitee::NOISE_MULTI_MAX];
    int64_t first[splitee::NOISE_MULTI_MAX + 1]; // prefix sums of the blocks' Philox block counts
    int64_t rep_stride[splitee::NOISE_MULTI_MAX];
    int count;
    uint64_t rep_sid_step;
};

__global__ void __launch_bounds__(256) noise_multi_kernel(NoiseBlocks nb, int mech, double scale, uint64_t seed,
                                                          uint64_t row0)
{
    const int64_t total = nb.first[nb.count];
    const int64_t r = blockIdx.y;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        int q = 0;
        while (q + 1 < nb.count && t >= nb.first[q + 1]) ++q;
        const int64_t bpr = nb.K[q] >> 2, u = t - nb.first[q];
        const int64_t i = u / bpr, c = u - i * bpr;
        const uint64_t b = (row0 + (uint64_t)i) * (uint64_t)bpr + (uint64_t)c;
        const uint64_t sid = nb.sid[q] + (uint64_t)r * nb.rep_sid_step;
        *reinterpret_cast<float4*>(nb.eta[q] + r * nb.rep_stride[q] + i * nb.ld[q] + 4 * c) =
            noise_block(mech, scale, b, (uint32_t)sid, (uint32_t)(sid >> 32), k0, k1);
    }
}

// Xt = fl32(X + eta) for the elements of one unit (see PAIR_BELOW) per thread; eta
// is generated (GEN) or read; output as float32, one bfloat16 plane, three bfloat16
// planes or (F64) the binary64 sum.  X may be null (X = 0).  Optionally zero-fills
// `zero_count` words at `zero_ptr` (the split-K tile counters of the GEMM that
// follows).
template <int PREC, bool GEN, bool PAIR>
__global__ void __launch_bounds__(256) mask_kernel(
    const float* __restrict__ X, int64_t ldx, const float* __restrict__ eta, int64_t ld_eta, int mech,
    double scale, uint64_t seed, uint64_t sid, uint64_t row0, void* __restrict__ Xt, int64_t ldxt,
    int64_t plane_stride, int64_t M, int64_t K, unsigned* __restrict__ zero_ptr, int64_t zero_count)
{
    constexpr int EPT = PAIR ? 2 : 4; // elements per thread
    const int64_t bpr = K >> 2;
    const int64_t upr = K / EPT;
    const int64_t flat = ((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t fstride = (int64_t)gridDim.x * gridDim.y * blockDim.x;
    for (int64_t z = flat; z < zero_count; z += fstride) zero_ptr[z] = 0u;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int64_t i = blockIdx.y; i < M; i += gridDim.y)
        for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < upr;
             u += (int64_t)gridDim.x * blockDim.x) {
            const int64_t c = EPT * u; // first element of the unit
            float x[4] = {0.f, 0.f, 0.f, 0.f}, e[4];
            if (EPT == 4) {
                if (X) {
                    const float4 v = *reinterpret_cast<const float4*>(X + i * ldx + c);
                    x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
                }
                float4 v;
                if (GEN) {
                    const uint64_t b = (row0 + (uint64_t)i) * (uint64_t)bpr + (uint64_t)u;
                    v = noise_block(mech, scale, b, (uint32_t)sid, (uint32_t)(sid >> 32), k0, k1);
                } else {
                    v = *reinterpret_cast<const float4*>(eta + i * ld_eta + c);
                }
                e[0] = v.x; e[1] = v.y; e[2] = v.z; e[3] = v.w;
            } else {
                if (X) {
                    const float2 v = *reinterpret_cast<const float2*>(X + i * ldx + c);
                    x[0] = v.x; x[1] = v.y;
                }
                float2 v;
                if (GEN) {
                    const uint64_t b = (row0 + (uint64_t)i) * (uint64_t)bpr + (uint64_t)(u >> 1);
                    v = noise_half(mech, scale, b, (int)(u & 1), (uint32_t)sid, (uint32_t)(sid >> 32), k0, k1);
                } else {
                    v = *reinterpret_cast<const float2*>(eta + i * ld_eta + c);
                }
                e[0] = v.x; e[1] = v.y; e[2] = 0.f; e[3] = 0.f;
            }
            if (PREC == SPLITEE_PREC_F64) {
                // one binary64 addition: exact whenever x and eta are within 2^29 of each other in magnitude
                double2* o = reinterpret_cast<double2*>(reinterpret_cast<double*>(Xt) + i * ldxt + c);
                for (int q = 0; q < EPT / 2; ++q)
                    o[q] = X ? make_double2((double)x[2 * q] + (double)e[2 * q], (double)x[2 * q + 1] + (double)e[2 * q + 1])
                             : make_double2((double)e[2 * q], (double)e[2 * q + 1]);
                continue;
            }
            float xt[4];
            for (int q = 0; q < EPT; ++q) xt[q] = X ? x[q] + e[q] : e[q];
            if (PREC == SPLITEE_PREC_F32) {
                float* o = reinterpret_cast<float*>(Xt) + i * ldxt + c;
                if (EPT == 4) *reinterpret_cast<float4*>(o) = make_float4(xt[0], xt[1], xt[2], xt[3]);
                else *reinterpret_cast<float2*>(o) = make_float2(xt[0], xt[1]);
                continue;
            }
            // bfloat16 planes: plane p of elements 2j, 2j + 1 packed in pk[p][j]
            uint32_t pk[3][2];
            for (int j = 0; j < EPT / 2; ++j) {
                if (PREC == SPLITEE_PREC_BF16) pk[0][j] = splitee::bf16x2_rne(xt[2 * j], xt[2 * j + 1]);
                else splitee::split3_bf16x2(xt[2 * j], xt[2 * j + 1], pk[0][j], pk[1][j], pk[2][j]);
            }
            constexpr int NPL = PREC == SPLITEE_PREC_BF16 ? 1 : 3;
            uint16_t* base = reinterpret_cast<uint16_t*>(Xt) + i * ldxt + c;
            for (int p = 0; p < NPL; ++p) {
                if (EPT == 4) *reinterpret_cast<uint2*>(base + p * plane_stride) = make_uint2(pk[p][0], pk[p][1]);
                else *reinterpret_cast<uint32_t*>(base + p * plane_stride) = pk[p][0];
            }
        }
}

__global__ void __launch_bounds__(256) unmask_kernel(const float* __restrict__ R, int64_t ldr,
                                                     const float* __restrict__ C, int64_t ldc,
                                                     float* __restrict__ Y, int64_t ldy, int64_t M,
                                                     int64_t N)
{
    const int64_t qpr = (N + 3) >> 2;
    const int64_t total = M * qpr;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = t / qpr, c = (t - i * qpr) * 4;
        if (c + 4 <= N) {
            float4 r = *reinterpret_cast<const float4*>(R + i * ldr + c);
            float4 cc = *reinterpret_cast<const float4*>(C + i * ldc + c);
            *reinterpret_cast<float4*>(Y + i * ldy + c) =
                make_float4(r.x - cc.x, r.y - cc.y, r.z - cc.z, r.w - cc.w);
        } else {
            for (int64_t j = c; j < N; ++j) Y[i * ldy + j] = R[i * ldr + j] - C[i * ldc + j];
        }
    }
}

__global__ void transform_probe_kernel(const uint32_t* __restrict__ w, int64_t n, int fn, int force_slow,
                                       float* __restrict__ out)
{
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n;
         t += (int64_t)gridDim.x * blockDim.x) {
        float v, s, c;
        switch (fn) {
        case 0: v = cr_laplace_t(w[t], force_slow != 0); break;
        case 1: v = cr_gauss_r(w[t], force_slow != 0); break;
        case 2: cr_sincos_2pi(w[t], force_slow != 0, s, c); v = c; break;
        default: cr_sincos_2pi(w[t], force_slow != 0, s, c); v = s; break;
        }
        out[t] = v;
    }
}

int grid_for(int64_t work_items, int threads)
{
    int64_t g = (work_items + threads - 1) / threads;
    const int64_t cap = 256 * 64; // enough resident waves; the kernels stride beyond
    if (g > cap) g = cap;
    if (g < 1) g = 1;
    return (int)g;
}

// Workgroup width of the row-walking kernels: the widest of 256, 128 and 64 threads
// that divides a row's units, so that no thread of a row's last workgroup idles (a
// row of 640 units -- K = 2560 -- takes five 128-thread workgroups, not three of 256).
int row_threads(int64_t units_per_row)
{
    for (int t = 256; t >= 64; t /= 2)
        if (units_per_row % t == 0) return t;
    return 256;
}

// Grid of the row-walking kernels: x covers a row's units (at most 4096 workgroups,
// the kernels stride beyond), y the rows (at most 65535, likewise).
dim3 row_grid(int64_t M, int64_t units_per_row, int threads)
{
    int64_t gx = (units_per_row + threads - 1) / threads, gy = M;
    gx = gx < 1 ? 1 : (gx > 4096 ? 4096 : gx);
    gy = gy < 1 ? 1 : (gy > 65535 ? 65535 : gy);
    return dim3((unsigned)gx, (unsigned)gy);
}

}  // namespace

namespace splitee_host {

int launch_noise(float* eta, int64_t ld_eta, int64_t M, int64_t K, int mech, double scale,
                 uint64_t seed, uint64_t sid, uint64_t row0, hipStream_t s)
{
    const int64_t work = M * (K / 4);
    if (work == 0) return SPLITEE_OK;
    const bool pair = work < PAIR_BELOW;
    const int64_t upr = K / (pair ? 2 : 4);
    const int nt = row_threads(upr);
    const dim3 g = row_grid(M, upr, nt);
    if (pair)
        hipLaunchKernelGGL(noise_kernel<true>, g, dim3(nt), 0, s, eta, ld_eta, M, K, mech, scale, seed, sid, row0);
    else
        hipLaunchKernelGGL(noise_kernel<false>, g, dim3(nt), 0, s, eta, ld_eta, M, K, mech, scale, seed, sid, row0);
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

int launch_mask(const float* X, int64_t ldx, const float* eta, int64_t ld_eta, int gen_mech,
                double scale, uint64_t seed, uint64_t sid, uint64_t row0, void* Xt, int prec,
                int64_t ldxt, int64_t plane_stride, int64_t M, int64_t K, unsigned* zero_ptr,
                int64_t zero_count, hipStream_t s)
{
    const int64_t work = M * (K / 4);
    if (work == 0 && zero_count == 0) return SPLITEE_OK;
    const bool gen = eta == nullptr;
    const bool pair = gen && work < PAIR_BELOW;
    const int64_t upr = K / (pair ? 2 : 4);
    const int nt = row_threads(upr);
    const dim3 g = row_grid(M, upr, nt), b(nt);
#define SPLITEE_MASK_LAUNCH(P, G, PR)                                                                  \
    hipLaunchKernelGGL((mask_kernel<P, G, PR>), g, b, 0, s, X, ldx, eta, ld_eta, gen_mech, scale, seed, \
                       sid, row0, Xt, ldxt, plane_stride, M, K, zero_ptr, zero_count)
#define SPLITEE_MASK_PREC(P)                                                                           \
    do {                                                                                               \
        if (!gen) SPLITEE_MASK_LAUNCH(P, false, false);                                               \
        else if (pair) SPLITEE_MASK_LAUNCH(P, true, true);                                            \
        else SPLITEE_MASK_LAUNCH(P, true, false);                                                     \
    } while (0)
    if (prec == SPLITEE_PREC_F32) SPLITEE_MASK_PREC(SPLITEE_PREC_F32);
    else if (prec == SPLITEE_PREC_BF16) SPLITEE_MASK_PREC(SPLITEE_PREC_BF16);
    else if (prec == SPLITEE_PREC_BF16X3) SPLITEE_MASK_PREC(SPLITEE_PREC_BF16X3);
    else SPLITEE_MASK_PREC(SPLITEE_PREC_F64);
#undef SPLITEE_MASK_PREC
#undef SPLITEE_MASK_LAUNCH
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

int launch_noise_multi(float* const* eta, const int64_t* ld, const int64_t* K, const uint64_t* sid, int count,
                       int reps, const int64_t* rep_stride, uint64_t rep_sid_step, int64_t M, int mech,
                       double scale, uint64_t seed, uint64_t row0, hipStream_t s)
{
    NoiseBlocks nb{};
    nb.count = count;
    nb.first[0] = 0;
    for (int q = 0; q < count; ++q) {
        nb.eta[q] = eta[q];
        nb.ld[q] = ld[q];
        nb.K[q] = K[q];
        nb.sid[q] = sid[q];
        nb.rep_stride[q] = rep_stride ? rep_stride[q] : 0;
        nb.first[q + 1] = nb.first[q] + M * (K[q] / 4);
    }
    nb.rep_sid_step = rep_sid_step;
    const int64_t work = nb.first[count];
    if (work == 0 || reps == 0) return SPLITEE_OK;
    hipLaunchKernelGGL(noise_multi_kernel, dim3(grid_for(work, 256), (unsigned)reps), dim3(256), 0, s, nb, mech,
                       scale, seed, row0);
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

int launch_unmask(const float* R, int64_t ldr, const float* C, int64_t ldc, float* Y, int64_t ldy,
                  int64_t M, int64_t N, hipStream_t s)
{
    int64_t work = M * ((N + 3) / 4);
    if (work == 0) return SPLITEE_OK;
    hipLaunchKernelGGL(unmask_kernel, dim3(grid_for(work, 256)), dim3(256), 0, s, R, ldr, C, ldc, Y,
                       ldy, M, N);
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

int launch_transform_probe(const uint32_t* w, int64_t n, int fn, int force_slow, float* out,
                           hipStream_t s)
{
    if (n == 0) return SPLITEE_OK;
    hipLaunchKernelGGL(transform_probe_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s, w, n, fn,
                       force_slow, out);
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

}  // namespace splitee_host
