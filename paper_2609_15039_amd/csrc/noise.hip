// Noise, mask and unmask kernels (gfx950).  The noise stream and its correctly
// rounded transforms are in noise_dev.hpp; the transforms' fast and slow paths
// are checked against each other on all 2^32 words and against a binary128
// reference on samples.
#include "noise_dev.hpp"

#pragma clang fp contract(off)

namespace {

// ------------------------------------------------------------------ kernels

// One thread per pair of elements (half a Philox block), one 8-byte store.
__global__ void __launch_bounds__(256) noise_kernel(float* __restrict__ eta, int64_t ld, int64_t M,
                                                    int64_t K, int mech, double scale, uint64_t seed,
                                                    uint64_t sid, uint64_t row0)
{
    const int64_t ppr = K >> 1; // pairs per row
    const int64_t total = M * ppr;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = t / ppr, c = t - i * ppr;
        const uint64_t b = (row0 + (uint64_t)i) * (uint64_t)(K >> 2) + (uint64_t)(c >> 1);
        float2 v = noise_pair(mech, scale, b, (int)(c & 1), (uint32_t)sid, (uint32_t)(sid >> 32), k0, k1);
        *reinterpret_cast<float2*>(eta + i * ld + 2 * c) = v;
    }
}

// Several noise blocks (same M, row0, mechanism and scale; own K, stream_id and
// output) in one launch, each repeated `reps` times: repetition r of block q
// writes at eta[q] + r * rep_stride[q] with stream id sid[q] + r * rep_sid_step.
// blockIdx.y is the repetition; thread t of it handles pair t of the
// concatenation of the blocks' M x K / 2 pairs.
struct NoiseBlocks {
    float* eta[splitee::NOISE_MULTI_MAX];
    int64_t ld[splitee::NOISE_MULTI_MAX];
    int64_t K[splitee::NOISE_MULTI_MAX];
    uint64_t sid[splitee::NOISE_MULTI_MAX];
    int64_t first[splitee::NOISE_MULTI_MAX + 1]; // prefix sums of the blocks' pair counts
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
        const int64_t K = nb.K[q], ppr = K >> 1, u = t - nb.first[q];
        const int64_t i = u / ppr, c = u - i * ppr;
        const uint64_t b = (row0 + (uint64_t)i) * (uint64_t)(K >> 2) + (uint64_t)(c >> 1);
        const uint64_t sid = nb.sid[q] + (uint64_t)r * nb.rep_sid_step;
        const float2 v = noise_pair(mech, scale, b, (int)(c & 1), (uint32_t)sid, (uint32_t)(sid >> 32), k0, k1);
        *reinterpret_cast<float2*>(nb.eta[q] + r * nb.rep_stride[q] + i * nb.ld[q] + 2 * c) = v;
    }
}

// Xt = fl32(X + eta) for 2 elements per thread; eta is generated (gen = true) or
// read; output as float32, one bfloat16 plane, or three bfloat16 planes.  X may
// be null (X = 0).  Optionally zero-fills `zero_count` words at `zero_ptr` (the
// split-K tile counters of the GEMM that follows).
template <int PREC, bool GEN>
__global__ void __launch_bounds__(256) mask_kernel(
    const float* __restrict__ X, int64_t ldx, const float* __restrict__ eta, int64_t ld_eta, int mech,
    double scale, uint64_t seed, uint64_t sid, uint64_t row0, void* __restrict__ Xt, int64_t ldxt,
    int64_t plane_stride, int64_t M, int64_t K, unsigned* __restrict__ zero_ptr, int64_t zero_count)
{
    const int64_t ppr = K >> 1;
    const int64_t total = M * ppr;
    const int64_t gtid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t gstride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t z = gtid; z < zero_count; z += gstride) zero_ptr[z] = 0u;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int64_t t = gtid; t < total; t += gstride) {
        const int64_t i = t / ppr, c = t - i * ppr;
        float2 e;
        if (GEN) {
            const uint64_t b = (row0 + (uint64_t)i) * (uint64_t)(K >> 2) + (uint64_t)(c >> 1);
            e = noise_pair(mech, scale, b, (int)(c & 1), (uint32_t)sid, (uint32_t)(sid >> 32), k0, k1);
        } else {
            e = *reinterpret_cast<const float2*>(eta + i * ld_eta + 2 * c);
        }
        if (PREC == SPLITEE_PREC_F64) {
            // one binary64 addition: exact whenever x and eta are within 2^29 of each other in magnitude
            double2 xd = make_double2((double)e.x, (double)e.y);
            if (X) {
                const float2 x = *reinterpret_cast<const float2*>(X + i * ldx + 2 * c);
                xd = make_double2((double)x.x + xd.x, (double)x.y + xd.y);
            }
            *reinterpret_cast<double2*>(reinterpret_cast<double*>(Xt) + i * ldxt + 2 * c) = xd;
            continue;
        }
        float2 xt;
        if (X) {
            const float2 x = *reinterpret_cast<const float2*>(X + i * ldx + 2 * c);
            xt = make_float2(x.x + e.x, x.y + e.y);
        } else {
            xt = e;
        }
        if (PREC == SPLITEE_PREC_F32) {
            *reinterpret_cast<float2*>(reinterpret_cast<float*>(Xt) + i * ldxt + 2 * c) = xt;
        } else if (PREC == SPLITEE_PREC_BF16) {
            *reinterpret_cast<uint32_t*>(reinterpret_cast<uint16_t*>(Xt) + i * ldxt + 2 * c) =
                splitee::bf16_bits_rne(xt.x) | (splitee::bf16_bits_rne(xt.y) << 16);
        } else {
            uint32_t h0, m0, l0, h1, m1, l1;
            splitee::split3_bf16(xt.x, h0, m0, l0);
            splitee::split3_bf16(xt.y, h1, m1, l1);
            uint16_t* base = reinterpret_cast<uint16_t*>(Xt) + i * ldxt + 2 * c;
            *reinterpret_cast<uint32_t*>(base) = h0 | (h1 << 16);
            *reinterpret_cast<uint32_t*>(base + plane_stride) = m0 | (m1 << 16);
            *reinterpret_cast<uint32_t*>(base + 2 * plane_stride) = l0 | (l1 << 16);
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

}  // namespace

namespace splitee_host {

int launch_noise(float* eta, int64_t ld_eta, int64_t M, int64_t K, int mech, double scale,
                 uint64_t seed, uint64_t sid, uint64_t row0, hipStream_t s)
{
    int64_t work = M * (K / 2);
    if (work == 0) return SPLITEE_OK;
    hipLaunchKernelGGL(noise_kernel, dim3(grid_for(work, 256)), dim3(256), 0, s, eta, ld_eta, M, K,
                       mech, scale, seed, sid, row0);
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

int launch_mask(const float* X, int64_t ldx, const float* eta, int64_t ld_eta, int gen_mech,
                double scale, uint64_t seed, uint64_t sid, uint64_t row0, void* Xt, int prec,
                int64_t ldxt, int64_t plane_stride, int64_t M, int64_t K, unsigned* zero_ptr,
                int64_t zero_count, hipStream_t s)
{
    int64_t work = M * (K / 2);
    int64_t items = work > zero_count ? work : zero_count;
    if (items == 0) return SPLITEE_OK;
    dim3 g(grid_for(items, 256)), b(256);
    const bool gen = eta == nullptr;
#define SPLITEE_MASK_LAUNCH(P, G)                                                                  \
    hipLaunchKernelGGL((mask_kernel<P, G>), g, b, 0, s, X, ldx, eta, ld_eta, gen_mech, scale, seed, \
                       sid, row0, Xt, ldxt, plane_stride, M, K, zero_ptr, zero_count)
    if (prec == SPLITEE_PREC_F32) {
        if (gen) SPLITEE_MASK_LAUNCH(SPLITEE_PREC_F32, true); else SPLITEE_MASK_LAUNCH(SPLITEE_PREC_F32, false);
    } else if (prec == SPLITEE_PREC_BF16) {
        if (gen) SPLITEE_MASK_LAUNCH(SPLITEE_PREC_BF16, true); else SPLITEE_MASK_LAUNCH(SPLITEE_PREC_BF16, false);
    } else if (prec == SPLITEE_PREC_BF16X3) {
        if (gen) SPLITEE_MASK_LAUNCH(SPLITEE_PREC_BF16X3, true); else SPLITEE_MASK_LAUNCH(SPLITEE_PREC_BF16X3, false);
    } else {
        if (gen) SPLITEE_MASK_LAUNCH(SPLITEE_PREC_F64, true); else SPLITEE_MASK_LAUNCH(SPLITEE_PREC_F64, false);
    }
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
        nb.first[q + 1] = nb.first[q] + M * (K[q] / 2);
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
