// Noise, mask and unmask kernels (gfx950).  The noise stream and its correctly
// rounded transforms are in noise_dev.hpp; the transforms' fast and slow paths
// are checked against each other on all 2^32 words and against a binary128
// reference on samples.
#include "noise_dev.hpp"

#pragma clang fp contract(off)

namespace {

// ------------------------------------------------------------------ kernels

// One thread per Philox block (four consecutive elements of a row), one 16-byte store.
__global__ void __launch_bounds__(256) noise_kernel(float* __restrict__ eta, int64_t ld, int64_t M,
                                                    int64_t K, int mech, double scale, uint64_t seed,
                                                    uint64_t sid, uint64_t row0)
{
    const int64_t bpr = K >> 2; // blocks per row
    const int64_t total = M * bpr;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = t / bpr, c = t - i * bpr;
        const uint64_t b = (row0 + (uint64_t)i) * (uint64_t)bpr + (uint64_t)c;
        *reinterpret_cast<float4*>(eta + i * ld + 4 * c) =
            noise_block(mech, scale, b, (uint32_t)sid, (uint32_t)(sid >> 32), k0, k1);
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

// Xt = fl32(X + eta) for the 4 elements of one Philox block per thread; eta is
// generated (gen = true) or read; output as float32, one bfloat16 plane, three
// bfloat16 planes or (F64) the binary64 sum.  X may be null (X = 0).  Optionally
// zero-fills `zero_count` words at `zero_ptr` (the split-K tile counters of the
// GEMM that follows).
template <int PREC, bool GEN>
__global__ void __launch_bounds__(256) mask_kernel(
    const float* __restrict__ X, int64_t ldx, const float* __restrict__ eta, int64_t ld_eta, int mech,
    double scale, uint64_t seed, uint64_t sid, uint64_t row0, void* __restrict__ Xt, int64_t ldxt,
    int64_t plane_stride, int64_t M, int64_t K, unsigned* __restrict__ zero_ptr, int64_t zero_count)
{
    const int64_t bpr = K >> 2;
    const int64_t total = M * bpr;
    const int64_t gtid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t gstride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t z = gtid; z < zero_count; z += gstride) zero_ptr[z] = 0u;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int64_t t = gtid; t < total; t += gstride) {
        const int64_t i = t / bpr, c = t - i * bpr;
        const float4 x = X ? *reinterpret_cast<const float4*>(X + i * ldx + 4 * c) : make_float4(0.f, 0.f, 0.f, 0.f);
        float4 e;
        if (GEN) {
            const uint64_t b = (row0 + (uint64_t)i) * (uint64_t)bpr + (uint64_t)c;
            e = noise_block(mech, scale, b, (uint32_t)sid, (uint32_t)(sid >> 32), k0, k1);
        } else {
            e = *reinterpret_cast<const float4*>(eta + i * ld_eta + 4 * c);
        }
        if (PREC == SPLITEE_PREC_F64) {
            // one binary64 addition: exact whenever x and eta are within 2^29 of each other in magnitude
            double2* o = reinterpret_cast<double2*>(reinterpret_cast<double*>(Xt) + i * ldxt + 4 * c);
            if (X) {
                o[0] = make_double2((double)x.x + (double)e.x, (double)x.y + (double)e.y);
                o[1] = make_double2((double)x.z + (double)e.z, (double)x.w + (double)e.w);
            } else {
                o[0] = make_double2((double)e.x, (double)e.y);
                o[1] = make_double2((double)e.z, (double)e.w);
            }
            continue;
        }
        const float4 xt = X ? make_float4(x.x + e.x, x.y + e.y, x.z + e.z, x.w + e.w) : e;
        if (PREC == SPLITEE_PREC_F32) {
            *reinterpret_cast<float4*>(reinterpret_cast<float*>(Xt) + i * ldxt + 4 * c) = xt;
        } else if (PREC == SPLITEE_PREC_BF16) {
            *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(Xt) + i * ldxt + 4 * c) =
                make_uint2(splitee::bf16_bits_rne(xt.x) | (splitee::bf16_bits_rne(xt.y) << 16),
                           splitee::bf16_bits_rne(xt.z) | (splitee::bf16_bits_rne(xt.w) << 16));
        } else {
            uint32_t h[4], m[4], l[4];
            splitee::split3_bf16(xt.x, h[0], m[0], l[0]);
            splitee::split3_bf16(xt.y, h[1], m[1], l[1]);
            splitee::split3_bf16(xt.z, h[2], m[2], l[2]);
            splitee::split3_bf16(xt.w, h[3], m[3], l[3]);
            uint16_t* base = reinterpret_cast<uint16_t*>(Xt) + i * ldxt + 4 * c;
            *reinterpret_cast<uint2*>(base) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
            *reinterpret_cast<uint2*>(base + plane_stride) = make_uint2(m[0] | (m[1] << 16), m[2] | (m[3] << 16));
            *reinterpret_cast<uint2*>(base + 2 * plane_stride) = make_uint2(l[0] | (l[1] << 16), l[2] | (l[3] << 16));
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
    int64_t work = M * (K / 4);
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
    int64_t work = M * (K / 4);
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
