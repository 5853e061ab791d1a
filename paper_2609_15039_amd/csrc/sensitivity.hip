// Noise scale of the masked projections (gfx950): the spectral norm ||W||_2 by the
// power method on W^T W, and the vector norms ||alpha||_4, ||beta||_2 that the
// sensitivity bounds of Theorems 1-3 take.
//
// One round of the power method (v unit, u = W v, sigma = ||u||, z = W^T u,
// v <- z / ||z||) reads W from HBM once.  A workgroup takes a tile of RB rows x K
// into registers (thread t holds columns 8 t + 2048 c .. + 7 of every row), forms
// the RB dot products with v (per-thread partials, then one cross-lane reduction
// for all RB rows at once), and folds the same registers into its running partial
// of W^T u.  Workgroups are persistent over row tiles, so the partial rows number
// at most PI_MAX_WGS whatever N is.  A second kernel sums the partial rows in a
// fixed order and leaves ||z||^2 as per-workgroup binary64 partial sums, from which
// the next round rescales instead of writing v.
// Products and row sums run in float32 (fma in k order, fixed reduction trees);
// squared norms accumulate in binary64.
#include <math.h>

#include "common.hpp"

namespace {

constexpr int WAVE = 64;
constexpr int PI_NT = 256;                 // threads of the power-method kernels
constexpr int PI_CW = 8 * PI_NT;           // columns of one register chunk
constexpr int PI_MAX_CH = 8;               // chunks per thread: K <= 16384
constexpr int PI_MAX_WGS = 512;            // workgroups (and partial rows) of a round
constexpr int PR_CT = 4;                   // partial-sum kernel: column threads (float4 each)
constexpr int PR_RT = PI_NT / PR_CT;       //   row threads
constexpr int PR_CB = 4 * PR_CT;           //   columns per workgroup
constexpr int PR_LOADS = PI_MAX_WGS / PR_RT; //   partial rows per row thread
static_assert(PR_LOADS * PR_RT == PI_MAX_WGS, "partial rows must fit the unrolled loads");
constexpr int PI_ZN_LOADS = PI_MAX_CH * PI_CW / PR_CB / WAVE; // partial norms per lane

// Rows per tile: two tiles of RB x CH x 8 W elements per thread (the one in use and
// the next, in flight) fit in 128 registers.
constexpr int pi_rows(int ch, bool bf16)
{
    int r = 16;
    while (r > 1 && 2 * r * ch * (bf16 ? 4 : 8) > 128) r /= 2;
    return r;
}
constexpr int ilog2(int x) { return x <= 1 ? 0 : 1 + ilog2(x / 2); }

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, WAVE);
    return v;
}

__device__ __forceinline__ double wave_sum(double v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, WAVE);
    return v;
}

// Wave sums of RB values at once: log2(RB) halving exchanges (distances 32, 16, ..)
// leave lane l one partial sum of row l >> (6 - log2 RB); full exchanges over the
// remaining distances complete it.  Each row's sum is a fixed 6-level tree.
template <int RB>
__device__ __forceinline__ float rows_wave_sum(float (&v)[RB], int lane)
{
    constexpr int LG = ilog2(RB);
#pragma unroll
    for (int s = 0; s < LG; ++s) {
        const int d = 32 >> s, h = RB >> (s + 1);
        const bool up = (lane & d) != 0;
#pragma unroll
        for (int i = 0; i < h; ++i) {
            const float send = up ? v[i] : v[i + h];
            const float keep = up ? v[i + h] : v[i];
            v[i] = keep + __shfl_xor(send, d, WAVE);
        }
    }
    float t = v[0];
#pragma unroll
    for (int d = 32 >> LG; d >= 1; d >>= 1) t += __shfl_xor(t, d, WAVE);
    return t;
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Byte offset that lies outside every buffer resource: such a load returns zeros.
constexpr uint32_t PI_OOB = 0x80000000u;

// Raw register storage of eight consecutive W elements, loaded through a buffer
// resource (one 32-bit lane offset per column chunk, the row offset uniform).
template <bool WBF16> struct W8;
template <> struct W8<true> {
    uint4 q;
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t voff, int soff)
    {
        const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, soff, 0);
        q = make_uint4(v.x, v.y, v.z, v.w);
    }
    __device__ __forceinline__ void zero() { q = make_uint4(0u, 0u, 0u, 0u); }
    // marks the packed words as changed, so that values unpacked before this point
    // are not kept alive for use after it (the tile stays in its packed form)
    __device__ __forceinline__ void fence() { asm volatile("" : "+v"(q.x), "+v"(q.y), "+v"(q.z), "+v"(q.w)); }
    __device__ __forceinline__ void get(float (&w)[8]) const
    {
        const uint32_t d[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            w[2 * e] = __uint_as_float(d[e] << 16);
            w[2 * e + 1] = __uint_as_float(d[e] & 0xFFFF0000u);
        }
    }
};
template <> struct W8<false> {
    float4 a, b;
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t voff, int soff)
    {
        const u32x4 u = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, soff, 0);
        const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(voff + 16), soff, 0);
        a = make_float4(__uint_as_float(u.x), __uint_as_float(u.y), __uint_as_float(u.z), __uint_as_float(u.w));
        b = make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z), __uint_as_float(v.w));
    }
    __device__ __forceinline__ void zero() { a = b = make_float4(0.f, 0.f, 0.f, 0.f); }
    __device__ __forceinline__ void fence() {}
    __device__ __forceinline__ void get(float (&w)[8]) const
    {
        w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
        w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
    }
};

// Tile rows n0 .. n0 + RB - 1.  Each row gets its own buffer resource of K elements
// (none for rows at or past N), so that every load is unconditional and loads past
// the row, or of a missing row, return zeros; voff[c] is the lane's byte offset of
// chunk c within a row, PI_OOB past column K.
template <int RB, int CH, bool WBF16>
__device__ __forceinline__ void load_tile(W8<WBF16> (&w)[RB][CH], const void* W, int64_t ldw, int N, int K, int n0,
                                          const uint32_t (&voff)[CH])
{
    constexpr int ES = WBF16 ? 2 : 4;
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char*>(reinterpret_cast<const char*>(W) + (int64_t)(n0 + r) * ldw * ES), (short)0,
            n0 + r < N ? K * ES : 0, 0x00020000);
#pragma unroll
        for (int c = 0; c < CH; ++c) w[r][c].load(rsrc, voff[c], 0);
    }
}

// Rows n0 .. n0 + RB - 1 of one round: u = (W z) / ||z|| (z's columns in x), sum u^2
// into uu (thread 0), zacc += W_tile^T u.
template <int RB, int CH, bool WBF16>
__device__ __forceinline__ void round_tile(W8<WBF16> (&w)[RB][CH], const float (&x)[CH][8], float (&zacc)[CH][8],
                                           float (*red)[RB], float* u_s, float inv, int N, int n0, int tid,
                                           double& uu)
{
    constexpr int LG = ilog2(RB);
    const int lane = tid % WAVE, wave = tid / WAVE;
    float acc[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        acc[r] = 0.f;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            float f[8];
            w[r][c].get(f);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[r] = fmaf(f[e], x[c][e], acc[r]);
        }
    }
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
        for (int c = 0; c < CH; ++c) w[r][c].fence();
    const float s = rows_wave_sum<RB>(acc, lane);
    if ((lane & ((WAVE >> LG) - 1)) == 0) red[wave][lane >> (6 - LG)] = s;
    __syncthreads();
    if (tid < RB) {
        float q = red[0][tid];
#pragma unroll
        for (int v = 1; v < PI_NT / WAVE; ++v) q += red[v][tid];
        u_s[tid] = n0 + tid < N ? q * inv : 0.f;
    }
    __syncthreads();
    if (tid == 0)
        for (int r = 0; r < RB; ++r) uu += (double)u_s[r] * (double)u_s[r];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        const float ur = u_s[r];
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            float f[8];
            w[r][c].get(f);
#pragma unroll
            for (int e = 0; e < 8; ++e) zacc[c][e] = fmaf(f[e], ur, zacc[c][e]);
        }
    }
}

// One round: for every row tile t = blockIdx.x, blockIdx.x + gridDim.x, .. (the next
// tile's loads issued before the current tile's arithmetic): u = (W z) / ||z|| over
// the tile's rows, then zacc += W_tile^T u.  At the end zpart[blockIdx.x][:] = zacc and
// upart[blockIdx.x] = sum of the u^2 of its tiles.  Requires gridDim.x <= tile count.
template <int CH, bool WBF16>
__global__ void __launch_bounds__(PI_NT) pi_round_kernel(const void* __restrict__ W, int64_t ldw, int N, int K,
                                                         const float* __restrict__ z,
                                                         const double* __restrict__ zn_part, int nzn,
                                                         double* __restrict__ upart, float* __restrict__ zpart)
{
    constexpr int RB = pi_rows(CH, WBF16);
    __shared__ float red[PI_NT / WAVE][RB];
    __shared__ float u_s[RB];
    const int tid = threadIdx.x, lane = tid % WAVE;
    const int ntiles = (N + RB - 1) / RB, G = gridDim.x;

    constexpr int ES = WBF16 ? 2 : 4;
    uint32_t voff[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int k = 8 * tid + PI_CW * c;
        voff[c] = k < K ? (uint32_t)(k * ES) : PI_OOB;
    }

    // this thread's columns of z (zeros past K), unconditional loads as for W
    const __amdgpu_buffer_rsrc_t rz =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(z), (short)0, K * 4, 0x00020000);
    float x[CH][8], zacc[CH][8];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const uint32_t xo = voff[c] == PI_OOB ? PI_OOB : voff[c] / ES * 4;
        const u32x4 a = __builtin_amdgcn_raw_buffer_load_b128(rz, (int)xo, 0, 0);
        const u32x4 b = __builtin_amdgcn_raw_buffer_load_b128(rz, (int)(xo + 16), 0, 0);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            x[c][e] = __uint_as_float(a[e]);
            x[c][4 + e] = __uint_as_float(b[e]);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) zacc[c][e] = 0.f;
    }

    W8<WBF16> wa[RB][CH], wb[RB][CH];
    int t = blockIdx.x;
    load_tile<RB, CH, WBF16>(wa, W, ldw, N, K, t * RB, voff);

    // 1 / ||z||, the same fixed-order sum in every wave (all loads issued first)
    const __amdgpu_buffer_rsrc_t rn =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<double*>(zn_part), (short)0, nzn * 8, 0x00020000);
    double zn[PI_ZN_LOADS];
#pragma unroll
    for (int j = 0; j < PI_ZN_LOADS; ++j) {
        const uint32_t i = (uint32_t)(lane + WAVE * j);
        zn[j] = __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(rn, (int)(i * 8), 0, 0));
    }
    double zz = zn[0];
#pragma unroll
    for (int j = 1; j < PI_ZN_LOADS; ++j) zz += zn[j];
    zz = wave_sum(zz);
    const float inv = zz > 0.0 ? (float)(1.0 / sqrt(zz)) : 0.f;

    double uu = 0.0;
    while (true) {
        const int t1 = t + G;
        if (t1 < ntiles) load_tile<RB, CH, WBF16>(wb, W, ldw, N, K, t1 * RB, voff);
        round_tile<RB, CH, WBF16>(wa, x, zacc, red, u_s, inv, N, t * RB, tid, uu);
        if (t1 >= ntiles) break;
        const int t2 = t1 + G;
        if (t2 < ntiles) load_tile<RB, CH, WBF16>(wa, W, ldw, N, K, t2 * RB, voff);
        round_tile<RB, CH, WBF16>(wb, x, zacc, red, u_s, inv, N, t1 * RB, tid, uu);
        if (t2 >= ntiles) break;
        t = t2;
    }
    float* zp = zpart + (int64_t)blockIdx.x * K;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int k = 8 * tid + PI_CW * c;
        if (k < K) {
            *reinterpret_cast<float4*>(zp + k) = make_float4(zacc[c][0], zacc[c][1], zacc[c][2], zacc[c][3]);
            *reinterpret_cast<float4*>(zp + k + 4) = make_float4(zacc[c][4], zacc[c][5], zacc[c][6], zacc[c][7]);
        }
    }
    if (tid == 0) upart[blockIdx.x] = uu;
}

// z[k] = sum over the nrows <= PI_MAX_WGS partial rows (row thread j sums rows j, j + PR_RT, ..;
// the row threads' sums meet in a fixed tree); zn_part[blockIdx.x] = sum of the
// block's z^2.  Workgroup 0 also writes *sig = sqrt(sum of upart) when sig is given.
__global__ void __launch_bounds__(PI_NT) pi_reduce_kernel(const float* __restrict__ zpart, int nrows, int K,
                                                          float* __restrict__ z, double* __restrict__ zn_part,
                                                          const double* __restrict__ upart, int nupart,
                                                          double* __restrict__ sig)
{
    __shared__ float4 red[PI_NT / WAVE][PR_CT];
    __shared__ double q[PR_CT];
    const int ct = threadIdx.x % PR_CT, rt = threadIdx.x / PR_CT;
    const int k = blockIdx.x * PR_CB + 4 * ct;
    // at most PR_LOADS rows per row-thread, all loads issued before the adds
    float4 p[PR_LOADS];
#pragma unroll
    for (int j = 0; j < PR_LOADS; ++j) {
        const int b = rt + PR_RT * j;
        p[j] = k < K && b < nrows ? *reinterpret_cast<const float4*>(zpart + (int64_t)b * K + k)
                                  : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    float4 acc = p[0];
#pragma unroll
    for (int j = 1; j < PR_LOADS; ++j) {
        acc.x += p[j].x; acc.y += p[j].y; acc.z += p[j].z; acc.w += p[j].w;
    }
    // row threads of a column group: 16 per wave (lanes ct, ct + 4, ..), then 4 waves
#pragma unroll
    for (int d = PR_CT; d < WAVE; d *= 2) {
        acc.x += __shfl_xor(acc.x, d, WAVE);
        acc.y += __shfl_xor(acc.y, d, WAVE);
        acc.z += __shfl_xor(acc.z, d, WAVE);
        acc.w += __shfl_xor(acc.w, d, WAVE);
    }
    const int wave = threadIdx.x / WAVE;
    if (threadIdx.x % WAVE < PR_CT) red[wave][ct] = acc;
    __syncthreads();
    if (threadIdx.x < PR_CT) {
        float4 t = red[0][ct];
        for (int j = 1; j < PI_NT / WAVE; ++j) {
            const float4 p = red[j][ct];
            t.x += p.x; t.y += p.y; t.z += p.z; t.w += p.w;
        }
        double sq = 0.0;
        if (k < K) {
            *reinterpret_cast<float4*>(z + k) = t;
            sq = (double)t.x * t.x + (double)t.y * t.y + (double)t.z * t.z + (double)t.w * t.w;
        }
        q[ct] = sq;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double s = 0.0;
        for (int c = 0; c < PR_CT; ++c) s += q[c];
        zn_part[blockIdx.x] = s;
    }
    if (sig && blockIdx.x == 0 && threadIdx.x < WAVE) {
        double s = 0.0;
        for (int i = threadIdx.x; i < nupart; i += WAVE) s += upart[i];
        s = wave_sum(s);
        if (threadIdx.x == 0) *sig = sqrt(s);
    }
}

// out[0] = sum alpha^4, out[1] = sum beta^2 (0 when beta is null), binary64, one workgroup.
__global__ void __launch_bounds__(PI_NT) vec_norms_kernel(const float* __restrict__ alpha,
                                                          const float* __restrict__ beta, int64_t d,
                                                          double* __restrict__ out)
{
    __shared__ double red[2][PI_NT / WAVE];
    const int lane = threadIdx.x % WAVE, wave = threadIdx.x / WAVE;
    double a4 = 0.0, b2 = 0.0;
    for (int64_t i = threadIdx.x; i < d; i += PI_NT) {
        const double a = alpha[i], a2 = a * a;
        a4 += a2 * a2;
        if (beta) b2 += (double)beta[i] * (double)beta[i];
    }
    a4 = wave_sum(a4);
    b2 = wave_sum(b2);
    if (lane == 0) {
        red[0][wave] = a4;
        red[1][wave] = b2;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double s0 = 0.0, s1 = 0.0;
        for (int w = 0; w < PI_NT / WAVE; ++w) {
            s0 += red[0][w];
            s1 += red[1][w];
        }
        out[0] = s0;
        out[1] = s1;
    }
}

inline size_t align256(size_t b) { return (b + 255) / 256 * 256; }

struct PiLayout {
    double* sig;     // iters
    double* upart;   // nwg
    double* zn_part; // nzn
    float* z;        // K
    float* zpart;    // nwg x K
    size_t bytes;
};

int pi_chunks(int64_t K) { return (int)((K + PI_CW - 1) / PI_CW); }

int pi_tile_rows(int ch, bool bf16) { return pi_rows(ch, bf16); }

// Workgroups of a round, one partial row each: at least 128 (bandwidth), about N / 16
// (partial rows written and read again stay near a quarter of the bfloat16 W
// bytes), at most PI_MAX_WGS and the tile count.
int64_t pi_workgroups(int64_t N, int64_t K, bool bf16)
{
    const int64_t rb = pi_tile_rows(std::max(pi_chunks(K), 1), bf16);
    const int64_t want = std::max<int64_t>(128, (N + 15) / 16);
    return std::max<int64_t>(1, std::min<int64_t>({(N + rb - 1) / rb, (int64_t)PI_MAX_WGS, want}));
}

PiLayout pi_layout(void* ws, int64_t N, int64_t K, int iters, bool bf16)
{
    const int64_t nwg = pi_workgroups(N, K, bf16), nzn = (K + PR_CB - 1) / PR_CB;
    const uintptr_t base = reinterpret_cast<uintptr_t>(ws);
    PiLayout L{};
    size_t off = 0;
    L.sig = reinterpret_cast<double*>(base + off);
    off += align256((size_t)iters * 8);
    L.upart = reinterpret_cast<double*>(base + off);
    off += align256((size_t)nwg * 8);
    L.zn_part = reinterpret_cast<double*>(base + off);
    off += align256((size_t)nzn * 8);
    L.z = reinterpret_cast<float*>(base + off);
    off += align256((size_t)K * 4);
    L.zpart = reinterpret_cast<float*>(base + off);
    off += align256((size_t)nwg * K * 4);
    L.bytes = off;
    return L;
}

template <int CH>
void launch_round(const void* W, bool bf16, int64_t ldw, int N, int K, const PiLayout& L, int nwg, int nzn,
                  hipStream_t s)
{
    if (bf16)
        hipLaunchKernelGGL((pi_round_kernel<CH, true>), dim3(nwg), dim3(PI_NT), 0, s, W, ldw, N, K,
                           (const float*)L.z, (const double*)L.zn_part, nzn, L.upart, L.zpart);
    else
        hipLaunchKernelGGL((pi_round_kernel<CH, false>), dim3(nwg), dim3(PI_NT), 0, s, W, ldw, N, K,
                           (const float*)L.z, (const double*)L.zn_part, nzn, L.upart, L.zpart);
}

}  // namespace

namespace splitee_host {

int spectral_max_k() { return PI_MAX_CH * PI_CW; }

size_t spectral_workspace_bytes(int64_t N, int64_t K, int iters)
{
    // the larger of the bfloat16 and float32 layouts: one size serves either type
    return std::max(pi_layout(nullptr, N, K, iters, true).bytes, pi_layout(nullptr, N, K, iters, false).bytes);
}

int launch_spectral_norm(const void* W, int w_type, int64_t ldw, int64_t N, int64_t K, int iters, uint64_t seed,
                         uint64_t sid, double* sigma, double* history, void* ws, hipStream_t s)
{
    const bool bf16 = w_type == SPLITEE_BF16;
    const PiLayout L = pi_layout(ws, N, K, iters, bf16);
    const int nwg = (int)pi_workgroups(N, K, bf16), nzn = (int)((K + PR_CB - 1) / PR_CB);
    const int ch = pi_chunks(K);
    // start: a standard Gaussian draw of the noise stream (seed, sid), row 0; its norm
    // is taken by the partial-sum kernel over one partial row
    int rc = launch_noise(L.zpart, K, 1, K, SPLITEE_MECH_GAUSSIAN, 1.0, seed, sid, 0, s);
    if (rc != SPLITEE_OK) return rc;
    hipLaunchKernelGGL(pi_reduce_kernel, dim3(nzn), dim3(PI_NT), 0, s, (const float*)L.zpart, 1, (int)K, L.z,
                       L.zn_part, (const double*)nullptr, 0, (double*)nullptr);
    for (int it = 0; it < iters; ++it) {
        switch (ch) {
        case 1: launch_round<1>(W, bf16, ldw, (int)N, (int)K, L, nwg, nzn, s); break;
        case 2: launch_round<2>(W, bf16, ldw, (int)N, (int)K, L, nwg, nzn, s); break;
        case 3: launch_round<3>(W, bf16, ldw, (int)N, (int)K, L, nwg, nzn, s); break;
        case 4: launch_round<4>(W, bf16, ldw, (int)N, (int)K, L, nwg, nzn, s); break;
        case 5: launch_round<5>(W, bf16, ldw, (int)N, (int)K, L, nwg, nzn, s); break;
        case 6: launch_round<6>(W, bf16, ldw, (int)N, (int)K, L, nwg, nzn, s); break;
        case 7: launch_round<7>(W, bf16, ldw, (int)N, (int)K, L, nwg, nzn, s); break;
        case 8: launch_round<8>(W, bf16, ldw, (int)N, (int)K, L, nwg, nzn, s); break;
        default: return SPLITEE_ERR_UNSUPPORTED;
        }
        hipLaunchKernelGGL(pi_reduce_kernel, dim3(nzn), dim3(PI_NT), 0, s, (const float*)L.zpart, nwg, (int)K,
                           L.z, L.zn_part, (const double*)L.upart, nwg, L.sig + it);
    }
    if (hipGetLastError() != hipSuccess) return SPLITEE_ERR_HIP;
    if (hipMemcpyAsync(sigma, L.sig + (iters - 1), sizeof(double), hipMemcpyDeviceToHost, s) != hipSuccess)
        return SPLITEE_ERR_HIP;
    if (history &&
        hipMemcpyAsync(history, L.sig, (size_t)iters * sizeof(double), hipMemcpyDeviceToHost, s) != hipSuccess)
        return SPLITEE_ERR_HIP;
    return hipStreamSynchronize(s) == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

int launch_vec_norms(const float* alpha, const float* beta, int64_t d, double* out_dev, double* out_host,
                     hipStream_t s)
{
    hipLaunchKernelGGL(vec_norms_kernel, dim3(1), dim3(PI_NT), 0, s, alpha, beta, d, out_dev);
    if (hipGetLastError() != hipSuccess) return SPLITEE_ERR_HIP;
    if (hipMemcpyAsync(out_host, out_dev, 2 * sizeof(double), hipMemcpyDeviceToHost, s) != hipSuccess)
        return SPLITEE_ERR_HIP;
    return hipStreamSynchronize(s) == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

}  // namespace splitee_host
