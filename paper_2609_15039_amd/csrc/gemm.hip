// MFMA GEMM kernels of the masked linear layer (gfx950).
//
//   Out = A . W^T            (R, the GPU's part: r = W (x + eta))
//   Out = fl32(A . W^T - C)  (fused unmask epilogue, Eq. add-and-then-subtract)
//
// A is the masked input in one of three forms: float32 (binary32 MFMA
// v_mfma_f32_16x16x4_f32), one bfloat16 plane, or three bfloat16 planes
// hi + mid + lo that sum exactly to the float32 masked input (three bfloat16
// MFMA passes v_mfma_f32_16x16x32_bf16 into one float32 accumulator).  W is
// N x K row-major (nn.Linear layout), float32 or bfloat16.
//
// Tiling: a workgroup owns a BM x BN output tile and a contiguous range of K
// tiles; 16-byte global loads are staged through padded LDS rows (16 bytes of
// padding keeps the 16-byte fragment reads conflict-free), the next K tile is
// prefetched into registers while the current one is multiplied.  When the
// K range is split over several workgroups (split-K, to fill 256 CUs at small
// M), each writes its float32 partial tile to the workspace and the last one to
// arrive (device-scope counter) sums the partials in split order and applies
// the epilogue, so results do not depend on arrival order.
#include "common.hpp"

#include <algorithm>
#include <type_traits>

namespace {

constexpr int WAVE = 64;
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

// Split-K hand-off between the workgroups of one output tile.  Partials are
// written with agent-scope relaxed atomic stores (or sc1 buffer stores) and read
// with sc1 buffer loads, which gfx950 performs write-through / coherently across
// the XCDs' L2 caches.  Each wave waits for its partial stores to complete before
// the workgroup bumps the tile counter, so the workgroup that sees the count reach
// ksplit-1 reads complete partials.  This is the ordering of an agent-scope
// release/acquire pair without its whole-L2 write-back and invalidate, which only
// non-coherent stores need.
__device__ __forceinline__ void store_partial(float* p, float v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Returns true in the last-arriving workgroup of the tile (all its threads),
// which then owns the reduction and resets the counter for the next call.
// `flag` is one LDS word the workgroup no longer needs for anything else.
__device__ __forceinline__ bool splitk_arrive(unsigned* counter, int ksplit, unsigned* flag)
{
    __builtin_amdgcn_s_waitcnt(0); // this wave's partial stores have completed
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned prev = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *flag = (prev == (unsigned)(ksplit - 1)) ? 1u : 0u;
    }
    __syncthreads();
    return *flag != 0u;
}

// The last workgroup's reduction of a BM x BN tile: the tile is walked row-major
// in 16-byte units, CH per thread at a time; for each chunk all loads of one
// split are issued together (agent-coherent buffer loads, sc1), then added in
// split order, then C is subtracted and Y stored with 16-byte accesses.
template <int BM, int BN, int NT, int CH>
__device__ __forceinline__ void splitk_reduce(const float* tp, int ksplit, int m0, int n0, int M, int N,
                                              const float* C, int64_t ldc, float* Out, int64_t ldo)
{
    constexpr int F4 = BM * BN / 4, ROW4 = BN / 4;
    static_assert(F4 % (NT * CH) == 0, "reduction chunks");
    const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(tp), (short)0,
                                                                       ksplit * BM * BN * 4, 0x00020000);
    constexpr int SC1 = 16; // cache policy: coherent at agent scope
    for (int c0 = 0; c0 < F4; c0 += NT * CH) {
        f32x4_t sum[CH];
#pragma unroll
        for (int c = 0; c < CH; ++c)
            sum[c] = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                rp, (c0 + c * NT + (int)threadIdx.x) * 16, 0, SC1));
        for (int q = 1; q < ksplit; ++q) {
            f32x4_t v[CH];
#pragma unroll
            for (int c = 0; c < CH; ++c)
                v[c] = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                    rp, (q * F4 + c0 + c * NT + (int)threadIdx.x) * 16, 0, SC1));
#pragma unroll
            for (int c = 0; c < CH; ++c) sum[c] += v[c];
        }
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int f = c0 + c * NT + (int)threadIdx.x;
            const int row = m0 + f / ROW4, col = n0 + (f % ROW4) * 4;
            if (row >= M) continue;
            f32x4_t y = sum[c];
            if (col + 4 <= N) {
                if (C) y -= __builtin_bit_cast(f32x4_t, *reinterpret_cast<const float4*>(C + (int64_t)row * ldc + col));
                *reinterpret_cast<float4*>(Out + (int64_t)row * ldo + col) = __builtin_bit_cast(float4, y);
            } else {
                for (int e = 0; e < 4 && col + e < N; ++e) {
                    float v = y[e];
                    if (C) v = v - C[(int64_t)row * ldc + col + e];
                    Out[(int64_t)row * ldo + col + e] = v;
                }
            }
        }
    }
}

__device__ __forceinline__ void splitk_reset(unsigned* counter)
{
    __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

constexpr int SC1 = 16;  // buffer cache policy: coherent at agent scope (write-through / bypass)
constexpr int KSMAX = 8; // largest split-K factor of the tiled kernels
constexpr uint32_t OOB_OFF = 0x80000000u;

// Finishes the workgroup's BM x BN accumulator tile.  The tile goes through LDS
// (row-major, rows padded by 4 floats) so that every global access below is a
// 16-byte access of consecutive columns:
//   ksplit == 1: Y = acc - C;
//   ksplit  > 1: this split's partial is written (agent-coherent), the tile
//                counter is bumped, and the last workgroup to arrive loads all
//                partials in one round, sums them in split order, subtracts C and
//                stores Y.
// `lds` must hold BM * (BN + 4) + 1 floats and be free (callers sync first).
template <int BM, int BN, int NT, int TM, int TN, int WTM, int WTN, int WGM>
__device__ __forceinline__ void finish_tile(const f32x4_t (&acc)[TM][TN], float* lds, int m0, int n0, int M, int N,
                                            const float* C, int64_t ldc, float* Out, int64_t ldo, int ksplit,
                                            int split, int tile, float* part, unsigned* counters)
{
    constexpr int LDT = BN + 4;
    constexpr int ROW4 = BN / 4, F4 = BM * BN / 4, PER = F4 / NT;
    constexpr int CH = PER < 4 ? PER : 4;
    static_assert(F4 % NT == 0 && PER % CH == 0, "epilogue split");
    const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
    const int wm = wave % WGM, wn = wave / WGM;
    const int erow = 4 * (lane / 16), ecol = lane % 16;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                lds[(wm * WTM + i * 16 + erow + r) * LDT + wn * WTN + j * 16 + ecol] = acc[i][j][r];
    __syncthreads();

    auto finish4 = [&](int f, f32x4_t y) {
        const int row = m0 + f / ROW4, col = n0 + (f % ROW4) * 4;
        if (row >= M) return;
        if (col + 4 <= N) {
            if (C) y -= __builtin_bit_cast(f32x4_t, *reinterpret_cast<const float4*>(C + (int64_t)row * ldc + col));
            *reinterpret_cast<float4*>(Out + (int64_t)row * ldo + col) = __builtin_bit_cast(float4, y);
        } else {
            for (int e = 0; e < 4 && col + e < N; ++e) {
                float v = y[e];
                if (C) v = v - C[(int64_t)row * ldc + col + e];
                Out[(int64_t)row * ldo + col + e] = v;
            }
        }
    };
    auto lds4 = [&](int f) {
        return *reinterpret_cast<const f32x4_t*>(&lds[(f / ROW4) * LDT + (f % ROW4) * 4]);
    };

    if (ksplit == 1) {
#pragma unroll
        for (int c = 0; c < PER; ++c) finish4(tid + c * NT, lds4(tid + c * NT));
        return;
    }
    const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc(
        part + (int64_t)tile * ksplit * (BM * BN), (short)0, ksplit * BM * BN * 4, 0x00020000);
#pragma unroll
    for (int c = 0; c < PER; ++c) {
        const int f = tid + c * NT;
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, lds4(f)), rp, (split * F4 + f) * 16, 0, SC1);
    }
    unsigned* flag = reinterpret_cast<unsigned*>(lds + BM * LDT);
    if (!splitk_arrive(counters + tile, ksplit, flag)) return;
#pragma unroll
    for (int c0 = 0; c0 < PER; c0 += CH) {
        f32x4_t v[KSMAX][CH];
#pragma unroll
        for (int q = 0; q < KSMAX; ++q)
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                const int f = tid + (c0 + c) * NT;
                const uint32_t off = q < ksplit ? (uint32_t)((q * F4 + f) * 16) : OOB_OFF;
                v[q][c] = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rp, (int)off, 0, SC1));
            }
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            f32x4_t sum = v[0][c];
#pragma unroll
            for (int q = 1; q < KSMAX; ++q)
                if (q < ksplit) sum += v[q][c];
            finish4(tid + (c0 + c) * NT, sum);
        }
    }
    if (tid == 0) splitk_reset(counters + tile);
}

// ------------------------------------------------- bounds-checked buffer loads
// Operands are read with buffer loads whose resource covers exactly the matrix:
// a lane whose row or k lies outside it gets an offset beyond the extent and
// reads zeros, which pads every tail.  A bfloat16 K tile is 64 k = 8 units of 16
// bytes per row.

constexpr int BK = 64;
constexpr uint32_t OOB = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 load16(__amdgpu_buffer_rsrc_t r, uint32_t voff)
{
    u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, 0, 0);
    return make_uint4(v.x, v.y, v.z, v.w);
}

// ----------------------------------------------- bf16 MFMA, W streamed (M > 16)
// For weight-streaming shapes W is the only large operand and is read once: each
// wave loads its own WN columns of W from HBM straight into MFMA B-operand
// registers, D K tiles ahead of use, so W needs no LDS space, no LDS bandwidth
// and no barrier of its own.  The masked input (NPL planes x BM rows x one K
// tile, shared by the 4 waves side by side along N) goes global -> LDS by
// buffer-load-to-LDS (no registers), in the swizzled layout of the tiled kernel,
// into a ring of D + 1 stages.  Both operands of tile t + D are issued together
// at tile t: vector-memory loads complete in order, so waiting for an older
// masked-input tile never waits for a younger W tile.  One barrier per K tile.
// Split over K, each workgroup writes its partial accumulators in register
// order (16-byte stores, no atomics) and `stream_sum_kernel` adds the splits in
// split order and applies the unmask epilogue.
//
// W in row-major order: lane (c, h) of a B-operand load reads 16 bytes of row c
// of a 32-row block, so one load touches 32 cache lines for 32 bytes each, and the
// vector L1 (which serves a 128-byte line access every other clock, however few
// bytes of it are used) delivers a quarter of its bandwidth.  W in the tiled order
// (TILED; splitee_tile_weights) stores each (32-row block, K tile, k step) as the
// 1 KB the 64 lanes load, so every load is 8 whole lines.  With tiled W the kernel
// runs 8 waves (two per SIMD): one wave's MFMAs overlap the other's load issue.

typedef __attribute__((address_space(3))) void* lds_ptr_t;

template <int I, int BYTES>
__device__ __forceinline__ unsigned char* stream_stage()
{
    __shared__ __attribute__((aligned(16))) unsigned char buf[BYTES];
    return buf;
}

// waits until at most N of this wave's vector-memory operations are outstanding
template <int N>
__device__ __forceinline__ void wait_vmem()
{
    static_assert(N >= 0 && N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

constexpr int ST_NW = 4; // waves per workgroup of the streamed kernel (WGM x WGN)
constexpr int ST_MIN_KT = 6, ST_MAX_KS = 12; // K split of the streamed kernel

// v_mfma_f32_32x32x16_bf16 operands: lane l holds row (A) or column (B) l % 32 and
// k = 8 (l / 32) .. + 7 of a 16-wide k step; result element e of lane l is row
// 8 (e / 4) + 4 (l / 32) + e % 4, column l % 32.
// LDS chunk swizzle of the 128-byte masked-input rows: 16-byte chunk c of row r sits
// in slot c ^ swizzle(r).  SW 0: r & 7; SW 1: (r >> 1) & 7 (pairs of rows share a
// pattern and differ in the upper half of a 64-bank array).
template <int SW>
__device__ __forceinline__ int lds_swizzle(int r)
{
    return SW == 0 ? (r & 7) : ((r >> 1) & 7);
}

// Unmask epilogue of an unsplit wave tile held in v_mfma_f32_32x32x16 accumulators
// (TM x TN blocks, rows r0 + 32 i + 8 (e / 4) + 4 h + e % 4, columns c0 + 32 j + c for
// lane (c, h)): Out = acc - C.  Every C load of the tile is issued before the first
// subtraction, so the wave waits for them once; loading and storing element by element
// made each load a separate round trip (64 per lane, about 30 us per workgroup while the
// other workgroups of the CU streamed their operands).  Elements outside M x N load C[0]
// (always valid: the kernels run only for M, N >= 1) and store nothing.
template <int TM, int TN>
__device__ __forceinline__ void store_tile(const f32x16_t (&acc)[TM][TN], const float* __restrict__ C, int64_t ldc,
                                           float* __restrict__ Out, int64_t ldo, int M, int N, int r0, int c0,
                                           int fc, int fh)
{
    float cv[TM][TN][16];
    if (C) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int col = c0 + j * 32 + fc;
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int row = r0 + i * 32 + 8 * (e / 4) + 4 * fh + (e % 4);
                    const bool ok = row < M && col < N;
                    cv[i][j][e] = C[ok ? (int64_t)row * ldc + col : 0];
                }
            }
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = c0 + j * 32 + fc;
            if (col >= N) continue;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = r0 + i * 32 + 8 * (e / 4) + 4 * fh + (e % 4);
                if (row < M) Out[(int64_t)row * ldo + col] = C ? acc[i][j][e] - cv[i][j][e] : acc[i][j][e];
            }
        }
}

template <int NPL, int BM, int BN, int WGM, int D, int NW = ST_NW, bool TILED = false, int SW = 1>
__global__ void __launch_bounds__(NW * WAVE, (TILED && NW == 4) ? 2 : 1)
gemm_stream_kernel(const uint16_t* __restrict__ A, int64_t lda, int64_t pstride,
                   const uint16_t* __restrict__ W, int64_t ldw, const float* __restrict__ C, int64_t ldc,
                   float* __restrict__ Out, int64_t ldo, int M, int N, int K, int mtiles, int ntiles,
                   int ksplit, int kt_per_split, float* __restrict__ part)
{
    constexpr int WGN = NW / WGM;
    constexpr int WTM = BM / WGM, WTN = BN / WGN; // wave tile
    constexpr int TM = WTM / 32, TN = WTN / 32;   // 32 x 32 MFMA blocks of the wave tile
    constexpr int S = D + 1;                  // masked-input stages = W register slots
    constexpr int AROWS = NPL * BM;           // 128-byte LDS rows per stage
    constexpr int SB = AROWS * 128;
    constexpr int LA = AROWS / 8 / NW;        // 1 KB LDS-DMA loads per wave per tile
    constexpr int LW = 4 * TN;                // W loads per wave per tile (4 k steps of 16)
    static_assert(WGM * WGN == NW && TM * 32 * WGM == BM && TN * 32 * WGN == BN, "wave tile");
    static_assert(AROWS % (8 * NW) == 0, "masked-input stage must split evenly over the waves");
    static_assert(S >= 2 && S <= 4, "stages");
    static_assert((D - 1) * (LA + LW) < 64, "loads in flight exceed the wait counter");

    const int tid = threadIdx.x, lane = tid % WAVE;
    const int wave = __builtin_amdgcn_readfirstlane(tid / WAVE);
    const int wm = wave / WGN, wn = wave % WGN;
    const uint32_t lb = splitee::xcd_logical_block(blockIdx.x, gridDim.x);
    const int tiles = mtiles * ntiles;
    const int split = (int)lb / tiles, tile = (int)lb % tiles;
    const int m0 = (tile % mtiles) * BM, n0 = (tile / mtiles) * BN;
    const int ktiles = (K + BK - 1) / BK;
    const int kt0 = split * kt_per_split;
    const int kt1 = min(kt0 + kt_per_split, ktiles);
    const int nk = kt1 > kt0 ? kt1 - kt0 : 0;
    // whole turns of the ring in the loop, the last partial turn after it (a test inside the
    // loop's steps made the compiler wait for every load at each of them); the loads issued
    // for tiles past the split's last read zeros

    const __amdgpu_buffer_rsrc_t ra = make_rsrc(A, (uint32_t)((NPL - 1) * pstride * 2 + (int64_t)M * lda * 2));
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(W, (uint32_t)(TILED ? (int64_t)((N + 31) / 32) * ktiles * 4096 : (int64_t)N * ldw * 2));

    // masked input: DMA load t of this wave fills 1 KB = stage rows 8j..8j+7 (j = wave + NW t);
    // lane l writes unit 64j + l: row u / 8, slot u % 8 holding k chunk slot ^ (row & 7)
    uint32_t aoff[LA];
    int akc[LA];
#pragma unroll
    for (int t = 0; t < LA; ++t) {
        const int u = (wave + NW * t) * WAVE + lane;
        const int row = u >> 3, kc = (u & 7) ^ lds_swizzle<SW>(row);
        const int p = row / BM, r = row - p * BM, gm = m0 + r;
        akc[t] = kc * 8;
        aoff[t] = gm < M ? (uint32_t)((p * pstride + (int64_t)gm * lda) * 2 + kc * 16) : OOB;
    }
    // W: lane (c = l % 32, h = l / 32) loads row n0 + WTN wn + 32 j + c, 16 bytes at k = 16 s + 8 h;
    // tiled, that is byte 16 l of the k step's 1 KB in block ((n0 + WTN wn + 32 j) / 32, K tile)
    const int fc = lane % 32, fh = lane / 32;
    uint32_t woff[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int gn = n0 + wn * WTN + j * 32 + fc;
        if (TILED)
            woff[j] = gn < N ? (uint32_t)((int64_t)(gn / 32) * ktiles * 4096 + lane * 16) : OOB;
        else
            woff[j] = gn < N ? (uint32_t)((int64_t)gn * ldw * 2 + fh * 16) : OOB;
    }

    unsigned char* const st0 = stream_stage<0, SB>();
    unsigned char* const st1 = stream_stage<1, SB>();
    unsigned char* const st2 = S > 2 ? stream_stage<2, SB>() : st0;
    unsigned char* const st3 = S > 3 ? stream_stage<3, SB>() : st0;
    auto stage = [&](auto sc) -> unsigned char* {
        constexpr int q = decltype(sc)::value;
        return q == 0 ? st0 : q == 1 ? st1 : q == 2 ? st2 : st3;
    };

    uint4 wb[S][TN][4];
    // part `part` (0..3) of the loads of relative tile t into ring slot q: W of k step
    // `part` and a quarter of the masked-input DMA (the remainder with the last part)
    constexpr int LA4 = LA / 4;
    auto issue_part = [&](int t, auto sc, int part) {
        constexpr int q = decltype(sc)::value;
        const int kt = kt0 + t, kb = kt * BK;
        const bool live = kt < kt1;
        unsigned char* sb = stage(sc);
        const int i0 = part * LA4, i1 = part == 3 ? LA : i0 + LA4;
#pragma unroll
        for (int i = 0; i < LA; ++i) {
            if (i < i0 || i >= i1) continue;
            const uint32_t off = (live && aoff[i] != OOB && kb + akc[i] < K) ? aoff[i] + (uint32_t)kb * 2 : OOB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr_t)(sb + (wave + NW * i) * 1024), 16, (int)off, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            if (TILED) { // k past K is zero padding of the tiled layout
                const bool ok = live && woff[j] != OOB;
                wb[q][j][part] = load16(rw, ok ? woff[j] + (uint32_t)(kt * 4 + part) * 1024 : OOB);
            } else {
                const bool ok = live && woff[j] != OOB && kb + 16 * part + 8 * fh < K;
                wb[q][j][part] = load16(rw, ok ? woff[j] + (uint32_t)(kb + 16 * part) * 2 : OOB);
            }
        }
    };
    auto issue = [&](int t, auto sc) {
#pragma unroll
        for (int part = 0; part < 4; ++part) issue_part(t, sc, part);
    };

    f32x16_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x16_t{};

    // fragments of k step s: every row block i of the wave tile and plane p
    auto read_a = [&](const unsigned char* sb, int s, bf16x8_t (&a)[NPL][TM]) {
        const int kc = s * 2 + fh;
#pragma unroll
        for (int p = 0; p < NPL; ++p)
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int r = p * BM + wm * WTM + i * 32 + fc;
                a[p][i] = as_bf16x8(*reinterpret_cast<const uint4*>(sb + r * 128 + ((kc ^ lds_swizzle<SW>(r)) << 4)));
            }
    };
    // k step s + 1's fragments are read while step s is multiplied; the MFMAs of a
    // step run plane-major so that the TM x TN accumulators are updated round-robin
    // (consecutive MFMAs on one accumulator would wait for each other's results).
    // The loads of the tile D ahead (slot nq) are issued a quarter per k step,
    // interleaved with the MFMAs, so the matrix cores keep working while they issue.
    auto compute = [&](int t, auto sc, auto nsc) {
        constexpr int q = decltype(sc)::value;
        const unsigned char* sb = stage(sc);
        bf16x8_t a[2][NPL][TM];
        read_a(sb, 0, a[0]);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            if (s + 1 < 4) read_a(sb, s + 1, a[(s + 1) & 1]);
            issue_part(t + D, nsc, s);
#pragma unroll
            for (int p = 0; p < NPL; ++p)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s & 1][p][i], as_bf16x8(wb[q][j][s]), acc[i][j], 0, 0, 0);
            // one group: this step's fragment reads first, then MFMAs with the loads in between
            __builtin_amdgcn_sched_group_barrier(0x100, NPL * TM, 0);
#pragma unroll
            for (int g = 0; g < (LA + 3) / 4 + TN; ++g) {
                __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, NPL * TM * TN, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // one K tile in slot q: this wave's loads of the tile are in (the D - 1 younger
    // tiles may still be in flight), barrier (everyone's are, and slot q - 1 is no
    // longer read), multiply slot q while refilling slot q - 1 with tile t + D
    auto step = [&](int t, auto sc) {
        constexpr int q = decltype(sc)::value;
        wait_vmem<(D - 1) * (LA + LW)>();
        __builtin_amdgcn_s_barrier();
        compute(t, sc, std::integral_constant<int, (q + D) % S>{});
    };

    issue(0, std::integral_constant<int, 0>{});
    if constexpr (D > 1) issue(1, std::integral_constant<int, 1>{});
    if constexpr (D > 2) issue(2, std::integral_constant<int, 2>{});
    int t = 0;
    for (; t + S <= nk; t += S) {
        step(t, std::integral_constant<int, 0>{});
        step(t + 1, std::integral_constant<int, 1>{});
        if constexpr (S > 2) step(t + 2, std::integral_constant<int, 2>{});
        if constexpr (S > 3) step(t + 3, std::integral_constant<int, 3>{});
    }
    // the last, partial turn: at most S - 1 tiles, the same count for every wave
    if (t < nk) step(t, std::integral_constant<int, 0>{});
    if constexpr (S > 2) if (t + 1 < nk) step(t + 1, std::integral_constant<int, 1>{});
    if constexpr (S > 3) if (t + 2 < nk) step(t + 2, std::integral_constant<int, 2>{});
    wait_vmem<0>(); // the loads issued past the last tile (zeros) have landed before the workgroup ends

    if (ksplit == 1) {
        store_tile<TM, TN>(acc, C, ldc, Out, ldo, M, N, m0 + wm * WTM, n0 + wn * WTN, fc, fh);
        return;
    }
    // partial in register order: float4 c of block (i, j) of lane l at ((i TN + j) 4 + c) 64 + l
    float4* mp = reinterpret_cast<float4*>(part) + (((int64_t)tile * ksplit + split) * NW + wave) * (TM * TN * 4 * 64);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int c = 0; c < 4; ++c)
                mp[((i * TN + j) * 4 + c) * 64 + lane] =
                    make_float4(acc[i][j][4 * c], acc[i][j][4 * c + 1], acc[i][j][4 * c + 2], acc[i][j][4 * c + 3]);
}

// The W-streamed kernel with the masked input formed in the kernel (64-row tiles,
// tiled W): for a mask eta drawn ahead, each thread loads 8 consecutive float32 of X
// and of eta of one row two K tiles ahead and, after the current tile's MFMAs, forms
// the next tile's fl32(X + eta), splits it into the NPL bfloat16 planes (the mask
// kernel's split, so the planes are the same bits) and writes them into the swizzled
// LDS stage the buffer-load-to-LDS fills in gemm_stream_kernel; W streams into
// registers D tiles ahead as there.  This saves
// the separate mask launch (and its planes' round trip through memory) where the
// masked input is read by few column tiles: up to 128 tokens.
template <int NPL, int BM, int BN, int WGM, int D, int NW>
__global__ void __launch_bounds__(NW * WAVE)
gemm_stream_masked_kernel(const float* __restrict__ X, int64_t ldx, const float* __restrict__ E, int64_t lde,
                          const uint16_t* __restrict__ W, const float* __restrict__ C, int64_t ldc,
                          float* __restrict__ Out, int64_t ldo, int M, int N, int K, int mtiles, int ntiles,
                          int ksplit, int kt_per_split, float* __restrict__ part)
{
    constexpr int WGN = NW / WGM;
    constexpr int WTM = BM / WGM, WTN = BN / WGN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    constexpr int S = D + 1;
    constexpr int SB = NPL * BM * 128;        // LDS bytes per stage
    constexpr int LW = 4 * TN;                // W loads per wave per tile
    static_assert(WGM * WGN == NW && TM * 32 * WGM == BM && TN * 32 * WGN == BN, "wave tile");
    static_assert(BM * 8 == NW * WAVE, "one 8-element unit of the masked input per thread");
    static_assert(S >= 3 && S <= 4 && (D - 1) * LW + 4 < 64, "stages");

    const int tid = threadIdx.x, lane = tid % WAVE;
    const int wave = __builtin_amdgcn_readfirstlane(tid / WAVE);
    const int wm = wave / WGN, wn = wave % WGN;
    const uint32_t lb = splitee::xcd_logical_block(blockIdx.x, gridDim.x);
    const int tiles = mtiles * ntiles;
    const int split = (int)lb / tiles, tile = (int)lb % tiles;
    const int m0 = (tile % mtiles) * BM, n0 = (tile / mtiles) * BN;
    const int ktiles = (K + BK - 1) / BK;
    const int kt0 = split * kt_per_split;
    const int kt1 = min(kt0 + kt_per_split, ktiles);
    const int nk = kt1 > kt0 ? kt1 - kt0 : 0;

    const __amdgpu_buffer_rsrc_t rx = make_rsrc(X, (uint32_t)((int64_t)M * ldx * 4));
    const __amdgpu_buffer_rsrc_t re = make_rsrc(E, (uint32_t)((int64_t)M * lde * 4));
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(W, (uint32_t)((int64_t)((N + 31) / 32) * ktiles * 4096));

    // this thread's unit: row ur of the tile, 8 k from 8 uc of every K tile
    const int ur = tid >> 3, uc = tid & 7;
    const int gm = m0 + ur;
    const uint32_t xoff = gm < M ? (uint32_t)(((int64_t)gm * ldx + uc * 8) * 4) : OOB;
    const uint32_t eoff = gm < M ? (uint32_t)(((int64_t)gm * lde + uc * 8) * 4) : OOB;
    const int wslot = (uc ^ lds_swizzle<1>(ur)) << 4; // the unit's 16-byte slot in each plane row
    const int fc = lane % 32, fh = lane / 32;
    uint32_t woff[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int gn = n0 + wn * WTN + j * 32 + fc;
        woff[j] = gn < N ? (uint32_t)((int64_t)(gn / 32) * ktiles * 4096 + lane * 16) : OOB;
    }

    unsigned char* const st0 = stream_stage<0, SB>();
    unsigned char* const st1 = stream_stage<1, SB>();
    unsigned char* const st2 = stream_stage<2, SB>();
    unsigned char* const st3 = S > 3 ? stream_stage<3, SB>() : st0;
    auto stage = [&](auto sc) -> unsigned char* {
        constexpr int q = decltype(sc)::value;
        return q == 0 ? st0 : q == 1 ? st1 : q == 2 ? st2 : st3;
    };

    uint4 xr[2], er[2];
    auto load_x = [&](int t) { // X and eta of relative tile t into registers (zeros past K or M)
        const int kt = kt0 + t, kb = kt * BK;
        const bool ok = kt < kt1 && kb + uc * 8 < K;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            xr[h] = load16(rx, ok && xoff != OOB ? xoff + (uint32_t)(kb * 4 + 16 * h) : OOB);
            er[h] = load16(re, ok && eoff != OOB ? eoff + (uint32_t)(kb * 4 + 16 * h) : OOB);
        }
    };
    auto write_x = [&](auto sc) { // fl32(X + eta), split, into the stage's plane rows
        unsigned char* sb = stage(sc);
        float x[8];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const float4 a = __builtin_bit_cast(float4, xr[h]), b = __builtin_bit_cast(float4, er[h]);
            x[4 * h + 0] = a.x + b.x;
            x[4 * h + 1] = a.y + b.y;
            x[4 * h + 2] = a.z + b.z;
            x[4 * h + 3] = a.w + b.w;
        }
        uint4 q[NPL];
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            if (NPL == 1) {
                reinterpret_cast<uint32_t*>(&q[0])[h] = splitee::bf16x2_rne(x[2 * h], x[2 * h + 1]);
            } else {
                splitee::split3_bf16x2(x[2 * h], x[2 * h + 1], reinterpret_cast<uint32_t*>(&q[0])[h],
                                       reinterpret_cast<uint32_t*>(&q[1])[h], reinterpret_cast<uint32_t*>(&q[2])[h]);
            }
        }
#pragma unroll
        for (int p = 0; p < NPL; ++p)
            *reinterpret_cast<uint4*>(sb + (p * BM + ur) * 128 + wslot) = q[p];
    };

    uint4 wb[S][TN][4];
    auto issue_w = [&](int t, auto sc, int part) {
        constexpr int q = decltype(sc)::value;
        const int kt = kt0 + t;
        const bool live = kt < kt1;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const bool ok = live && woff[j] != OOB;
            wb[q][j][part] = load16(rw, ok ? woff[j] + (uint32_t)(kt * 4 + part) * 1024 : OOB);
        }
    };

    f32x16_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x16_t{};

    auto read_a = [&](const unsigned char* sb, int s, bf16x8_t (&a)[NPL][TM]) {
        const int kc = s * 2 + fh;
#pragma unroll
        for (int p = 0; p < NPL; ++p)
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int r = p * BM + wm * WTM + i * 32 + fc;
                a[p][i] = as_bf16x8(*reinterpret_cast<const uint4*>(sb + r * 128 + ((kc ^ lds_swizzle<1>(r)) << 4)));
            }
    };
    // step t: barrier (tile t's stage, written at the end of step t - 1, is complete
    // everywhere, and stage t - 1 is no longer read), multiply tile t from W slot t while
    // W of tile t + D is issued, then the masked input of tile t + 1 (its X and eta loaded
    // at the end of step t - 1) goes into its stage and the X and eta of tile t + 2 are
    // issued.  Loads complete in order: at that wait only W of tile t + D is younger than
    // tile t + 1's X and eta.  Stage t + 1 was last read at step t + 1 - S <= t - 2, which
    // every wave finished before this step's barrier.
    auto step = [&](int t, auto sc) {
        constexpr int q = decltype(sc)::value;
        __builtin_amdgcn_s_barrier();
        const unsigned char* sb = stage(sc);
        bf16x8_t a[2][NPL][TM];
        read_a(sb, 0, a[0]);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            if (s + 1 < 4) read_a(sb, s + 1, a[(s + 1) & 1]);
            issue_w(t + D, std::integral_constant<int, (q + D) % S>{}, s);
#pragma unroll
            for (int p = 0; p < NPL; ++p)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s & 1][p][i], as_bf16x8(wb[q][j][s]), acc[i][j], 0, 0, 0);
        }
        wait_vmem<LW>();
        write_x(std::integral_constant<int, (q + 1) % S>{});
        load_x(t + 2);
        __builtin_amdgcn_s_waitcnt((0 << 8) | (7 << 4) | 15 | (3 << 14)); // lgkmcnt(0): this wave's LDS writes done
    };

    // prologue: tile 0's masked input into stage 0, W of tiles 0 .. D - 1 and tile 1's X
    // and eta issued, W of tile 0 landed (the younger loads may be in flight)
    load_x(0);
#pragma unroll
    for (int part = 0; part < 4; ++part) issue_w(0, std::integral_constant<int, 0>{}, part);
    wait_vmem<LW>();
    write_x(std::integral_constant<int, 0>{});
#pragma unroll
    for (int part = 0; part < 4; ++part) issue_w(1, std::integral_constant<int, 1>{}, part);
    if constexpr (D > 2) {
#pragma unroll
        for (int part = 0; part < 4; ++part) issue_w(2, std::integral_constant<int, 2>{}, part);
    }
    load_x(1);
    wait_vmem<(D - 1) * LW + 4>();
    __builtin_amdgcn_s_waitcnt((0 << 8) | (7 << 4) | 15 | (3 << 14));
    // whole turns of the ring, then the last partial turn (at most S - 1 tiles)
    int t = 0;
    for (; t + S <= nk; t += S) {
        step(t, std::integral_constant<int, 0>{});
        step(t + 1, std::integral_constant<int, 1>{});
        step(t + 2, std::integral_constant<int, 2>{});
        if constexpr (S > 3) step(t + 3, std::integral_constant<int, 3>{});
    }
    if (t < nk) step(t, std::integral_constant<int, 0>{});
    if (t + 1 < nk) step(t + 1, std::integral_constant<int, 1>{});
    if constexpr (S > 3) if (t + 2 < nk) step(t + 2, std::integral_constant<int, 2>{});
    wait_vmem<0>();

    if (ksplit == 1) {
        store_tile<TM, TN>(acc, C, ldc, Out, ldo, M, N, m0 + wm * WTM, n0 + wn * WTN, fc, fh);
        return;
    }
    float4* mp = reinterpret_cast<float4*>(part) + (((int64_t)tile * ksplit + split) * NW + wave) * (TM * TN * 4 * 64);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int c = 0; c < 4; ++c)
                mp[((i * TN + j) * 4 + c) * 64 + lane] =
                    make_float4(acc[i][j][4 * c], acc[i][j][4 * c + 1], acc[i][j][4 * c + 2], acc[i][j][4 * c + 3]);
}

// Sums the split-K partials of gemm_stream_kernel in split order and applies the
// unmask epilogue.  Thread u handles one float4 of one wave's partial (the
// register order the partials were written in): rows 8 c + 4 (l / 32) + 0..3 of
// block (i, j), column l % 32.
template <int BM, int BN, int WGM, int WGN>
__global__ void __launch_bounds__(256)
stream_sum_kernel(const float* __restrict__ part, int ksplit, const float* __restrict__ C, int64_t ldc,
                  float* __restrict__ Out, int64_t ldo, int M, int N, int mtiles, int tiles)
{
    constexpr int NW = WGM * WGN, WTM = BM / WGM, WTN = BN / WGN, TM = WTM / 32, TN = WTN / 32;
    constexpr int PER_WAVE = TM * TN * 4 * 64; // float4 units
    const int64_t total = (int64_t)tiles * NW * PER_WAVE;
    const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (u >= total) return;
    const int tile = (int)(u / (NW * PER_WAVE));
    const int rem = (int)(u - (int64_t)tile * NW * PER_WAVE);
    const int wave = rem / PER_WAVE, e = rem - wave * PER_WAVE;
    const int lane = e % 64, ijc = e / 64, c = ijc % 4, ij = ijc / 4, i = ij / TN, j = ij % TN;
    const int m0 = (tile % mtiles) * BM, n0 = (tile / mtiles) * BN;
    const int wm = wave / WGN, wn = wave % WGN;
    const int col = n0 + wn * WTN + j * 32 + lane % 32;
    const int row0 = m0 + wm * WTM + i * 32 + 8 * c + 4 * (lane / 32);
    // C first, then every split's partial: all loads in flight together (an element outside
    // M x N loads C[0], so no load sits behind a branch of its own)
    float cv[4] = {0.f, 0.f, 0.f, 0.f};
    if (C) {
#pragma unroll
        for (int r = 0; r < 4; ++r) cv[r] = C[row0 + r < M && col < N ? (int64_t)(row0 + r) * ldc + col : 0];
    }
    // the partials through a buffer resource: a split past ksplit takes an out-of-range offset
    // and reads zeros, so every load is unconditional (a load behind a branch of its own made
    // the compiler wait for the loads before it); the host keeps the partials below 2 GB
    const __amdgpu_buffer_rsrc_t rp = make_rsrc(part, (uint32_t)((int64_t)tiles * ksplit * NW * PER_WAVE * 16));
    const uint32_t off0 = (uint32_t)((((int64_t)tile * ksplit * NW + wave) * PER_WAVE + e) * 16);
    f32x4_t v[ST_MAX_KS];
#pragma unroll
    for (int q = 0; q < ST_MAX_KS; ++q)
        v[q] = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                   rp, (int)(q < ksplit ? off0 + (uint32_t)(q * NW * PER_WAVE * 16) : OOB), 0, 0));
    f32x4_t sum = v[0];
#pragma unroll
    for (int q = 1; q < ST_MAX_KS; ++q)
        if (q < ksplit) sum += v[q];
    if (col >= N) return;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int row = row0 + r;
        if (row < M) {
            float y = sum[r];
            if (C) y = y - cv[r];
            Out[(int64_t)row * ldo + col] = y;
        }
    }
}

// --------------------------------------------------------------- f32 MFMA
// v_mfma_f32_16x16x4_f32 takes one k per lane group; four instructions cover a
// 16-wide k slice whose elements are assigned so that each lane reads one
// 16-byte run (k = 4 * (lane/16) + j in instruction j), identically for A and W.

template <int BM, int BN, int BK, int WGM, int WGN, bool WBF16>
__global__ void __launch_bounds__(WGM * WGN * WAVE)
gemm_f32_kernel(const float* __restrict__ A, int64_t lda, const void* __restrict__ Wv, int64_t ldw,
                const float* __restrict__ C, int64_t ldc, float* __restrict__ Out, int64_t ldo, int M,
                int N, int K, int mtiles, int ntiles, int ksplit, int kt_per_split,
                float* __restrict__ part, unsigned* __restrict__ counters)
{
    constexpr int NT = WGM * WGN * WAVE;
    constexpr int LDK = BK + 4;
    constexpr int WTM = BM / WGM, WTN = BN / WGN;
    constexpr int TM = WTM / 16, TN = WTN / 16;
    constexpr int CPR = BK / 4;                  // 16-byte float chunks per row
    constexpr int WCPR = WBF16 ? BK / 8 : BK / 4; // 16-byte W chunks per row
    constexpr int ACH = BM * CPR / NT, BCH = BN * WCPR / NT;
    static_assert(ACH * NT == BM * CPR && BCH * NT == BN * WCPR, "tile/thread mismatch");
    static_assert(BK % 16 == 0, "k tile");

    __shared__ __attribute__((aligned(16))) float sA[BM * LDK];
    __shared__ __attribute__((aligned(16))) float sB[BN * LDK];

    const int tid = threadIdx.x, lane = tid % WAVE, wave = tid / WAVE;
    const int wm = wave % WGM, wn = wave / WGM;
    const uint32_t lb = splitee::xcd_logical_block(blockIdx.x, gridDim.x);
    const int tiles = mtiles * ntiles;
    const int split = (int)lb / tiles, tile = (int)lb % tiles;
    const int m0 = (tile % mtiles) * BM, n0 = (tile / mtiles) * BN;
    const int ktiles = (K + BK - 1) / BK;
    const int kt0 = split * kt_per_split;
    const int kt1 = min(kt0 + kt_per_split, ktiles);

    uint4 ra[ACH], rb[BCH];
    auto gload = [&](int kt) {
        const int kb = kt * BK;
#pragma unroll
        for (int c = 0; c < ACH; ++c) {
            const int idx = tid + c * NT, row = idx / CPR, col = (idx % CPR) * 4;
            const int gm = m0 + row, gk = kb + col;
            ra[c] = (gm < M && gk < K) ? *reinterpret_cast<const uint4*>(A + (int64_t)gm * lda + gk)
                                       : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int c = 0; c < BCH; ++c) {
            const int idx = tid + c * NT, row = idx / WCPR, col = (idx % WCPR) * (WBF16 ? 8 : 4);
            const int gn = n0 + row, gk = kb + col;
            const bool ok = gn < N && gk < K;
            if (WBF16)
                rb[c] = ok ? *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(Wv) + (int64_t)gn * ldw + gk)
                           : make_uint4(0, 0, 0, 0);
            else
                rb[c] = ok ? *reinterpret_cast<const uint4*>(reinterpret_cast<const float*>(Wv) + (int64_t)gn * ldw + gk)
                           : make_uint4(0, 0, 0, 0);
        }
    };
    auto swrite = [&]() {
#pragma unroll
        for (int c = 0; c < ACH; ++c) {
            const int idx = tid + c * NT, row = idx / CPR, col = (idx % CPR) * 4;
            *reinterpret_cast<uint4*>(&sA[row * LDK + col]) = ra[c];
        }
#pragma unroll
        for (int c = 0; c < BCH; ++c) {
            const int idx = tid + c * NT, row = idx / WCPR, col = (idx % WCPR) * (WBF16 ? 8 : 4);
            if (WBF16) {
                // bfloat16 -> float32 is exact: the 16 bits become the upper half
                const uint4 v = rb[c];
                uint4 lo = make_uint4(v.x << 16, v.x & 0xFFFF0000u, v.y << 16, v.y & 0xFFFF0000u);
                uint4 hi = make_uint4(v.z << 16, v.z & 0xFFFF0000u, v.w << 16, v.w & 0xFFFF0000u);
                *reinterpret_cast<uint4*>(&sB[row * LDK + col]) = lo;
                *reinterpret_cast<uint4*>(&sB[row * LDK + col + 4]) = hi;
            } else {
                *reinterpret_cast<uint4*>(&sB[row * LDK + col]) = rb[c];
            }
        }
    };

    f32x4_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const int frow = lane % 16, fk = (lane / 16) * 4;
    if (kt0 < kt1) gload(kt0);
    for (int kt = kt0; kt < kt1; ++kt) {
        __syncthreads();
        swrite();
        __syncthreads();
        if (kt + 1 < kt1) gload(kt + 1);
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            float4 af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                af[i] = *reinterpret_cast<const float4*>(&sA[(wm * WTM + i * 16 + frow) * LDK + ks * 16 + fk]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                bfr[j] = *reinterpret_cast<const float4*>(&sB[(wn * WTN + j * 16 + frow) * LDK + ks * 16 + fk]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i].x, bfr[j].x, acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i].y, bfr[j].y, acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i].z, bfr[j].z, acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i].w, bfr[j].w, acc[i][j], 0, 0, 0);
                }
        }
    }

    const int erow = 4 * (lane / 16), ecol = lane % 16;
    if (ksplit == 1) {
        // every C load of the wave tile before the first subtraction (one wait, not one per
        // element); elements outside M x N load C[0] and store nothing
        float cv[TM][TN][4];
        if (C) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int row = m0 + wm * WTM + i * 16 + erow + r, col = n0 + wn * WTN + j * 16 + ecol;
                        cv[i][j][r] = C[row < M && col < N ? (int64_t)row * ldc + col : 0];
                    }
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = m0 + wm * WTM + i * 16 + erow + r, col = n0 + wn * WTN + j * 16 + ecol;
                    if (row < M && col < N)
                        Out[(int64_t)row * ldo + col] = C ? acc[i][j][r] - cv[i][j][r] : acc[i][j][r];
                }
        return;
    }
    float* mypart = part + ((int64_t)tile * ksplit + split) * (BM * BN);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                store_partial(&mypart[(wm * WTM + i * 16 + erow + r) * BN + wn * WTN + j * 16 + ecol], acc[i][j][r]);
    if (!splitk_arrive(counters + tile, ksplit, reinterpret_cast<unsigned*>(sA))) return;
    splitk_reduce<BM, BN, WGM * WGN * WAVE, (BM * BN / 4 / (WGM * WGN * WAVE) < 8 ? BM * BN / 4 / (WGM * WGN * WAVE) : 8)>(part + (int64_t)tile * ksplit * (BM * BN), ksplit, m0, n0, M, N, C,
                                          ldc, Out, ldo);
    if (tid == 0) splitk_reset(counters + tile);
}

// --------------------------------------------------------- skinny (M <= 16)
// Decode-shaped GEMM, bound by the single pass over W.  A workgroup owns 64
// output columns (4 waves x 16) and a range of 32-wide k steps; the number of
// k splits is the largest that keeps the grid within one round of two
// workgroups per CU.  The workgroup's slice of the masked input (the M <= 16
// rows, every plane, this k range) is copied to LDS once; its loads are issued
// before W's so that they do not queue behind them.  W is streamed from HBM
// straight into MFMA operand registers through a ring of R k steps per lane.
// Split-K partials cover rows < M only and are summed in split order by the last
// workgroup of the tile to arrive.

constexpr int SK_BN = 64;
// The planner deals the k steps out in granules of SK_RING (a split fills at least one, the
// LDS slice is sized for whole granules); the kernel's W ring is shallower: 4 k steps per
// lane up to 8 rows, 8 above (sk_ring).  Against a 16-step ring with the same splits, the
// four Qwen3-4B projections of a decode step took 11-12% less time at 3-4 rows, 9% at 8, 7-8%
// at 12-16 (same results): the deep ring's 16 KB per wave of W in flight bought no bandwidth.
constexpr int SK_RING = 16;
constexpr int sk_ring(int64_t M) { return M <= 8 ? 4 : 8; }
constexpr int SK_LDS_MAX = 64 * 1024; // masked-input slice per workgroup (two workgroups per CU)
constexpr int SK_TARGET_WGS = 512;
constexpr int SK_CP = SK_LDS_MAX / 16 / 256; // slice units per thread (16 at 64 KB)

// Where the skinny kernel's masked input comes from: NPL bfloat16 planes A
// (plane p at A + p * pstride), or (MASK) float32 X and mask eta, from which the
// kernel forms fl32(X + eta) and its planes itself.
struct SkSrc {
    const uint16_t* A; int64_t lda, pstride;
    const float* X; int64_t ldx;
    const float* eta; int64_t ld_eta;
};

// Masked-input units (8 float32 of X and of eta) per thread per load round of the skinny
// kernel when it forms the mask: 2 up to 8 rows, 4 above, so that at 16 rows and 16 k steps
// per split the whole slice is requested before the W ring (a round issued after the ring
// waits for all of it, since a wave's loads complete in order).  Measured on the Qwen3-4B
// projections: 4 per round made 16 rows 4.8% faster and 4 rows 3.7% slower.
constexpr int SK_MCP_SMALL = 2, SK_MCP_LARGE = 4;

template <int NPL>
__device__ __forceinline__ void planes_of(const float (&x)[8], uint4 (&q)[NPL])
{
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        if (NPL == 1) {
            reinterpret_cast<uint32_t*>(&q[0])[h] = splitee::bf16x2_rne(x[2 * h], x[2 * h + 1]);
        } else {
            splitee::split3_bf16x2(x[2 * h], x[2 * h + 1], reinterpret_cast<uint32_t*>(&q[0])[h],
                                   reinterpret_cast<uint32_t*>(&q[1])[h], reinterpret_cast<uint32_t*>(&q[2])[h]);
        }
    }
}

template <int NPL, int R, bool MASK, bool TILED = false, int MCP = SK_MCP_SMALL>
__global__ void __launch_bounds__(256)
skinny_kernel(SkSrc src, const uint16_t* __restrict__ W, int64_t ldw, const float* __restrict__ C, int64_t ldc,
              float* __restrict__ Out, int64_t ldo, int M, int N, int K, int ntiles, int ksplit,
              int steps_per_split, float* __restrict__ part, unsigned* __restrict__ counters)
{
    static_assert(R >= 2 && R % 2 == 0 && R <= SK_RING, "W ring: whole pairs of k steps, within the planner's granule");
    extern __shared__ __attribute__((aligned(16))) unsigned char sa[];
    const int tid = threadIdx.x, lane = tid % WAVE;
    const int wave = __builtin_amdgcn_readfirstlane(tid / WAVE);
    const uint32_t lb = splitee::xcd_logical_block(blockIdx.x, gridDim.x);
    const int split = (int)lb / ntiles, tile = (int)lb % ntiles;
    const int n0 = tile * SK_BN;
    const int ksteps = (K + 31) / 32;
    const int s0 = split * steps_per_split;
    const int ns = max(min(s0 + steps_per_split, ksteps) - s0, 0);
    const int SA = (steps_per_split + R - 1) / R * R; // steps held in LDS (zero past ns)
    const int RS = SA * 64 + 16;                      // LDS row pitch; 16 bytes of padding
    const int fr = lane % 16, fq = lane / 16;

    // the W ring.  Lane (r, q) loads row gn = n0 + 16 wave + r, 16 bytes at k = 32 J + 8 q
    // of k step J.  Tiled (32-row blocks of 64-k tiles, 1 KB per 16-k step, 16 bytes per
    // (k half h, row c) at (32 h + c) 16), that chunk sits at block (gn / 32, J / 2),
    // step 2 (J % 2) + q / 2, half q % 2: a constant per lane plus 2048 J, and the 64 lanes
    // read four 256-byte runs (whole cache lines)
    const int gn = n0 + wave * 16 + fr;
    const int kt64 = (K + 63) / 64;
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(W, (uint32_t)(TILED ? (int64_t)((N + 31) / 32) * kt64 * 4096 : (int64_t)N * ldw * 2));
    const uint32_t wbase = gn >= N ? OOB
                           : TILED ? (uint32_t)((int64_t)(gn / 32) * kt64 * 4096 + (fq / 2) * 1024 +
                                                ((fq % 2) * 32 + gn % 32) * 16)
                                   : (uint32_t)((int64_t)gn * ldw * 2 + fq * 16);
    auto wload = [&](int j) {
        const bool ok = wbase != OOB && j < ns && (s0 + j) * 32 + fq * 8 < K;
        return load16(rw, ok ? wbase + (uint32_t)(s0 + j) * (TILED ? 2048 : 64) : OOB);
    };
    uint4 ring[R];

    if constexpr (!MASK) {
        // 1. slice loads: plane p, row r < M, 16-byte unit c of the row's SA * 64 bytes
        const int upr = SA * 4, units = NPL * M * upr;
        uint4 av[SK_CP];
        const __amdgpu_buffer_rsrc_t ra =
            make_rsrc(src.A, (uint32_t)((NPL - 1) * src.pstride * 2 + (int64_t)M * src.lda * 2));
#pragma unroll
        for (int i = 0; i < SK_CP; ++i) {
            const int u = i * 256 + tid;
            const int pr = u / upr, c = u - pr * upr;
            const int p = pr / M, r = pr - p * M;
            const int k = s0 * 32 + c * 8;
            const bool ok = u < units && c < ns * 4 && k < K;
            av[i] = load16(ra, ok ? (uint32_t)((p * src.pstride + (int64_t)r * src.lda + k) * 2) : OOB);
        }
        // 2. the ring, queued behind the slice
#pragma unroll
        for (int u = 0; u < R; ++u) ring[u] = wload(u);
        // 3. slice to LDS (waits for the slice loads only: loads complete in order)
#pragma unroll
        for (int i = 0; i < SK_CP; ++i) {
            const int u = i * 256 + tid;
            if (u < units) {
                const int pr = u / upr, c = u - pr * upr;
                *reinterpret_cast<uint4*>(sa + pr * RS + c * 16) = av[i];
            }
        }
    } else {
        // 1-3 with the mask formed here: unit c of row r is 8 float32 of X and of
        // eta at k = s0 * 32 + 8 c; the unit's fl32(X + eta) is split into the NPL
        // planes and stored where the plane form would have put it.  The first
        // round's loads go out before the ring, the rest after it.
        const int upr = SA * 4, units = M * upr;
        const __amdgpu_buffer_rsrc_t rx = make_rsrc(src.X, (uint32_t)((int64_t)M * src.ldx * 4));
        const __amdgpu_buffer_rsrc_t re = make_rsrc(src.eta, (uint32_t)((int64_t)M * src.ld_eta * 4));
        auto unit_ok = [&](int u, int& r, int& c, int& k) {
            r = u / upr;
            c = u - r * upr;
            k = s0 * 32 + c * 8;
            return u < units && c < ns * 4 && k < K;
        };
        auto round_load = [&](int base, uint4 (&xv)[MCP][2], uint4 (&ev)[MCP][2]) {
#pragma unroll
            for (int i = 0; i < MCP; ++i) {
                int r, c, k;
                const bool ok = unit_ok(base + i * 256 + tid, r, c, k);
                const uint32_t ox = ok ? (uint32_t)(((int64_t)r * src.ldx + k) * 4) : OOB;
                const uint32_t oe = ok ? (uint32_t)(((int64_t)r * src.ld_eta + k) * 4) : OOB;
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    ev[i][h] = load16(re, oe == OOB ? OOB : oe + 16 * h);
                    xv[i][h] = load16(rx, ox == OOB ? OOB : ox + 16 * h);
                }
            }
        };
        auto round_store = [&](int base, const uint4 (&xv)[MCP][2], const uint4 (&ev)[MCP][2]) {
#pragma unroll
            for (int i = 0; i < MCP; ++i) {
                const int u = base + i * 256 + tid;
                if (u < units) {
                    const int r = u / upr, c = u - r * upr;
                    float x[8];
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const float4 e = __builtin_bit_cast(float4, ev[i][h]);
                        const float4 v = __builtin_bit_cast(float4, xv[i][h]);
                        x[4 * h + 0] = v.x + e.x;
                        x[4 * h + 1] = v.y + e.y;
                        x[4 * h + 2] = v.z + e.z;
                        x[4 * h + 3] = v.w + e.w;
                    }
                    uint4 q[NPL];
                    planes_of<NPL>(x, q);
#pragma unroll
                    for (int p = 0; p < NPL; ++p)
                        *reinterpret_cast<uint4*>(sa + (p * M + r) * RS + c * 16) = q[p];
                }
            }
        };
        uint4 xv[MCP][2], ev[MCP][2];
        round_load(0, xv, ev);
#pragma unroll
        for (int u = 0; u < R; ++u) ring[u] = wload(u);
        round_store(0, xv, ev);
        for (int base = MCP * 256; base < units; base += MCP * 256) {
            round_load(base, xv, ev);
            round_store(base, xv, ev);
        }
    }
    __syncthreads();

    // 4. stream: fragments of step j + 1 are read while step j is multiplied; two
    // accumulator chains (even / odd steps) so consecutive MFMAs are independent
    const bool arow = fr < M;
    auto read_a = [&](int j, bf16x8_t (&a)[NPL]) {
        const int jj = min(j, SA - 1);
#pragma unroll
        for (int p = 0; p < NPL; ++p)
            a[p] = arow ? as_bf16x8(*reinterpret_cast<const uint4*>(sa + (p * M + fr) * RS + jj * 64 + fq * 16))
                        : as_bf16x8(make_uint4(0, 0, 0, 0));
    };
    f32x4_t acc2[2] = {f32x4_t{0.f, 0.f, 0.f, 0.f}, f32x4_t{0.f, 0.f, 0.f, 0.f}};
    bf16x8_t a[2][NPL];
    read_a(0, a[0]);
    const int nloop = (ns + R - 1) / R * R;
    for (int j = 0; j < nloop; j += R) {
#pragma unroll
        for (int u = 0; u < R; ++u) {
            read_a(j + u + 1, a[(u + 1) & 1]);
#pragma unroll
            for (int p = 0; p < NPL; ++p)
                acc2[u & 1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u & 1][p], as_bf16x8(ring[u]), acc2[u & 1], 0, 0, 0);
            ring[u] = wload(j + u + R);
        }
    }
    const f32x4_t acc = acc2[0] + acc2[1];

    // 5. epilogue.  Accumulator element r: row 4*(lane/16) + r, column gn.
    const int erow = 4 * (lane / 16);
    if (ksplit == 1) {
        // the four C loads first, then the stores (one wait, not one per element)
        float cv[4] = {0.f, 0.f, 0.f, 0.f};
        if (C) {
#pragma unroll
            for (int r = 0; r < 4; ++r) cv[r] = C[erow + r < M && gn < N ? (int64_t)(erow + r) * ldc + gn : 0];
        }
#pragma unroll
        for (int r = 0; r < 4; ++r)
            if (erow + r < M && gn < N) Out[(int64_t)(erow + r) * ldo + gn] = C ? acc[r] - cv[r] : acc[r];
        return;
    }
    float* mypart = part + ((int64_t)tile * ksplit + split) * (16 * SK_BN);
#pragma unroll
    for (int r = 0; r < 4; ++r)
        if (erow + r < M) store_partial(&mypart[(erow + r) * SK_BN + wave * 16 + fr], acc[r]);
    if (!splitk_arrive(counters + tile, ksplit, reinterpret_cast<unsigned*>(sa))) return;

    // last workgroup: thread t sums the float4 at row t / 16, columns 4 * (t % 16)..+3
    // over the splits in split order, eight splits' loads in flight at a time; its C
    // float4 is loaded first, so that it arrives with the partials
    const int row = tid / 16, c4 = (tid % 16) * 4;
    if (row < M) {
        const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc(
            part + (int64_t)tile * ksplit * (16 * SK_BN), (short)0, ksplit * 16 * SK_BN * 4, 0x00020000);
        const int gc = n0 + c4;
        f32x4_t cv = f32x4_t{0.f, 0.f, 0.f, 0.f};
        if (C && gc + 4 <= N) cv = __builtin_bit_cast(f32x4_t, *reinterpret_cast<const float4*>(C + (int64_t)row * ldc + gc));
        f32x4_t sum = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int q0 = 0; q0 < ksplit; q0 += 8) {
            f32x4_t v[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const uint32_t off = q0 + i < ksplit ? (uint32_t)(((q0 + i) * 16 * SK_BN + row * SK_BN + c4) * 4) : OOB_OFF;
                v[i] = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rp, (int)off, 0, SC1));
            }
#pragma unroll
            for (int i = 0; i < 8; ++i)
                if (q0 + i < ksplit) sum = (q0 + i == 0) ? v[i] : sum + v[i];
        }
        if (gc + 4 <= N) {
            if (C) sum -= cv;
            *reinterpret_cast<float4*>(Out + (int64_t)row * ldo + gc) = __builtin_bit_cast(float4, sum);
        } else {
            for (int e = 0; e < 4 && gc + e < N; ++e) {
                float y = sum[e];
                if (C) y = y - C[(int64_t)row * ldc + gc + e];
                Out[(int64_t)row * ldo + gc + e] = y;
            }
        }
    }
    if (tid == 0) splitk_reset(counters + tile);
}

// ---------------------------------------------------------------- GEMV (M <= 2)
// Decode with one or two tokens is a matrix-vector product bound by the single
// pass over W, so it runs on the vector ALUs: a wave owns `ppw` consecutive pairs
// of W rows (output columns) and the whole of K, so no K split and no hand-off
// between workgroups is needed; the grid is at most two workgroups per CU and
// the W ring runs on across a wave's row pairs.  The workgroup first writes the masked
// input x~ (M x K float32) to LDS: fl32(X + eta), or the sum of its bfloat16
// planes (exact: the planes split a float32 exactly), rounded to bfloat16 for the
// single-plane precision.  The W loads of the first GV_RING chunks are issued
// before the masked-input loads, so that the two latencies overlap (loads
// complete in order).  Lane l then streams k = 512 j + 8 l .. + 7 of its rows
// (16-byte loads, GV_RING chunks in flight), accumulates fma(x~, w, acc) in
// float32 in k order, and the wave sums its lanes with a fixed butterfly.

constexpr int GV_WAVES = 4;  // waves per workgroup
constexpr int GV_NR = 2;     // W rows per wave
constexpr int GV_RING = 8;   // 512-k chunks per row in flight
constexpr int GV_XR = 2;     // masked-input units (8 k) per thread per load round
constexpr int GV_MMAX = 2;   // largest M
constexpr int GV_MAX_WGS = 1024; // four workgroups per CU

__device__ __forceinline__ float gv_wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, WAVE);
    return v;
}

template <int NPL, bool MASK, int MR>
__global__ void __launch_bounds__(GV_WAVES * WAVE)
gemv_kernel(SkSrc src, const uint16_t* __restrict__ W, int64_t ldw, const float* __restrict__ C, int64_t ldc,
            float* __restrict__ Out, int64_t ldo, int N, int K, int ppw)
{
    extern __shared__ __attribute__((aligned(16))) float xs[]; // MR x K
    constexpr int NT = GV_WAVES * WAVE;
    const int tid = threadIdx.x, lane = tid % WAVE;
    const int wave = __builtin_amdgcn_readfirstlane(tid / WAVE);
    const uint32_t lb = splitee::xcd_logical_block(blockIdx.x, gridDim.x);
    const int n0 = ((int)lb * GV_WAVES + wave) * GV_NR * ppw; // first row of the wave

    // 1. the W ring, then x~ to LDS (8 consecutive k per unit, GV_XR units per thread and round)
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(W, (uint32_t)((int64_t)N * ldw * 2));
    const int nchunk = (K + 511) / 512;
    const int units_w = ppw * nchunk; // (row pair, 512-k chunk) units of the wave, pair-major
    auto wload = [&](int r, int t) {
        const int pr = t / nchunk, j = t - pr * nchunk;
        const int n = n0 + pr * GV_NR + r, k = 512 * j + 8 * lane;
        const bool ok = t < units_w && n < N && k < K;
        return load16(rw, ok ? (uint32_t)(((int64_t)n * ldw + k) * 2) : OOB);
    };
    uint4 ring[GV_RING][GV_NR];
#pragma unroll
    for (int t = 0; t < GV_RING; ++t)
#pragma unroll
        for (int r = 0; r < GV_NR; ++r) ring[t][r] = wload(r, t);

    const int upr = K / 8, units = MR * upr;
    for (int u0 = 0; u0 < units; u0 += GV_XR * NT) {
        float x[GV_XR][8];
        if (MASK) {
            float4 xv[GV_XR][2], ev[GV_XR][2];
#pragma unroll
            for (int i = 0; i < GV_XR; ++i) {
                const int u = u0 + i * NT + tid;
                const int m = u < units ? u / upr : 0, k = u < units ? (u - m * upr) * 8 : 0;
                const float4* xp = reinterpret_cast<const float4*>(src.X + (int64_t)m * src.ldx + k);
                const float4* ep = reinterpret_cast<const float4*>(src.eta + (int64_t)m * src.ld_eta + k);
                xv[i][0] = xp[0]; xv[i][1] = xp[1]; ev[i][0] = ep[0]; ev[i][1] = ep[1];
            }
#pragma unroll
            for (int i = 0; i < GV_XR; ++i) {
                const float* a = reinterpret_cast<const float*>(xv[i]);
                const float* e = reinterpret_cast<const float*>(ev[i]);
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    float v = a[q] + e[q];
                    if (NPL == 1) v = splitee::bf16_bits_to_f32(splitee::bf16_bits_rne(v));
                    x[i][q] = v;
                }
            }
        } else {
            uint4 pl[GV_XR][NPL];
#pragma unroll
            for (int i = 0; i < GV_XR; ++i) {
                const int u = u0 + i * NT + tid;
                const int m = u < units ? u / upr : 0, k = u < units ? (u - m * upr) * 8 : 0;
#pragma unroll
                for (int p = 0; p < NPL; ++p)
                    pl[i][p] = *reinterpret_cast<const uint4*>(src.A + p * src.pstride + (int64_t)m * src.lda + k);
            }
#pragma unroll
            for (int i = 0; i < GV_XR; ++i)
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    float v = 0.f;
#pragma unroll
                    for (int p = 0; p < NPL; ++p) {
                        const uint32_t wd = reinterpret_cast<const uint32_t*>(&pl[i][p])[q / 2];
                        const float t = splitee::bf16_bits_to_f32((q & 1) ? (wd >> 16) : (wd & 0xFFFFu));
                        v = p == 0 ? t : v + t; // hi + mid, then + lo: exact
                    }
                    x[i][q] = v;
                }
        }
#pragma unroll
        for (int i = 0; i < GV_XR; ++i) {
            const int u = u0 + i * NT + tid;
            if (u < units) {
                const int m = u / upr, k = (u - m * upr) * 8;
                *reinterpret_cast<float4*>(xs + (int64_t)m * K + k) = make_float4(x[i][0], x[i][1], x[i][2], x[i][3]);
                *reinterpret_cast<float4*>(xs + (int64_t)m * K + k + 4) = make_float4(x[i][4], x[i][5], x[i][6], x[i][7]);
            }
        }
    }
    __syncthreads();

    // 2. stream the wave's rows (waves past N run on zeros and store nothing)
    float acc[MR][GV_NR];
#pragma unroll
    for (int m = 0; m < MR; ++m)
#pragma unroll
        for (int r = 0; r < GV_NR; ++r) acc[m][r] = 0.f;
    // unit t = (row pair pr, chunk j); the ring refill is unit t + GV_RING = (prr, jr).
    // The masked input of the next unit is read from LDS while this one is multiplied.
    auto load_x = [&](float (&x)[MR][8], int j) {
        const int k = 512 * j + 8 * lane;
#pragma unroll
        for (int m = 0; m < MR; ++m) {
            float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
            if (k < K) {
                a = *reinterpret_cast<const float4*>(xs + (int64_t)m * K + k);
                b = *reinterpret_cast<const float4*>(xs + (int64_t)m * K + k + 4);
            }
            x[m][0] = a.x; x[m][1] = a.y; x[m][2] = a.z; x[m][3] = a.w;
            x[m][4] = b.x; x[m][5] = b.y; x[m][6] = b.z; x[m][7] = b.w;
        }
    };
    const int nloop = (units_w + GV_RING - 1) / GV_RING * GV_RING;
    int pr = 0, j = 0;
    int prr = GV_RING / nchunk, jr = GV_RING - (GV_RING / nchunk) * nchunk;
    float xc[MR][8];
    load_x(xc, 0);
    for (int t0 = 0; t0 < nloop; t0 += GV_RING) {
#pragma unroll
        for (int u = 0; u < GV_RING; ++u) {
            const int t = t0 + u;
            int jn = j + 1, prn = pr;
            if (jn == nchunk) { jn = 0; ++prn; }
            float xn[MR][8];
            load_x(xn, jn);
#pragma unroll
            for (int r = 0; r < GV_NR; ++r) {
                const uint4 wv = ring[u][r];
                const uint32_t wd[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float w = splitee::bf16_bits_to_f32((e & 1) ? (wd[e / 2] >> 16) : (wd[e / 2] & 0xFFFFu));
#pragma unroll
                    for (int m = 0; m < MR; ++m) acc[m][r] = fmaf(xc[m][e], w, acc[m][r]);
                }
                const int n = n0 + prr * GV_NR + r, k = 512 * jr + 8 * lane;
                const bool ok = t + GV_RING < units_w && n < N && k < K;
                ring[u][r] = load16(rw, ok ? (uint32_t)(((int64_t)n * ldw + k) * 2) : OOB);
            }
            if (++jr == nchunk) { jr = 0; ++prr; }
            // last chunk of a row pair: wave sums, unmask, store, restart
            if (j == nchunk - 1 && t < units_w) {
#pragma unroll
                for (int m = 0; m < MR; ++m)
#pragma unroll
                    for (int r = 0; r < GV_NR; ++r) {
                        const float y = gv_wave_sum(acc[m][r]);
                        const int64_t col = n0 + pr * GV_NR + r;
                        if (lane == 0 && col < N) Out[(int64_t)m * ldo + col] = C ? y - C[(int64_t)m * ldc + col] : y;
                        acc[m][r] = 0.f;
                    }
            }
#pragma unroll
            for (int m = 0; m < MR; ++m)
#pragma unroll
                for (int e = 0; e < 8; ++e) xc[m][e] = xn[m][e];
            j = jn;
            pr = prn;
        }
    }
}

// GEMV with K split over the waves (K <= 16384 and fewer than GS_MAX_PAIRS row pairs;
// the kernel above serves longer rows and the widest N).
// A workgroup owns GS_ROWS (4 or 5) W rows; wave w takes the 512-k chunks j = w, w + 4, ..
// of each row, issues the loads of its chunks' masked input and then all of its W loads
// at once, forms the masked input in registers (from X + eta or from the planes,
// exactly as above) while W is in flight, accumulates fma(x~, w, acc) in chunk and k order,
// sums its lanes with the same butterfly, and the four waves' sums are added in
// wave order.
constexpr int GS_MAX_CH = 8;  // chunks per wave: K <= 4 x 8 x 512

template <int NPL, bool MASK, int MR, int CH, int GS_ROWS>
__global__ void __launch_bounds__(GV_WAVES * WAVE)
gemv_split_kernel(SkSrc src, const uint16_t* __restrict__ W, int64_t ldw, const float* __restrict__ C,
                  int64_t ldc, float* __restrict__ Out, int64_t ldo, int N, int K)
{
    __shared__ float red[GV_WAVES][MR][GS_ROWS];
    const int tid = threadIdx.x, lane = tid % WAVE;
    const int wave = __builtin_amdgcn_readfirstlane(tid / WAVE);
    const uint32_t lb = splitee::xcd_logical_block(blockIdx.x, gridDim.x);
    const int n0 = (int)lb * GS_ROWS;
    const int nchunk = (K + 511) / 512;
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(W, (uint32_t)((int64_t)N * ldw * 2));

    // the masked input through buffer resources so that its loads are unconditional (past K
    // they read zeros); loads issued after W's would hold its conversion until all of W had
    // landed (two tokens 13% faster on the Qwen3-4B and Llama-3.2-3B projections with the
    // masked input first)
    const int MRr = MR;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(MASK ? (const void*)src.X : (const void*)src.A,
                                                MASK ? (uint32_t)((int64_t)MRr * src.ldx * 4)
                                                     : (uint32_t)(((NPL - 1) * src.pstride + (int64_t)MRr * src.lda) * 2));
    const __amdgpu_buffer_rsrc_t re = make_rsrc(MASK ? (const void*)src.eta : (const void*)src.A,
                                                MASK ? (uint32_t)((int64_t)MRr * src.ld_eta * 4) : 0u);
    // raw masked-input words of chunk c, row m: X and eta (two 16-byte loads each) or the
    // NPL bfloat16 planes
    constexpr int XW = MASK ? 4 : NPL;
    uint4 xr[CH][MR][XW];
    auto load_x = [&](int c) {
        const int j = wave + GV_WAVES * c, k = 512 * j + 8 * lane;
        const bool ok = j < nchunk && k < K;
#pragma unroll
        for (int m = 0; m < MR; ++m) {
            if (MASK) {
                const uint32_t xo = ok ? (uint32_t)(((int64_t)m * src.ldx + k) * 4) : OOB;
                const uint32_t eo = ok ? (uint32_t)(((int64_t)m * src.ld_eta + k) * 4) : OOB;
                xr[c][m][0] = load16(rx, xo);
                xr[c][m][1] = load16(rx, ok ? xo + 16 : OOB);
                xr[c][m][2] = load16(re, eo);
                xr[c][m][3] = load16(re, ok ? eo + 16 : OOB);
            } else {
#pragma unroll
                for (int p = 0; p < NPL; ++p)
                    xr[c][m][p] = load16(rx, ok ? (uint32_t)((p * src.pstride + (int64_t)m * src.lda + k) * 2) : OOB);
            }
        }
    };
    float x[CH][MR][8];
    auto convert_x = [&](int c) {
#pragma unroll
        for (int m = 0; m < MR; ++m) {
            if (MASK) {
                const float* a = reinterpret_cast<const float*>(&xr[c][m][0]);
                const float* e = reinterpret_cast<const float*>(&xr[c][m][2]);
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    float v = a[q] + e[q];
                    if (NPL == 1) v = splitee::bf16_bits_to_f32(splitee::bf16_bits_rne(v));
                    x[c][m][q] = v;
                }
            } else {
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    float v = 0.f;
#pragma unroll
                    for (int p = 0; p < NPL; ++p) {
                        const uint32_t wd = reinterpret_cast<const uint32_t*>(&xr[c][m][p])[q / 2];
                        const float t = splitee::bf16_bits_to_f32((q & 1) ? (wd >> 16) : (wd & 0xFFFFu));
                        v = p == 0 ? t : v + t; // hi + mid, then + lo: exact
                    }
                    x[c][m][q] = v;
                }
            }
        }
    };
    uint4 wv[CH][GS_ROWS];
    auto load_w = [&](int c) {
        const int j = wave + GV_WAVES * c, k = 512 * j + 8 * lane;
#pragma unroll
        for (int r = 0; r < GS_ROWS; ++r) {
            const bool ok = j < nchunk && k < K && n0 + r < N;
            wv[c][r] = load16(rw, ok ? (uint32_t)(((int64_t)(n0 + r) * ldw + k) * 2) : OOB);
        }
    };
    // the masked input's loads first (a wave's loads complete in order, so the conversion
    // never waits for W), then, where the raw input words and all of W fit the registers of
    // four waves per SIMD, every W load before the conversion, so that the two latencies
    // overlap; otherwise the conversion first, then every W load
    constexpr bool EARLY_W = CH * (GS_ROWS + MR * XW) * 4 <= 96;
#pragma unroll
    for (int c = 0; c < CH; ++c) load_x(c);
    if constexpr (EARLY_W) {
#pragma unroll
        for (int c = 0; c < CH; ++c) load_w(c);
#pragma unroll
        for (int c = 0; c < CH; ++c) convert_x(c);
    } else {
#pragma unroll
        for (int c = 0; c < CH; ++c) convert_x(c);
#pragma unroll
        for (int c = 0; c < CH; ++c) load_w(c);
    }
    float acc[MR][GS_ROWS];
#pragma unroll
    for (int m = 0; m < MR; ++m)
#pragma unroll
        for (int r = 0; r < GS_ROWS; ++r) acc[m][r] = 0.f;
#pragma unroll
    for (int c = 0; c < CH; ++c)
#pragma unroll
        for (int r = 0; r < GS_ROWS; ++r) {
            const uint32_t wd[4] = {wv[c][r].x, wv[c][r].y, wv[c][r].z, wv[c][r].w};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float w = splitee::bf16_bits_to_f32((e & 1) ? (wd[e / 2] >> 16) : (wd[e / 2] & 0xFFFFu));
#pragma unroll
                for (int m = 0; m < MR; ++m) acc[m][r] = fmaf(x[c][m][e], w, acc[m][r]);
            }
        }
#pragma unroll
    for (int m = 0; m < MR; ++m)
#pragma unroll
        for (int r = 0; r < GS_ROWS; ++r) {
            const float y = gv_wave_sum(acc[m][r]);
            if (lane == 0) red[wave][m][r] = y;
        }
    __syncthreads();
    if (tid < MR * GS_ROWS) {
        const int m = tid / GS_ROWS, r = tid % GS_ROWS, col = n0 + r;
        if (col < N) {
            float y = red[0][m][r];
#pragma unroll
            for (int v = 1; v < GV_WAVES; ++v) y += red[v][m][r];
            Out[(int64_t)m * ldo + col] = C ? y - C[(int64_t)m * ldc + col] : y;
        }
    }
}


// ------------------------------------------------ decode, M <= 2, tiled W
// A workgroup of 4 waves owns one 32-row block of tiled W and a range of its 64-k
// tiles.  Lane l of a wave holds row l % 32 and k half l / 32 of every 16-k step, so
// each W load is the block's contiguous 1 KB step (whole cache lines).  The masked
// input of the range is formed once into LDS (fl32(X + eta), rounded to bfloat16 for
// single-pass BF16, or the exact sum of the planes).  Wave w takes the range's tiles
// w, w + 4, ..; W flows through a ring of GT_RING tiles.  Each lane accumulates
// fma(x~, w, acc) in k order; the two k halves, the four waves and (K split over
// workgroups) the splits are then added in that order, so results are deterministic.
constexpr int GT_RING = 2; // 2 against 3, 4 and 6 on the Qwen3-4B projections: 1-7% faster at one and two tokens
constexpr int GT_LDS_MAX = 64 * 1024;

template <int NPL, bool MASK, int MR>
__global__ void __launch_bounds__(GV_WAVES * WAVE)
gemv_tiled_kernel(SkSrc src, const uint16_t* __restrict__ W, const float* __restrict__ C, int64_t ldc,
                  float* __restrict__ Out, int64_t ldo, int N, int K, int nblocks, int ksplit, int kt_per_split,
                  float* __restrict__ part, unsigned* __restrict__ counters)
{
    extern __shared__ __attribute__((aligned(16))) float xs[]; // MR rows of 64 kt_per_split floats
    __shared__ float red[GV_WAVES][MR][32];
    __shared__ unsigned flag;
    const int tid = threadIdx.x, lane = tid % WAVE;
    const int wave = __builtin_amdgcn_readfirstlane(tid / WAVE);
    const uint32_t lb = splitee::xcd_logical_block(blockIdx.x, gridDim.x);
    const int split = (int)lb / nblocks, cb = (int)lb % nblocks;
    const int ktiles = (K + 63) / 64;
    const int kt0 = split * kt_per_split, kt1 = min(kt0 + kt_per_split, ktiles);
    const int nkt = kt1 > kt0 ? kt1 - kt0 : 0;
    const int XW = 64 * kt_per_split;
    const int njw = nkt > wave ? (nkt - wave + GV_WAVES - 1) / GV_WAVES : 0; // this wave's tiles

    // 1. the first turn of the W ring (wave-local tile j = range tile wave + 4 j into slot j % GT_RING)
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(W, (uint32_t)((int64_t)((N + 31) / 32) * ktiles * 4096));
    const uint32_t wbase = (uint32_t)((int64_t)cb * ktiles * 4096 + lane * 16);
    uint4 ring[GT_RING][4];
    auto wload = [&](int j, uint4 (&dst)[4]) {
        const int kt = kt0 + wave + GV_WAVES * j;
        const bool ok = j < njw;
#pragma unroll
        for (int st = 0; st < 4; ++st) dst[st] = load16(rw, ok ? wbase + (uint32_t)(kt * 4 + st) * 1024 : OOB);
    };
#pragma unroll
    for (int u = 0; u < GT_RING; ++u) wload(u, ring[u]);

    // 2. the masked input of the range: unit t = 8 floats of row m at k = 64 kt0 + 8 (t % (XW / 8))
    {
        const int upr = XW / 8, units = MR * upr;
        const int MRr = MR;
        const __amdgpu_buffer_rsrc_t rx = make_rsrc(MASK ? (const void*)src.X : (const void*)src.A,
                                                    MASK ? (uint32_t)((int64_t)MRr * src.ldx * 4)
                                                         : (uint32_t)(((NPL - 1) * src.pstride + (int64_t)MRr * src.lda) * 2));
        const __amdgpu_buffer_rsrc_t re = make_rsrc(MASK ? (const void*)src.eta : (const void*)src.A,
                                                    MASK ? (uint32_t)((int64_t)MRr * src.ld_eta * 4) : 0u);
        for (int t = tid; t < units; t += GV_WAVES * WAVE) {
            const int m = t / upr, c = t - m * upr, k = 64 * kt0 + 8 * c;
            const bool ok = k < K;
            float v[8];
            if (MASK) {
                const uint32_t xo = ok ? (uint32_t)(((int64_t)m * src.ldx + k) * 4) : OOB;
                const uint32_t eo = ok ? (uint32_t)(((int64_t)m * src.ld_eta + k) * 4) : OOB;
                const uint4 xv[2] = {load16(rx, xo), load16(rx, ok ? xo + 16 : OOB)};
                const uint4 ev[2] = {load16(re, eo), load16(re, ok ? eo + 16 : OOB)};
                const float* a = reinterpret_cast<const float*>(xv);
                const float* e = reinterpret_cast<const float*>(ev);
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    float x = a[q] + e[q];
                    if (NPL == 1) x = splitee::bf16_bits_to_f32(splitee::bf16_bits_rne(x));
                    v[q] = x;
                }
            } else {
                uint4 pl[NPL];
#pragma unroll
                for (int p = 0; p < NPL; ++p)
                    pl[p] = load16(rx, ok ? (uint32_t)((p * src.pstride + (int64_t)m * src.lda + k) * 2) : OOB);
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    float x = 0.f;
#pragma unroll
                    for (int p = 0; p < NPL; ++p) {
                        const uint32_t wd = reinterpret_cast<const uint32_t*>(&pl[p])[q / 2];
                        const float t2 = splitee::bf16_bits_to_f32((q & 1) ? (wd >> 16) : (wd & 0xFFFFu));
                        x = p == 0 ? t2 : x + t2; // hi + mid, then + lo: exact
                    }
                    v[q] = x;
                }
            }
            float4* d = reinterpret_cast<float4*>(xs + m * XW + 8 * c);
            d[0] = make_float4(v[0], v[1], v[2], v[3]);
            d[1] = make_float4(v[4], v[5], v[6], v[7]);
        }
    }
    __syncthreads();

    // 3. stream W through the ring
    const int h = lane / 32;
    float acc[MR];
#pragma unroll
    for (int m = 0; m < MR; ++m) acc[m] = 0.f;
    for (int j0 = 0; j0 < njw; j0 += GT_RING) {
#pragma unroll
        for (int u = 0; u < GT_RING; ++u) {
            const int j = j0 + u;
            if (j < njw) {
                const int lt = wave + GV_WAVES * j; // tile within the range
#pragma unroll
                for (int st = 0; st < 4; ++st) {
                    const uint32_t wd[4] = {ring[u][st].x, ring[u][st].y, ring[u][st].z, ring[u][st].w};
#pragma unroll
                    for (int m = 0; m < MR; ++m) {
                        const float4* xp = reinterpret_cast<const float4*>(xs + m * XW + 64 * lt + 16 * st + 8 * h);
                        const float4 x0 = xp[0], x1 = xp[1];
                        const float xv[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const float w = splitee::bf16_bits_to_f32((e & 1) ? (wd[e / 2] >> 16) : (wd[e / 2] & 0xFFFFu));
                            acc[m] = fmaf(xv[e], w, acc[m]);
                        }
                    }
                }
            }
            wload(j + GT_RING, ring[u]);
        }
    }

    // 4. lanes l and l + 32 (the two k halves of row l), then the waves in order
#pragma unroll
    for (int m = 0; m < MR; ++m) {
        const float o = __shfl_xor(acc[m], 32);
        if (lane < 32) red[wave][m][lane] = acc[m] + o;
    }
    __syncthreads();
    const bool owner = tid < MR * 32;
    const int om = tid / 32, orow = tid % 32, col = 32 * cb + orow;
    float y = 0.f;
    if (owner) {
        y = red[0][om][orow];
#pragma unroll
        for (int v = 1; v < GV_WAVES; ++v) y += red[v][om][orow];
    }
    if (ksplit == 1) {
        if (owner && col < N) Out[(int64_t)om * ldo + col] = C ? y - C[(int64_t)om * ldc + col] : y;
        return;
    }
    if (owner) store_partial(&part[(((int64_t)cb * ksplit + split) * MR + om) * 32 + orow], y);
    if (!splitk_arrive(counters + cb, ksplit, &flag)) return;
    if (owner) {
        // C first, then the splits' partials eight at a time (agent-coherent buffer loads; a
        // split past ksplit reads zeros and is not added), summed in split order
        const float cv = C && col < N ? C[(int64_t)om * ldc + col] : 0.f;
        const __amdgpu_buffer_rsrc_t rp = make_rsrc(part + (int64_t)cb * ksplit * MR * 32, (uint32_t)(ksplit * MR * 32 * 4));
        float sum = 0.f;
        for (int q0 = 0; q0 < ksplit; q0 += 8) {
            float v[8];
#pragma unroll
            for (int i = 0; i < 8; ++i)
                v[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                           rp, (int)(q0 + i < ksplit ? (uint32_t)((((q0 + i) * MR + om) * 32 + orow) * 4) : OOB_OFF), 0, SC1));
#pragma unroll
            for (int i = 0; i < 8; ++i)
                if (q0 + i < ksplit) sum = (q0 + i == 0) ? v[i] : sum + v[i];
        }
        if (col < N) Out[(int64_t)om * ldo + col] = C ? sum - cv : sum;
    }
    if (tid == 0) splitk_reset(counters + cb);
}

// ------------------------------------------------------------ host planning

struct Plan {
    int bm, bn, bk;
    int mtiles, ntiles, ktiles;
    int ksplit, kt_per_split;
    size_t part_bytes, counter_bytes;
    int variant; // which instantiation
};

constexpr int TARGET_WGS = 512; // two workgroups per CU on 256 CUs

// The W-streamed kernel serves every bfloat16 GEMM that does not take the skinny
// kernel (M <= 16 with a workspace).  Tiles, measured on the Llama-3.2-3B
// projections at 128 and 512 tokens:
//   M <= 64:       64 x 256, 4 waves side by side  (variants 11 bf16x3, 13 bf16)
//   64 < M <= 128: 128 x 128, 2 x 2 waves          (variants 14 bf16x3, 15 bf16)
//   M > 128:       128 x 256, 4 waves side by side (variants 10 bf16x3, 12 bf16)
// With tiled W, 8 waves per workgroup, measured on the same projections and the
// Qwen3-4B ones at 32, 64 and 1024 tokens:
//   M <= 128: 64-row tiles (two M tiles above 64 rows: half the masked-input stage of a
//             128-row tile, so the 160 KB hold a third K tile in flight): 64 x 128 on
//             2 x 4 waves, 3 K tiles ahead (variants 26, 27), or 64 x 256 on 8 waves
//             side by side, 2 ahead (variants 24, 25) when N has 64 or more 256-column
//             tiles
//   M > 128:  128 x 256, 2 x 4 waves, 2 ahead (variants 22, 23); 64 x 256 when the 128-row
//             tiles take more than one round of 256 workgroups and half-height tiles end
//             in a fuller last round (Qwen3-4B gate/up at 1024 tokens: 608 tiles, 3
//             rounds, against 1216 half tiles, 2.5 rounds' work: 361 -> 334 us), for three
//             planes on 4 waves of 64 x 64 in workgroups of their own, two per CU (variant
//             30: each workgroup waits at its own barrier, so one's loads run under the
//             other's MFMAs, and a masked-input fragment feeds two MFMAs instead of one;
//             the same gate/up 332 -> 287 us against 8 waves side by side); else
//             128 x 192 on 4 x 2 waves (variants 28, 29) where split_cost says it is
//             cheaper than 128 x 256 (a sweep of 2 x 4 and 4 x 2 waves on 64 x 256,
//             128 x 128 and 128 x 256 tiles found no other shape faster on these
//             projections); three planes with K up to 4096 and at most 256 tiles of 64 x 192:
//             those on 2 x 2 waves (variant 31)
// The K split fills about 256 CUs, keeps at least ST_MIN_KT K tiles per split and
// at most ST_MAX_KS splits; below that cap it takes the split count with the fewest
// rounds of 256 workgroups times K tiles per split rounded up to whole turns of the
// ring (the rest of a turn runs on zero tiles), the fewer splits on a tie.

// The K split of the streamed kernel for `tiles` output tiles of `ktiles` K tiles and
// its cost: the split count (at most ST_MAX_KS, at least ST_MIN_KT K tiles per split,
// at most 256 workgroups) with the fewest rounds of 256 workgroups times K tiles per
// split rounded up to whole ring turns, the fewer splits on a tie.
std::pair<int, int64_t> stream_split(int tiles, int ktiles, int ring)
{
    int ks = 1;
    int64_t best = ((int64_t)tiles + 255) / 256 * ((ktiles + ring - 1) / ring * ring);
    if (ktiles > 0) {
        int ks_max = 256 / tiles;
        if (ks_max > ktiles / ST_MIN_KT) ks_max = ktiles / ST_MIN_KT;
        if (ks_max > ST_MAX_KS) ks_max = ST_MAX_KS;
        for (int c = 2; c <= ks_max; ++c) {
            const int64_t kps = (ktiles + c - 1) / c;
            const int64_t cost = ((int64_t)tiles * c + 255) / 256 * ((kps + ring - 1) / ring * ring);
            if (cost < best) { best = cost; ks = c; }
        }
    }
    return {ks, best};
}

// Work of the busiest CU for bm x bn tiles split as stream_split chooses: rounds of
// workgroups times tile area times K tiles per split; ties go to fewer splits by
// comparing the split counts second.
int64_t split_cost(int64_t M, int64_t N, int64_t K, int bm, int bn, int ring, bool allow_split)
{
    const int tiles = (int)(((M + bm - 1) / bm) * ((N + bn - 1) / bn));
    const int ktiles = (int)((K + 63) / 64);
    const std::pair<int, int64_t> sp = allow_split ? stream_split(tiles, ktiles, ring)
                                                   : std::pair<int, int64_t>{1, ((int64_t)tiles + 255) / 256 *
                                                                                    ((ktiles + ring - 1) / ring * ring)};
    return (sp.second * bm * bn) * 16 + sp.first;
}

bool use_stream(int prec, int w_type)
{
    return prec != SPLITEE_PREC_F32 && (w_type == SPLITEE_BF16 || w_type == SPLITEE_BF16_TILED);
}

Plan plan_stream(int64_t M, int64_t N, int64_t K, int prec, int w_type, bool allow_split)
{
    Plan p{};
    const bool x3 = prec == SPLITEE_PREC_BF16X3;
    p.bk = 64;
    if (w_type == SPLITEE_BF16_TILED) {
        if (M <= 128 && (N + 255) / 256 < 64) {
            p.bm = 64; p.bn = 128; p.variant = x3 ? 26 : 27;
        } else if (M <= 128) {
            p.bm = 64; p.bn = 256; p.variant = x3 ? 24 : 25;
        } else if (const int64_t t128 = (M + 127) / 128 * ((N + 255) / 256), t64 = (M + 63) / 64 * ((N + 255) / 256);
                   t128 > 256 && (t64 + 255) / 256 < 2 * ((t128 + 255) / 256)) {
            // three planes: half-height tiles on 4 waves, two workgroups per CU (72 KB of LDS
            // each); one plane keeps 8 waves (its gate/up at 1024 tokens: 170 us against 212)
            p.bm = 64; p.bn = 256; p.variant = x3 ? 30 : 25;
        } else {
            p.bm = 128; p.bn = 256; p.variant = x3 ? 22 : 23;
            // 128 x 192 tiles on 4 x 2 waves when they cost less by split_cost (rounds of
            // workgroups times tile area times K tiles per split): Qwen3-4B QKV at 1024
            // tokens, 192 tiles of 128 x 256 on 256 CUs against exactly 256 of 128 x 192
            // (116 -> 100 us); Llama-3.2-3B QKV, O and Down at 512 tokens by 1-6%
            if (split_cost(M, N, K, 128, 192, 3, allow_split) < split_cost(M, N, K, 128, 256, 3, allow_split)) {
                p.bn = 192; p.variant = x3 ? 28 : 29;
            }
            // three planes, K up to 4096 and at most 256 tiles of 64 x 192: those tiles on 2 x 2
            // waves (variant 31; the K split then fills 256 CUs): on the QKV and O projections of
            // Qwen3-4B and Llama-3.2-3B at 256-1024 tokens 2-15% faster than the 8-wave tiles
            // (512-token QKV 51.8 -> 44.6 us, 256-token O 25.4 -> 21.6); with more tiles (1024-token
            // QKV, 256-token gate/up) and on Down (K 8192, 9728) as fast or slower, up to 23%
            if (x3 && K <= 4096 && (M + 63) / 64 * ((N + 191) / 192) <= 256) {
                p.bm = 64; p.bn = 192; p.variant = 31;
            }
        }
    } else if (M <= 64) {
        p.bm = 64; p.bn = 256; p.variant = x3 ? 11 : 13;
    } else if (M <= 128) {
        p.bm = 128; p.bn = 128; p.variant = x3 ? 14 : 15;
    } else {
        p.bm = 128; p.bn = 256; p.variant = x3 ? 10 : 12;
    }
    p.mtiles = (int)((M + p.bm - 1) / p.bm);
    p.ntiles = (int)((N + p.bn - 1) / p.bn);
    p.ktiles = (int)((K + p.bk - 1) / p.bk);
    const int tiles = p.mtiles * p.ntiles;
    // ring stages (K tiles in flight + 1) of the variant
    const int ring = (p.variant == 11 || p.variant == 13 || p.variant == 26 || p.variant == 27) ? 4 : 3;
    const int ks = allow_split ? stream_split(tiles, p.ktiles, ring).first : 1;
    p.kt_per_split = p.ktiles > 0 ? (p.ktiles + ks - 1) / ks : 1;
    p.ksplit = p.ktiles > 0 ? (p.ktiles + p.kt_per_split - 1) / p.kt_per_split : 1;
    p.counter_bytes = 0; // the partials are summed by a second kernel: no counters
    p.part_bytes = p.ksplit > 1 ? (size_t)tiles * p.ksplit * p.bm * p.bn * 4 : 0;
    return p;
}

Plan plan_tiled(int64_t M, int64_t N, int64_t K, int prec, int w_type, bool allow_split)
{
    if (use_stream(prec, w_type)) return plan_stream(M, N, K, prec, w_type, allow_split);
    Plan p{}; // float32 MFMA
    p.bm = 128; p.bn = 128; p.bk = 32; p.variant = 0;
    if (M <= 64) { p.bm = 64; p.bn = 64; p.variant = 1; }
    (void)w_type;
    p.mtiles = (int)((M + p.bm - 1) / p.bm);
    p.ntiles = (int)((N + p.bn - 1) / p.bn);
    p.ktiles = (int)((K + p.bk - 1) / p.bk);
    int tiles = p.mtiles * p.ntiles;
    int ks = 1;
    if (allow_split && tiles < TARGET_WGS / 2) {
        ks = (TARGET_WGS / 2 + tiles - 1) / tiles;
        int max_ks = p.ktiles / 4; // keep at least 4 K tiles per split
        if (ks > max_ks) ks = max_ks;
        if (ks > KSMAX) ks = KSMAX;
        if (ks < 1) ks = 1;
    }
    p.kt_per_split = p.ktiles > 0 ? (p.ktiles + ks - 1) / ks : 1;
    p.ksplit = p.ktiles > 0 ? (p.ktiles + p.kt_per_split - 1) / p.kt_per_split : 1;
    p.counter_bytes = p.ksplit > 1 ? (((size_t)tiles * 4 + 255) / 256) * 256 : 0;
    p.part_bytes = p.ksplit > 1 ? (size_t)tiles * p.ksplit * p.bm * p.bn * 4 : 0;
    return p;
}

// Masked-input slice bytes of one skinny workgroup holding `steps` k steps.
size_t skinny_lds_bytes(int64_t M, int npl, int steps)
{
    const int sa = (steps + SK_RING - 1) / SK_RING * SK_RING;
    return (size_t)npl * (size_t)M * (size_t)(sa * 64 + 16);
}

Plan plan_skinny(int64_t M, int64_t N, int64_t K, int prec)
{
    Plan p{};
    const int npl = prec == SPLITEE_PREC_BF16X3 ? 3 : 1;
    p.bm = 16; p.bn = SK_BN; p.bk = 32;
    p.mtiles = 1;
    p.ntiles = (int)((N + SK_BN - 1) / SK_BN);
    p.ktiles = (int)((K + 31) / 32);
    int ks = SK_TARGET_WGS / p.ntiles;
    if (p.ntiles <= 256 && p.ktiles > 0) {
        // up to 256 tiles: splits of whole 16-step granules, the fewest granules per split whose
        // workgroups still fit one round of two per CU (Qwen3-4B O, 40 tiles of 128 steps, 8
        // splits of 16 instead of 12 of 11: 9.3 -> 8.5 us at 4 tokens, 10.9 -> 9.8 at 16; Down,
        // 304 steps, 10 splits of 32 instead of 12 of 26: 13.0 -> 12.5 at 4 tokens)
        int g = 1;
        while (p.ntiles * ((p.ktiles + 16 * g - 1) / (16 * g)) > SK_TARGET_WGS) ++g;
        ks = (p.ktiles + 16 * g - 1) / (16 * g);
    }
    // more than 256 tiles: split up to 1536 workgroups (three rounds) while every split
    // still holds a granule of 16 k steps (measured on the Qwen3-4B gate/up projection, 304
    // tiles: 5 splits of 16 steps against 3 of 27 at 4 tokens 21.1 -> 20.4 us, at 8 tokens
    // 24.7 -> 21.2 us; an LM head's thousands of tiles keep one split)
    if (p.ntiles > 256) ks = std::max(1, std::min(p.ktiles / SK_RING, 1536 / p.ntiles));
    if (ks > p.ktiles) ks = p.ktiles;
    if (ks < 1) ks = 1;
    int sps = p.ktiles > 0 ? (p.ktiles + ks - 1) / ks : 1;
    while (sps > 1 && skinny_lds_bytes(M > 0 ? M : 1, npl, sps) > (size_t)SK_LDS_MAX) --sps;
    // the same number of splits, evened out (an LDS-limited split count can leave a short
    // last split: the Llama-3.2-3B LM head at 4 tokens, 96 steps, took 80 + 16)
    if (p.ktiles > 0) sps = (p.ktiles + (p.ktiles + sps - 1) / sps - 1) / ((p.ktiles + sps - 1) / sps);
    p.kt_per_split = sps;
    p.ksplit = p.ktiles > 0 ? (p.ktiles + sps - 1) / sps : 1;
    p.counter_bytes = p.ksplit > 1 ? (((size_t)p.ntiles * 4 + 255) / 256) * 256 : 0;
    p.part_bytes = p.ksplit > 1 ? (size_t)p.ntiles * p.ksplit * 16 * SK_BN * 4 : 0;
    return p;
}

// Tiled GEMV (M <= 2, tiled W): the K split (at most 16, at least one 64-k tile per
// wave, at most about two workgroups per CU) that leaves the busiest CU the fewest
// tiles when the workgroups are dealt out over 256 CUs (the fewer splits on a tie),
// then further splits while the masked input of a range exceeds GT_LDS_MAX.
struct GtPlan {
    int nblocks, ksplit, kt_per_split;
    size_t counter_bytes, part_bytes, lds;
};

GtPlan plan_gemv_tiled(int64_t M, int64_t N, int64_t K)
{
    GtPlan p{};
    p.nblocks = (int)((N + 31) / 32);
    const int ktiles = (int)((K + 63) / 64);
    const int ks_max = std::max(1, std::min(std::min(16, ktiles / GV_WAVES), 512 / std::max(p.nblocks, 1)));
    int ks = 1;
    int64_t best = -1;
    for (int c = 1; c <= ks_max; ++c) {
        const int64_t kps_c = (ktiles + c - 1) / c;
        const int64_t busiest = ((int64_t)p.nblocks * c + 255) / 256 * kps_c;
        if (best < 0 || busiest < best) { best = busiest; ks = c; }
    }
    int kps = ktiles > 0 ? (ktiles + ks - 1) / ks : 1;
    while (kps > 1 && (size_t)M * 64 * kps * 4 > (size_t)GT_LDS_MAX) kps = (kps + 1) / 2;
    p.kt_per_split = std::max(kps, 1);
    p.ksplit = ktiles > 0 ? (ktiles + p.kt_per_split - 1) / p.kt_per_split : 1;
    p.counter_bytes = p.ksplit > 1 ? (((size_t)p.nblocks * 4 + 255) / 256) * 256 : 0;
    p.part_bytes = p.ksplit > 1 ? (size_t)p.nblocks * p.ksplit * M * 32 * 4 : 0;
    p.lds = (size_t)M * 64 * p.kt_per_split * 4;
    return p;
}

// K split over the waves of a workgroup: measured on the Qwen3-4B decode projections
// (N 2560 .. 19456) 10-40% faster than the streaming GEMV, and 1-3% slower on the LM
// heads (N 128256, 151936), which keep the streaming kernel.  Rows per workgroup: 4 or
// 5, whichever gives the busiest CU (256 CUs, workgroups dealt out evenly) the fewest
// rows, 4 on a tie (4 beat 1, 2 and 8 rows at N = 2560, 6144 and 19456).
constexpr int64_t GS_MAX_PAIRS = 32768;

int gs_rows(int64_t N)
{
    auto busiest = [&](int64_t r) { return ((N + r - 1) / r + 255) / 256 * r; };
    return busiest(5) < busiest(4) ? 5 : 4;
}

template <bool MASK>
int launch_gemv_split(const SkSrc& src, int prec, const void* W, int64_t ldw, const float* C, int64_t ldc,
                      float* Out, int64_t ldo, int64_t M, int64_t N, int64_t K, hipStream_t s)
{
    const int ch = (int)(((K + 511) / 512 + GV_WAVES - 1) / GV_WAVES);
    const int rows = gs_rows(N);
    const dim3 grid((unsigned)((N + rows - 1) / rows));
    const uint16_t* w = reinterpret_cast<const uint16_t*>(W);
#define GS_LAUNCH(NP, MR, CHN)                                                                                      \
    do {                                                                                                            \
        if (rows == 5)                                                                                              \
            hipLaunchKernelGGL((gemv_split_kernel<NP, MASK, MR, CHN, 5>), grid, dim3(GV_WAVES * WAVE), 0, s, src, w, \
                               ldw, C, ldc, Out, ldo, (int)N, (int)K);                                              \
        else                                                                                                        \
            hipLaunchKernelGGL((gemv_split_kernel<NP, MASK, MR, CHN, 4>), grid, dim3(GV_WAVES * WAVE), 0, s, src, w, \
                               ldw, C, ldc, Out, ldo, (int)N, (int)K);                                              \
    } while (0)
#define GS_CH(NP, MR)                                                                        \
    switch (ch) {                                                                            \
    case 1: GS_LAUNCH(NP, MR, 1); break;                                                     \
    case 2: GS_LAUNCH(NP, MR, 2); break;                                                     \
    case 3: GS_LAUNCH(NP, MR, 3); break;                                                     \
    case 4: GS_LAUNCH(NP, MR, 4); break;                                                     \
    case 5: GS_LAUNCH(NP, MR, 5); break;                                                     \
    case 6: GS_LAUNCH(NP, MR, 6); break;                                                     \
    case 7: GS_LAUNCH(NP, MR, 7); break;                                                     \
    default: GS_LAUNCH(NP, MR, 8); break;                                                    \
    }
    if (prec == SPLITEE_PREC_BF16) { if (M == 1) { GS_CH(1, 1) } else { GS_CH(1, 2) } }
    else { if (M == 1) { GS_CH(3, 1) } else { GS_CH(3, 2) } }
#undef GS_CH
#undef GS_LAUNCH
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

// M <= GV_MMAX: the GEMV kernels (x~ of all K sits in LDS for the streaming one).
template <bool MASK>
int launch_gemv(const SkSrc& src, int prec, const void* W, int64_t ldw, const float* C, int64_t ldc, float* Out,
                int64_t ldo, int64_t M, int64_t N, int64_t K, hipStream_t s)
{
    if ((N + GV_NR - 1) / GV_NR < GS_MAX_PAIRS && K <= (int64_t)GV_WAVES * GS_MAX_CH * 512)
        return launch_gemv_split<MASK>(src, prec, W, ldw, C, ldc, Out, ldo, M, N, K, s);
    const size_t lds = (size_t)M * (size_t)K * 4;
    if (lds > 160 * 1024) return SPLITEE_ERR_UNSUPPORTED;
    // row pairs per wave: the fewest that keep the grid within two workgroups per CU
    const int64_t pairs = (N + GV_NR - 1) / GV_NR;
    const int ppw = (int)((pairs + GV_MAX_WGS * GV_WAVES - 1) / (GV_MAX_WGS * GV_WAVES));
    const int64_t waves = (pairs + ppw - 1) / ppw;
    dim3 grid((unsigned)((waves + GV_WAVES - 1) / GV_WAVES));
    const uint16_t* w = reinterpret_cast<const uint16_t*>(W);
#define GV_LAUNCH(NP, MR) hipLaunchKernelGGL((gemv_kernel<NP, MASK, MR>), grid, dim3(GV_WAVES * WAVE), lds, s, src, w, ldw, C, ldc, Out, ldo, (int)N, (int)K, ppw)
    if (prec == SPLITEE_PREC_BF16) { if (M == 1) GV_LAUNCH(1, 1); else GV_LAUNCH(1, 2); }
    else { if (M == 1) GV_LAUNCH(3, 1); else GV_LAUNCH(3, 2); }
#undef GV_LAUNCH
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

// ------------------------------------------------------ tiled weight order
// Thread t writes 16-byte chunk t of the tiled buffer: chunk 64 (4 (B kt64 + kt) + s) + l
// holds W[32 B + l % 32][64 kt + 16 s + 8 (l / 32) .. + 7] (zeros past N or K).
__global__ void __launch_bounds__(256) tile_weights_kernel(const uint16_t* __restrict__ W, int64_t ldw, int64_t N,
                                                           int64_t K, uint16_t* __restrict__ Wt, int64_t chunks)
{
    const int64_t kt64 = (K + 63) / 64;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < chunks;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int l = (int)(t % 64);
        const int64_t rest = t / 64, st = rest % 4, blk = rest / 4;
        const int64_t kt = blk % kt64, cb = blk / kt64;
        const int64_t n = 32 * cb + l % 32, k = 64 * kt + 16 * st + 8 * (l / 32);
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (n < N && k < K) v = *reinterpret_cast<const uint4*>(W + n * ldw + k);
        *reinterpret_cast<uint4*>(Wt + 8 * t) = v;
    }
}

}  // namespace

namespace splitee_host {

int launch_tile_weights(const uint16_t* W, int64_t ldw, int64_t N, int64_t K, uint16_t* Wt, hipStream_t s)
{
    const int64_t chunks = (int64_t)(splitee::tiled_weights_bytes(N, K) / 16);
    if (chunks == 0) return SPLITEE_OK;
    int64_t g = (chunks + 255) / 256;
    if (g > 256 * 64) g = 256 * 64;
    hipLaunchKernelGGL(tile_weights_kernel, dim3((unsigned)g), dim3(256), 0, s, W, ldw, N, K, Wt, chunks);
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K, int prec, int w_type)
{
    Plan p = plan_tiled(M, N, K, prec, w_type, true);
    return p.counter_bytes + p.part_bytes;
}

size_t gemm_counter_bytes(int64_t M, int64_t N, int64_t K, int prec, int w_type)
{
    return plan_tiled(M, N, K, prec, w_type, true).counter_bytes;
}

int launch_gemm(const void* A, int prec, int64_t lda, int64_t pstride, const void* W, int w_type,
                int64_t ldw, const float* C, int64_t ldc, float* Out, int64_t ldo, int64_t M,
                int64_t N, int64_t K, void* ws, size_t ws_bytes, hipStream_t s)
{
    if (M == 0 || N == 0) return SPLITEE_OK;
    const bool allow_split = ws != nullptr;
    Plan p = plan_tiled(M, N, K, prec, w_type, allow_split);
    if (p.ksplit > 1 && ws_bytes < p.counter_bytes + p.part_bytes) return SPLITEE_ERR_WORKSPACE;
    unsigned* counters = p.ksplit > 1 ? reinterpret_cast<unsigned*>(ws) : nullptr;
    float* part = p.ksplit > 1 ? reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + p.counter_bytes) : nullptr;
    dim3 grid((unsigned)(p.mtiles * p.ntiles * p.ksplit));
    const int m = (int)M, n = (int)N, k = (int)K;
    if (prec == SPLITEE_PREC_F32) {
        const float* a = reinterpret_cast<const float*>(A);
        if (w_type == SPLITEE_BF16) {
            if (p.variant == 0)
                hipLaunchKernelGGL((gemm_f32_kernel<128, 128, 32, 2, 2, true>), grid, dim3(256), 0, s, a, lda, W, ldw, C, ldc, Out, ldo, m, n, k, p.mtiles, p.ntiles, p.ksplit, p.kt_per_split, part, counters);
            else
                hipLaunchKernelGGL((gemm_f32_kernel<64, 64, 32, 2, 2, true>), grid, dim3(256), 0, s, a, lda, W, ldw, C, ldc, Out, ldo, m, n, k, p.mtiles, p.ntiles, p.ksplit, p.kt_per_split, part, counters);
        } else {
            if (p.variant == 0)
                hipLaunchKernelGGL((gemm_f32_kernel<128, 128, 32, 2, 2, false>), grid, dim3(256), 0, s, a, lda, W, ldw, C, ldc, Out, ldo, m, n, k, p.mtiles, p.ntiles, p.ksplit, p.kt_per_split, part, counters);
            else
                hipLaunchKernelGGL((gemm_f32_kernel<64, 64, 32, 2, 2, false>), grid, dim3(256), 0, s, a, lda, W, ldw, C, ldc, Out, ldo, m, n, k, p.mtiles, p.ntiles, p.ksplit, p.kt_per_split, part, counters);
        }
    } else {
        const uint16_t* a = reinterpret_cast<const uint16_t*>(A);
        const uint16_t* w = reinterpret_cast<const uint16_t*>(W);
        // the buffer loads address each operand with 31-bit byte offsets
        const int64_t planes = prec == SPLITEE_PREC_BF16X3 ? 3 : 1;
        const int64_t wbytes = w_type == SPLITEE_BF16_TILED ? (int64_t)splitee::tiled_weights_bytes(N, K) : N * ldw * 2;
        if ((planes - 1) * pstride * 2 + M * lda * 2 >= (int64_t(1) << 31) || wbytes >= (int64_t(1) << 31) ||
            p.part_bytes >= (size_t(1) << 31))
            return SPLITEE_ERR_UNSUPPORTED;
        float* pp = reinterpret_cast<float*>(ws);
#define ST_LAUNCH(NP, BM_, BN_, WGM_, D_, NW_, T_) hipLaunchKernelGGL((gemm_stream_kernel<NP, BM_, BN_, WGM_, D_, NW_, T_>), grid, dim3(NW_ * WAVE), 0, s, a, lda, pstride, w, ldw, C, ldc, Out, ldo, m, n, k, p.mtiles, p.ntiles, p.ksplit, p.kt_per_split, pp)
#define ST_SUM(BM_, BN_, WGM_, WGN_) hipLaunchKernelGGL((stream_sum_kernel<BM_, BN_, WGM_, WGN_>), g2, dim3(256), 0, s, pp, p.ksplit, C, ldc, Out, ldo, m, n, p.mtiles, tiles)
        switch (p.variant) {
        case 10: ST_LAUNCH(3, 128, 256, 1, 2, 4, false); break;
        case 11: ST_LAUNCH(3, 64, 256, 1, 3, 4, false); break;
        case 12: ST_LAUNCH(1, 128, 256, 1, 2, 4, false); break;
        case 13: ST_LAUNCH(1, 64, 256, 1, 3, 4, false); break;
        case 14: ST_LAUNCH(3, 128, 128, 2, 2, 4, false); break;
        case 15: ST_LAUNCH(1, 128, 128, 2, 2, 4, false); break;
        case 22: ST_LAUNCH(3, 128, 256, 2, 2, 8, true); break;
        case 23: ST_LAUNCH(1, 128, 256, 2, 2, 8, true); break;
        case 24: ST_LAUNCH(3, 64, 256, 1, 2, 8, true); break;
        case 25: ST_LAUNCH(1, 64, 256, 1, 2, 8, true); break;
        case 26: ST_LAUNCH(3, 64, 128, 2, 3, 8, true); break;
        case 28: ST_LAUNCH(3, 128, 192, 4, 2, 8, true); break;
        case 29: ST_LAUNCH(1, 128, 192, 4, 2, 8, true); break;
        case 30: ST_LAUNCH(3, 64, 256, 1, 2, 4, true); break;
        case 31: ST_LAUNCH(3, 64, 192, 2, 2, 4, true); break;
        default: ST_LAUNCH(1, 64, 128, 2, 3, 8, true); break;
        }
        if (p.ksplit > 1) {
            const int tiles = p.mtiles * p.ntiles;
            const int64_t units = (int64_t)tiles * p.bm * p.bn / 4; // float4 units of the partial tiles
            const dim3 g2((unsigned)((units + 255) / 256));
            switch (p.variant) {
            case 10: case 12: ST_SUM(128, 256, 1, 4); break;
            case 11: case 13: ST_SUM(64, 256, 1, 4); break;
            case 14: case 15: ST_SUM(128, 128, 2, 2); break;
            case 22: case 23: ST_SUM(128, 256, 2, 4); break;
            case 24: case 25: ST_SUM(64, 256, 1, 8); break;
            case 28: case 29: ST_SUM(128, 192, 4, 2); break;
            case 30: ST_SUM(64, 256, 1, 4); break;
            case 31: ST_SUM(64, 192, 2, 2); break;
            default: ST_SUM(64, 128, 2, 4); break;
            }
        }
#undef ST_SUM
#undef ST_LAUNCH
    }
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

size_t skinny_workspace_bytes(int64_t M, int64_t N, int64_t K, int prec, int w_type)
{
    if (w_type == SPLITEE_BF16_TILED && M <= GV_MMAX) {
        const GtPlan g = plan_gemv_tiled(M, N, K);
        return g.counter_bytes + g.part_bytes;
    }
    Plan p = plan_skinny(M, N, K, prec);
    return p.counter_bytes + p.part_bytes;
}

size_t skinny_counter_bytes(int64_t M, int64_t N, int64_t K, int prec, int w_type)
{
    if (w_type == SPLITEE_BF16_TILED && M <= GV_MMAX) return plan_gemv_tiled(M, N, K).counter_bytes;
    return plan_skinny(M, N, K, prec).counter_bytes;
}

// The skinny kernel for one decode GEMM (plan, workspace split, instantiation).
template <bool MASK>
int run_skinny(const SkSrc& src, int prec, const void* W, bool tiled, int64_t ldw, const float* C, int64_t ldc,
               float* Out, int64_t ldo, int64_t M, int64_t N, int64_t K, void* ws, size_t ws_bytes, hipStream_t s)
{
    const int npl = prec == SPLITEE_PREC_BF16X3 ? 3 : 1;
    Plan p = plan_skinny(M, N, K, prec);
    const size_t lds = skinny_lds_bytes(M, npl, p.kt_per_split);
    if (lds > (size_t)SK_LDS_MAX) return SPLITEE_ERR_UNSUPPORTED;
    if (p.ksplit > 1 && (ws == nullptr || ws_bytes < p.counter_bytes + p.part_bytes)) return SPLITEE_ERR_WORKSPACE;
    unsigned* counters = p.ksplit > 1 ? reinterpret_cast<unsigned*>(ws) : nullptr;
    float* part = p.ksplit > 1 ? reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + p.counter_bytes) : nullptr;
    dim3 grid((unsigned)(p.ntiles * p.ksplit));
    const uint16_t* w = reinterpret_cast<const uint16_t*>(W);
#define SK_LAUNCHR(NP, RR, T, MC) hipLaunchKernelGGL((skinny_kernel<NP, RR, MASK, T, MC>), grid, dim3(256), lds, s, src, w, ldw, C, ldc, Out, ldo, (int)M, (int)N, (int)K, p.ntiles, p.ksplit, p.kt_per_split, part, counters)
    // ring depth and slice round by M: (4 steps, 2 units) up to 8 rows, (8, 4 with the mask) above
#define SK_LAUNCH(NP, T)                                                                     \
    do {                                                                                     \
        if (sk_ring(M) == 4) SK_LAUNCHR(NP, 4, T, SK_MCP_SMALL);                             \
        else SK_LAUNCHR(NP, 8, T, (MASK ? SK_MCP_LARGE : SK_MCP_SMALL));                     \
    } while (0)
    if (npl == 1) { if (tiled) SK_LAUNCH(1, true); else SK_LAUNCH(1, false); }
    else { if (tiled) SK_LAUNCH(3, true); else SK_LAUNCH(3, false); }
#undef SK_LAUNCHR
#undef SK_LAUNCH
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

template <bool MASK>
int run_gemv_tiled(const SkSrc& src, int prec, const void* W, const float* C, int64_t ldc, float* Out, int64_t ldo,
                   int64_t M, int64_t N, int64_t K, void* ws, size_t ws_bytes, hipStream_t s)
{
    const GtPlan p = plan_gemv_tiled(M, N, K);
    if (p.lds > (size_t)GT_LDS_MAX) return SPLITEE_ERR_UNSUPPORTED;
    if (p.ksplit > 1 && (ws == nullptr || ws_bytes < p.counter_bytes + p.part_bytes)) return SPLITEE_ERR_WORKSPACE;
    unsigned* counters = p.ksplit > 1 ? reinterpret_cast<unsigned*>(ws) : nullptr;
    float* part = p.ksplit > 1 ? reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + p.counter_bytes) : nullptr;
    const dim3 grid((unsigned)((int64_t)p.nblocks * p.ksplit));
    const uint16_t* w = reinterpret_cast<const uint16_t*>(W);
#define GT_LAUNCH(NP, MR) hipLaunchKernelGGL((gemv_tiled_kernel<NP, MASK, MR>), grid, dim3(GV_WAVES * WAVE), p.lds, s, src, w, C, ldc, Out, ldo, (int)N, (int)K, p.nblocks, p.ksplit, p.kt_per_split, part, counters)
    if (prec == SPLITEE_PREC_BF16) { if (M == 1) GT_LAUNCH(1, 1); else GT_LAUNCH(1, 2); }
    else { if (M == 1) GT_LAUNCH(3, 1); else GT_LAUNCH(3, 2); }
#undef GT_LAUNCH
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

// M <= 2 runs on the vector-ALU GEMV kernels: whole rows of row-major W, or 32-row
// blocks of tiled W.
int launch_skinny(const void* A, int prec, int64_t lda, int64_t pstride, const void* W, int w_type, int64_t ldw,
                  const float* C, int64_t ldc, float* Out, int64_t ldo, int64_t M, int64_t N,
                  int64_t K, void* ws, size_t ws_bytes, hipStream_t s)
{
    if (M == 0 || N == 0) return SPLITEE_OK;
    if (M > 16 || prec == SPLITEE_PREC_F32) return SPLITEE_ERR_UNSUPPORTED;
    const int npl = prec == SPLITEE_PREC_BF16X3 ? 3 : 1;
    const bool tiled = w_type == SPLITEE_BF16_TILED;
    const int64_t wbytes = tiled ? (int64_t)splitee::tiled_weights_bytes(N, K) : N * ldw * 2;
    if ((npl - 1) * pstride * 2 + M * lda * 2 >= (int64_t(1) << 31) || wbytes >= (int64_t(1) << 31))
        return SPLITEE_ERR_UNSUPPORTED;
    const SkSrc src{reinterpret_cast<const uint16_t*>(A), lda, pstride, nullptr, 0, nullptr, 0};
    if (M <= GV_MMAX)
        return tiled ? run_gemv_tiled<false>(src, prec, W, C, ldc, Out, ldo, M, N, K, ws, ws_bytes, s)
                     : launch_gemv<false>(src, prec, W, ldw, C, ldc, Out, ldo, M, N, K, s);
    return run_skinny<false>(src, prec, W, tiled, ldw, C, ldc, Out, ldo, M, N, K, ws, ws_bytes, s);
}

int launch_skinny_masked(const float* X, int64_t ldx, const float* eta, int64_t ld_eta, int prec,
                         const void* W, int w_type, int64_t ldw, const float* C, int64_t ldc, float* Out,
                         int64_t ldo, int64_t M, int64_t N, int64_t K, void* ws, size_t ws_bytes, hipStream_t s)
{
    if (M == 0 || N == 0) return SPLITEE_OK;
    if (M > 16 || prec == SPLITEE_PREC_F32) return SPLITEE_ERR_UNSUPPORTED;
    if (!X || !eta) return SPLITEE_ERR_ARG;
    if (K % 8 != 0 || ld_eta < K || ldx < K) return SPLITEE_ERR_SHAPE;
    const bool tiled = w_type == SPLITEE_BF16_TILED;
    const int64_t wbytes = tiled ? (int64_t)splitee::tiled_weights_bytes(N, K) : N * ldw * 2;
    if (M * ld_eta * 4 >= (int64_t(1) << 31) || M * ldx * 4 >= (int64_t(1) << 31) || wbytes >= (int64_t(1) << 31))
        return SPLITEE_ERR_UNSUPPORTED;
    const SkSrc src{nullptr, 0, 0, X, ldx, eta, ld_eta};
    if (M <= GV_MMAX)
        return tiled ? run_gemv_tiled<true>(src, prec, W, C, ldc, Out, ldo, M, N, K, ws, ws_bytes, s)
                     : launch_gemv<true>(src, prec, W, ldw, C, ldc, Out, ldo, M, N, K, s);
    return run_skinny<true>(src, prec, W, tiled, ldw, C, ldc, Out, ldo, M, N, K, ws, ws_bytes, s);
}

// The streamed GEMM with the masked input formed in-kernel from X and a given mask eta
// (both M x K float32), for the plans with 64-row tiles on tiled W (M <= 128);
// SPLITEE_ERR_UNSUPPORTED for any other plan, which the caller then runs as the mask
// launch followed by launch_gemm.
int launch_gemm_masked(const float* X, int64_t ldx, const float* eta, int64_t ld_eta, int prec, const void* W,
                       int w_type, const float* C, int64_t ldc, float* Out, int64_t ldo, int64_t M, int64_t N,
                       int64_t K, void* ws, size_t ws_bytes, hipStream_t s)
{
    if (M == 0 || N == 0) return SPLITEE_OK;
    if (prec == SPLITEE_PREC_F32 || w_type != SPLITEE_BF16_TILED || M > 128) return SPLITEE_ERR_UNSUPPORTED;
    if (!X || !eta) return SPLITEE_ERR_ARG;
    if (K % 8 != 0 || ld_eta < K || ldx < K) return SPLITEE_ERR_SHAPE;
    if (M * ld_eta * 4 >= (int64_t(1) << 31) || M * ldx * 4 >= (int64_t(1) << 31) ||
        (int64_t)splitee::tiled_weights_bytes(N, K) >= (int64_t(1) << 31))
        return SPLITEE_ERR_UNSUPPORTED;
    const bool allow_split = ws != nullptr;
    Plan p = plan_tiled(M, N, K, prec, w_type, allow_split);
    if (p.variant != 24 && p.variant != 25 && p.variant != 26 && p.variant != 27) return SPLITEE_ERR_UNSUPPORTED;
    if (p.ksplit > 1 && ws_bytes < p.counter_bytes + p.part_bytes) return SPLITEE_ERR_WORKSPACE;
    if (p.part_bytes >= (size_t(1) << 31)) return SPLITEE_ERR_UNSUPPORTED; // the sum kernel's buffer offsets
    float* pp = reinterpret_cast<float*>(ws);
    const uint16_t* w = reinterpret_cast<const uint16_t*>(W);
    dim3 grid((unsigned)(p.mtiles * p.ntiles * p.ksplit));
    const int m = (int)M, n = (int)N, k = (int)K;
#define SM_LAUNCH(NP, BM_, BN_, WGM_, D_) hipLaunchKernelGGL((gemm_stream_masked_kernel<NP, BM_, BN_, WGM_, D_, 8>), grid, dim3(8 * WAVE), 0, s, X, ldx, eta, ld_eta, w, C, ldc, Out, ldo, m, n, k, p.mtiles, p.ntiles, p.ksplit, p.kt_per_split, pp)
    switch (p.variant) {
    case 24: SM_LAUNCH(3, 64, 256, 1, 2); break;
    case 25: SM_LAUNCH(1, 64, 256, 1, 2); break;
    case 26: SM_LAUNCH(3, 64, 128, 2, 3); break;
    default: SM_LAUNCH(1, 64, 128, 2, 3); break;
    }
#undef SM_LAUNCH
    if (p.ksplit > 1) {
        const int tiles = p.mtiles * p.ntiles;
        const int64_t units = (int64_t)tiles * p.bm * p.bn / 4;
        const dim3 g2((unsigned)((units + 255) / 256));
        if (p.variant == 24 || p.variant == 25)
            hipLaunchKernelGGL((stream_sum_kernel<64, 256, 1, 8>), g2, dim3(256), 0, s, pp, p.ksplit, C, ldc, Out, ldo, m, n, p.mtiles, tiles);
        else
            hipLaunchKernelGGL((stream_sum_kernel<64, 128, 2, 4>), g2, dim3(256), 0, s, pp, p.ksplit, C, ldc, Out, ldo, m, n, p.mtiles, tiles);
    }
    return hipGetLastError() == hipSuccess ? SPLITEE_OK : SPLITEE_ERR_HIP;
}

}  // namespace splitee_host
