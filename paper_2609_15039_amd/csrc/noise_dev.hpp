// Device-side noise stream of the masked linear layer (gfx950): Philox4x32-10
// words and the correctly rounded binary32 transforms (Laplace inverse CDF,
// Box-Muller radius and angle) scaled by Delta / eps.  The noise law is Prop. 2
// (Gaussian, std Delta/eps) or Laplace of scale Delta/eps; the generator and the
// rounding are the library's definition given in include/splitee.h.  Every
// transform value is the correctly rounded binary32 value of the real function:
// it is evaluated in binary64 and kept when the binary64 value is on the right
// side of every binary32 rounding boundary by more than a relative error budget
// of 2^-48 (at least 16 binary64 ulps, above the error of the log, sqrt, sin and
// cos written here for the transforms' arguments), and otherwise
// recomputed in double-double arithmetic (about 100 correct bits) -- Ziv's
// strategy.  Included by the noise / mask kernels and by the decode GEMM, which
// generates its masked-input slice itself.
#pragma once
#include "common.hpp"
#include "noise_tables.hpp"
#include <math.h>

#pragma clang fp contract(off)

namespace {  // internal to each translation unit that includes this header

// ------------------------------------------------------------- Philox4x32-10
// Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC'11.
struct u32x4 { uint32_t x, y, z, w; };

__device__ __forceinline__ u32x4 philox4x32_10(u32x4 c, uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        // the full 64-bit products: one v_mad_u64_u32 each instead of a mul_lo / mul_hi pair
        const uint64_t p0 = (uint64_t)0xD2511F53u * c.x, p1 = (uint64_t)0xCD9E8D57u * c.z;
        c = u32x4{(uint32_t)(p1 >> 32) ^ c.y ^ k0, (uint32_t)p1, (uint32_t)(p0 >> 32) ^ c.w ^ k1, (uint32_t)p0};
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return c;
}

// --------------------------------------------------- double-double arithmetic
// Dekker (1971) / Knuth error-free transformations; fma gives the exact product
// error.  Contraction is off in this file so every other operation is one IEEE
// binary64 rounding.
struct dd { double hi, lo; };

__device__ __forceinline__ dd two_sum(double a, double b)
{
    double s = a + b, bb = s - a;
    return dd{s, (a - (s - bb)) + (b - bb)};
}
__device__ __forceinline__ dd fast_two_sum(double a, double b)
{
    double s = a + b;
    return dd{s, b - (s - a)};
}
__device__ __forceinline__ dd two_prod(double a, double b)
{
    double p = a * b;
    return dd{p, __builtin_fma(a, b, -p)};
}
__device__ __forceinline__ dd dd_add(dd x, dd y)
{
    dd s = two_sum(x.hi, y.hi), t = two_sum(x.lo, y.lo);
    s.lo += t.hi;
    s = fast_two_sum(s.hi, s.lo);
    s.lo += t.lo;
    return fast_two_sum(s.hi, s.lo);
}
__device__ __forceinline__ dd dd_neg(dd x) { return dd{-x.hi, -x.lo}; }
__device__ __forceinline__ dd dd_mul(dd x, dd y)
{
    dd p = two_prod(x.hi, y.hi);
    p.lo += x.hi * y.lo + x.lo * y.hi;
    return fast_two_sum(p.hi, p.lo);
}
__device__ __forceinline__ dd dd_mul_d(dd x, double y)
{
    dd p = two_prod(x.hi, y);
    p.lo += x.lo * y;
    return fast_two_sum(p.hi, p.lo);
}
__device__ __forceinline__ dd dd_div(dd a, dd b)
{
    double q1 = a.hi / b.hi;
    dd r = dd_add(a, dd_neg(dd_mul_d(b, q1)));
    double q2 = r.hi / b.hi;
    r = dd_add(r, dd_neg(dd_mul_d(b, q2)));
    double q3 = r.hi / b.hi;
    dd q = fast_two_sum(q1, q2);
    return dd_add(q, dd{q3, 0.0});
}
__device__ __forceinline__ dd dd_div_d(dd a, double b) { return dd_div(a, dd{b, 0.0}); }

// ln 2 and 2 pi as double-double (each pair within 1e-32 relative of the constant)
#define DD_LN2_HI 0x1.62e42fefa39efp-1
#define DD_LN2_LO 0x1.abc9e3b39803fp-56
#define DD_2PI_HI 0x1.921fb54442d18p+2
#define DD_2PI_LO 0x1.1a62633145c07p-52

// ln x for a positive normal binary64 x.  x = m 2^e with m in [sqrt(1/2), sqrt(2)),
// ln m = 2 atanh(s), s = (m - 1)/(m + 1), |s| < 0.172, and
// atanh(s)/s = sum_k s^(2k) / (2k + 1), 25 terms (s^50 < 2^-127).
__device__ __attribute__((noinline)) dd dd_log(double x)
{
    int e;
    double m = frexp(x, &e); // m in [1/2, 1)
    if (m < 0.70710678118654752440) {
        m *= 2.0;
        e -= 1;
    }
    dd num = two_sum(m, -1.0), den = two_sum(m, 1.0);
    dd s = dd_div(num, den);
    dd z = dd_mul(s, s);
    const int NT = 25;
    dd acc = dd_div_d(dd{1.0, 0.0}, (double)(2 * NT + 1));
    for (int k = NT - 1; k >= 0; --k)
        acc = dd_add(dd_mul(acc, z), dd_div_d(dd{1.0, 0.0}, (double)(2 * k + 1)));
    dd lnm = dd_mul_d(dd_mul(s, acc), 2.0);
    dd eln2 = dd_add(two_prod((double)e, DD_LN2_HI), dd{(double)e * DD_LN2_LO, 0.0});
    return dd_add(eln2, lnm);
}

__device__ dd dd_sqrt(dd v)
{
    double r = sqrt(v.hi);
    dd r2 = two_prod(r, r);
    double corr = ((v.hi - r2.hi) - r2.lo + v.lo) / (2.0 * r);
    return fast_two_sum(r, corr);
}

// sin and cos of g = 2 pi f for exact f in [0, 1/8], Taylor series to degree 31.
__device__ void dd_sincos_2pi_small(double f, dd& sn, dd& cs)
{
    dd g = dd_add(two_prod(DD_2PI_HI, f), dd{DD_2PI_LO * f, 0.0});
    dd g2 = dd_mul(g, g);
    dd ts = g, ssum = g, tc = dd{1.0, 0.0}, csum = dd{1.0, 0.0};
    for (int n = 1; n <= 15; ++n) {
        ts = dd_div_d(dd_mul(ts, g2), (double)((2 * n) * (2 * n + 1)));
        tc = dd_div_d(dd_mul(tc, g2), (double)((2 * n - 1) * (2 * n)));
        if (n & 1) {
            ssum = dd_add(ssum, dd_neg(ts));
            csum = dd_add(csum, dd_neg(tc));
        } else {
            ssum = dd_add(ssum, ts);
            csum = dd_add(csum, tc);
        }
    }
    sn = ssum;
    cs = csum;
}

// sin and cos of 2 pi u(w) in double-double: octant reduction of the exact
// u = j / 2^33 (j = 2w + 1), then the series on an argument in [0, pi/4].  Returned
// by value (in registers), so that the kernels that call it need no scratch memory.
struct dd_pair { dd s, c; };
__device__ __attribute__((noinline)) dd_pair dd_sincos_2pi(uint32_t w)
{
    uint64_t j = 2ull * (uint64_t)w + 1ull;
    int oct = (int)(j >> 30);
    uint64_t jf = j - ((uint64_t)oct << 30);
    double f = (double)jf * 0x1p-33;                     // u - oct/8
    double h = (double)((1ull << 30) - jf) * 0x1p-33;    // (oct+1)/8 - u
    // angle within the octant measured from its nearer axis: even octants from
    // the start (f), odd octants from the end (h)
    dd s1, c1;
    dd_sincos_2pi_small((oct & 1) ? h : f, s1, c1);
    dd s, c;
    switch (oct) {
    case 0: s = s1;         c = c1;         break;
    case 1: s = c1;         c = s1;         break;
    case 2: s = c1;         c = dd_neg(s1); break;
    case 3: s = s1;         c = dd_neg(c1); break;
    case 4: s = dd_neg(s1); c = dd_neg(c1); break;
    case 5: s = dd_neg(c1); c = dd_neg(s1); break;
    case 6: s = dd_neg(c1); c = s1;         break;
    default: s = dd_neg(s1); c = c1;        break;
    }
    return dd_pair{s, c};
}

// --------------------------------------------------- rounding to binary32

// Neighbour of nonzero finite binary32 f in the direction of `up` (toward +inf if up).
__device__ __forceinline__ float f32_step(float f, bool up)
{
    uint32_t b = __float_as_uint(f);
    bool mag_up = (up == (f > 0.0f));
    return __uint_as_float(mag_up ? b + 1u : b - 1u);
}

// RN32 of a double-double value (hi + lo, |lo| <= ulp(hi)/2).  Only when hi is
// exactly a binary32 midpoint can lo change the result.
__device__ __forceinline__ float round_dd_f32(dd v)
{
    float f = (float)v.hi;
    double fd = (double)f;
    if (v.hi != fd && v.lo != 0.0) {
        float g = f32_step(f, v.hi > fd);
        double mid = 0.5 * (fd + (double)g);
        if (v.hi == mid) {
            bool toward_g = (g > f) ? (v.lo > 0.0) : (v.lo < 0.0);
            return toward_g ? g : f;
        }
    }
    return f;
}

// RN32(r) is the correctly rounded value of the real function whenever the true
// value lies within |r| 2^-48 of r and no binary32 midpoint lies that close to r.
// In the binade [2^E, 2^(E+1)) of r the binary32 midpoints are the odd multiples of
// 2^(E-24), i.e. the binary64 values whose low 29 significand bits read 2^28, and
// |r| 2^-48 < 2^(E-47) is 32 units of r's last place, 2^(E-52); the nearest midpoint
// outside the binade is at least 2^(E-25) away.  So r is safe iff its low 29 bits
// differ from 2^28 by more than 32 (an exact integer test), provided RN32(r) is a
// normal binary32 number (else the slow path).
__device__ __forceinline__ bool round_f32_safe(double r, float& out)
{
    out = (float)r;
    const uint64_t b = (uint64_t)__double_as_longlong(r);
    const uint32_t lo = (uint32_t)b & 0x1FFFFFFFu;
    const uint32_t ex = (uint32_t)(b >> 52) & 0x7FFu;
    const uint32_t d = lo > 0x10000000u ? lo - 0x10000000u : 0x10000000u - lo;
    return d > 32u && ex >= 1023u - 126u && ex <= 1023u + 126u;
}

// -------------------------------------- binary64 log, sin(pi x), cos(pi x): fast path
// Written for the arguments the transforms pass: log of a positive normal x with
// at most 33 significant bits in (2^-34, 1), sqrt of -2 log u, sin / cos of pi x for
// x = (2w + 1) 2^-32.
// Each stays within a few binary64 ulps (relative error about 2^-51), inside the
// 2^-48 budget of round_f32_safe; the fast and slow paths of every transform are
// compared on all 2^32 words.  Both reductions read a small table written by
// gen_noise_tables.py (noise_tables.hpp).

// ln 2 = LN2_HI + LN2_LO to about 2^-98; LN2_HI has 44 significant bits, so e LN2_HI
// is exact for every binary64 exponent e.
constexpr double LN2_HI = 0x1.62e42fefa38p-1;
constexpr double LN2_LO = 0x1.ef35793c7673p-45;
// pi = PI_HI + PI_LO to about 2^-74; PI_HI has 22 significant bits, so PI_HI d is exact
// for d = k 2^-32, |k| <= 2^30.
constexpr double PI_HI = 0x1.921fbp+1;
constexpr double PI_LO = 0x1.5110b4611a626p-21;

// log x = e ln 2 - log rc + log1p(r) for x = 2^e m', with m' in [0.70703125, 1.4140625)
// (the binary64 significand, halved when its top 7 fraction bits i are 53 or more),
// rc the table's reciprocal of the centre of entry i (20 significant bits, or 1 next
// to m' = 1) and r = m' rc - 1, exact because m' has at most 33 significant bits;
// |r| <= 2^-7, so log1p(r) to r^8 leaves out less than 2^-59 of its value, and -log rc
// comes from the table as hi + lo.  Near x = 1 (rc = 1) nothing cancels.
__device__ __forceinline__ double log_fast(double x)
{
    const uint64_t b = (uint64_t)__double_as_longlong(x);
    int e = (int)(b >> 52) - 1023;
    const int i = (int)((b >> 45) & 127u);
    uint64_t mb = (b & 0x000FFFFFFFFFFFFFull) | 0x3FF0000000000000ull; // m in [1, 2)
    if (i >= 53) { mb -= 0x0010000000000000ull; ++e; }                 // m' = m / 2
    const double m = __longlong_as_double((long long)mb);
    const double2 t0 = *reinterpret_cast<const double2*>(&NOISE_LOG_TABLE[i][0]); // rc, -log rc (hi)
    const double t1 = NOISE_LOG_TABLE[i][2];                                       // -log rc (lo)
    const double r = fma(m, t0.x, -1.0);
    const double z = r * r;
    double p = -1.0 / 8.0;
    p = fma(p, r, 1.0 / 7.0);
    p = fma(p, r, -1.0 / 6.0);
    p = fma(p, r, 1.0 / 5.0);
    p = fma(p, r, -0.25);
    p = fma(p, r, 1.0 / 3.0);
    p = fma(p, r, -0.5);
    const double l1p = fma(z, p, r); // r - r^2/2 + r^3/3 - ... - r^8/8
    const double de = (double)e;
    return fma(de, LN2_HI, t0.y) + fma(de, LN2_LO, t1 + l1p);
}

// sqrt v for positive normal v, within about one binary64 ulp: the hardware
// reciprocal square root refined by two coupled Newton steps on (g, h) ~ (sqrt v,
// 1 / (2 sqrt v)) and a final correction g + h (v - g^2) (Goldschmidt's method).
__device__ __forceinline__ double sqrt_fast(double v)
{
    const double y = __builtin_amdgcn_rsq(v);
    double g = v * y, h = 0.5 * y;
    double r = fma(-g, h, 0.5);
    g = fma(g, r, g);
    h = fma(h, r, h);
    r = fma(-g, h, 0.5);
    g = fma(g, r, g);
    h = fma(h, r, h);
    return fma(fma(-g, g, v), h, g);
}

// sin(pi x) and cos(pi x) for x = (2w + 1) 2^-32 in (0, 2): x = j/64 + d with j the nearest
// integer to 64x (0..128) and |d| <= 2^-7 + 2^-32, both exact in 32-bit integer arithmetic;
// sin and cos of pi d by Taylor polynomials to degree 7 and 8 (|pi d| <= pi/128: the first
// terms left out are below 2^-61 of the value), combined with the table's sin and cos of
// pi j / 64 (the whole circle, exact zeros) by the angle-sum formulas.  Next to a zero of sin
// or cos the table's entry there is 0 and the result is +-sin(pi d) itself; elsewhere no more
// than one bit cancels.
__device__ __forceinline__ void sincospi_fast(uint32_t w, double& sn, double& cs)
{
    // 64x = (w + 1/2) 2^-25, so j = (w >> 25) + bit 24 of w, and x - j/64 = dn 2^-32 with
    // dn = 2 (w - j 2^25) + 1 (j 2^25 taken modulo 2^32: j = 128 only for w near 2^32)
    const uint32_t j = (w >> 25) + ((w >> 24) & 1u);
    const int32_t dn = 2 * (int32_t)(w - (j << 25)) + 1;
    const double d = (double)dn * 0x1p-32;
    const double t = fma(PI_LO, d, PI_HI * d);     // pi d
    const double z = t * t;
    double ps = -1.0 / 5040.0;                     // 1/7!
    ps = fma(ps, z, 1.0 / 120.0);                  // 1/5!
    ps = fma(ps, z, -1.0 / 6.0);                   // 1/3!
    const double st = fma(t * z, ps, t);           // sin(pi d)
    double pc = 1.0 / 40320.0;                     // 1/8!
    pc = fma(pc, z, -1.0 / 720.0);                 // 1/6!
    pc = fma(pc, z, 1.0 / 24.0);                   // 1/4!
    pc = fma(pc, z, -0.5);                         // 1/2!
    const double ct = fma(z, pc, 1.0);             // cos(pi d)
    const double2 tab = *reinterpret_cast<const double2*>(&NOISE_SINCOS_TABLE[j][0]);
    sn = fma(tab.x, ct, tab.y * st);               // sin(pi (j/64 + d))
    cs = fma(tab.y, ct, -(tab.x * st));            // cos(pi (j/64 + d))
}

// ---------------------------------------------------- the four transforms

__device__ __forceinline__ float cr_laplace_t(uint32_t w, bool force_slow)
{
    const bool upper = w >= 0x80000000u;
    // 2u = (2w + 1) 2^-32 and 2 - 2u = (2^33 - 2w - 1) 2^-32, both exact
    const uint64_t j = upper ? ((1ull << 33) - 2ull * (uint64_t)w - 1ull) : (2ull * (uint64_t)w + 1ull);
    const double x = (double)j * 0x1p-32;
    float f;
    if (force_slow || !round_f32_safe(log_fast(x), f)) f = round_dd_f32(dd_log(x));
    return upper ? -f : f;
}

__device__ __forceinline__ float cr_gauss_r(uint32_t w, bool force_slow)
{
    const double u = ((double)w + 0.5) * 0x1p-32;
    float f;
    if (force_slow || !round_f32_safe(sqrt_fast(-2.0 * log_fast(u)), f))
        f = round_dd_f32(dd_sqrt(dd_mul_d(dd_log(u), -2.0)));
    return f;
}

__device__ __forceinline__ void cr_sincos_2pi(uint32_t w, bool force_slow, float& sn, float& cs)
{
    double s64, c64;
    sincospi_fast(w, s64, c64); // of 2u = (2w + 1) 2^-32
    bool ok_s = !force_slow && round_f32_safe(s64, sn);
    bool ok_c = !force_slow && round_f32_safe(c64, cs);
    if (!(ok_s && ok_c)) {
        const dd_pair p = dd_sincos_2pi(w);
        if (!ok_s) sn = round_dd_f32(p.s);
        if (!ok_c) cs = round_dd_f32(p.c);
    }
}

// eta for the four elements of Philox block b (lanes 0..3): one Philox call, four
// Laplace transforms or two Box-Muller pairs (words (w0, w1) -> lanes 0, 1 and
// (w2, w3) -> lanes 2, 3).
__device__ __forceinline__ float4 noise_block(int mech, double scale, uint64_t b, uint32_t sid_lo, uint32_t sid_hi,
                                              uint32_t k0, uint32_t k1)
{
    if (mech == SPLITEE_MECH_NONE) return make_float4(0.f, 0.f, 0.f, 0.f);
    const u32x4 w = philox4x32_10(u32x4{(uint32_t)b, (uint32_t)(b >> 32), sid_lo, sid_hi}, k0, k1);
    float4 o;
    if (mech == SPLITEE_MECH_LAPLACE) {
        o.x = (float)(scale * (double)cr_laplace_t(w.x, false));
        o.y = (float)(scale * (double)cr_laplace_t(w.y, false));
        o.z = (float)(scale * (double)cr_laplace_t(w.z, false));
        o.w = (float)(scale * (double)cr_laplace_t(w.w, false));
    } else {
        const float r0 = cr_gauss_r(w.x, false), r1 = cr_gauss_r(w.z, false);
        float s0, c0, s1, c1;
        cr_sincos_2pi(w.y, false, s0, c0);
        cr_sincos_2pi(w.w, false, s1, c1);
        // r * c is exact in binary64 (24 + 24 significant bits)
        o.x = (float)(scale * ((double)r0 * (double)c0));
        o.y = (float)(scale * ((double)r0 * (double)s0));
        o.z = (float)(scale * ((double)r1 * (double)c1));
        o.w = (float)(scale * ((double)r1 * (double)s1));
    }
    return o;
}

// Half h (0 or 1) of Philox block b: lanes 2h and 2h + 1 of noise_block, i.e. the
// Box-Muller pair of words (w_2h, w_2h+1) or their two Laplace transforms.  Two
// threads that each take one half of a block produce noise_block's values with
// half of its serial chain of binary64 transforms each.
__device__ __forceinline__ float2 noise_half(int mech, double scale, uint64_t b, int h, uint32_t sid_lo,
                                             uint32_t sid_hi, uint32_t k0, uint32_t k1)
{
    if (mech == SPLITEE_MECH_NONE) return make_float2(0.f, 0.f);
    const u32x4 w = philox4x32_10(u32x4{(uint32_t)b, (uint32_t)(b >> 32), sid_lo, sid_hi}, k0, k1);
    const uint32_t wa = h ? w.z : w.x, wb = h ? w.w : w.y;
    float2 o;
    if (mech == SPLITEE_MECH_LAPLACE) {
        o.x = (float)(scale * (double)cr_laplace_t(wa, false));
        o.y = (float)(scale * (double)cr_laplace_t(wb, false));
    } else {
        const float r = cr_gauss_r(wa, false);
        float sn, cs;
        cr_sincos_2pi(wb, false, sn, cs);
        o.x = (float)(scale * ((double)r * (double)cs));
        o.y = (float)(scale * ((double)r * (double)sn));
    }
    return o;
}

}  // namespace
