/*
 * oracle/noise_ref.c -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow CPU reference for the noise stream of the DP-masked linear layer.
 * Only the test suite, the smoke check and the CPU-baseline leg of the benchmark
 * may load this code; the product path never does.  It shares no code, header or
 * constant table with the HIP library.
 *
 * What the paper fixes (Prop. 2; Sec. "Making the Process Differentially Private"):
 * the mask is eta ~ N(0, (Delta/eps)^2 I), drawn per token and never reused
 * (Sec. "Precomputing the Mask and Noise Correction").  The paper names no random
 * number generator, counter scheme or rounding; the reading implemented here
 * (one of the build's stated readings) is:
 *
 *   element (i, k) of an M x K block, absolute index e = (row0 + i) * K + k,
 *   block b = e / 4, lane = e % 4,
 *   (w0..w3) = Philox4x32-10(counter = (b_lo, b_hi, sid_lo, sid_hi),
 *                            key     = (seed_lo, seed_hi))
 *   [Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3",
 *    SC'11: multipliers 0xD2511F53 / 0xCD9E8D57, Weyl key bumps 0x9E3779B9 /
 *    0xBB67AE85, ten rounds],
 *   u(w) = (w + 1/2) * 2^-32 in (0, 1), exact in binary64,
 *   s = fl64(Delta / eps),
 *   Laplace:  t = RN32(F^-1(u)),  F^-1(u) = ln(2u) for u < 1/2, -ln(2 - 2u) otherwise
 *             eta = RN32(fl64(s * t))
 *   Gaussian: words (w0,w1) feed lanes 0,1 and (w2,w3) feed lanes 2,3 (Box-Muller):
 *             r = RN32(sqrt(-2 ln u(w_a))),  c = RN32(cos 2 pi u(w_b)), s' = RN32(sin 2 pi u(w_b))
 *             even lane: eta = RN32(fl64(s * (r * c)))   (r * c is exact in binary64)
 *             odd lane:  eta = RN32(fl64(s * (r * s')))
 *   None:     eta = 0.
 *
 * RN32(f) denotes the correctly rounded (nearest-even) binary32 value of the real
 * number f.  The oracle evaluates f in binary128 (libquadmath) and rounds; it
 * checks that the binary128 value is far (2^-100 relative) from every binary32
 * rounding boundary, so the rounding cannot depend on the last bits of the
 * binary128 evaluation.  A value too close to a boundary is reported through the
 * status code instead of being returned silently.
 */
#include <math.h>
#include <omp.h>
#include <quadmath.h>
#include <stdint.h>
#include <string.h>

#define ORC_OK 0
#define ORC_ERR_SHAPE (-2)
#define ORC_ERR_ARG (-1)
#define ORC_ERR_HARD_ROUNDING (-7)

/* Number of OpenMP threads the oracle runs on. */
int oracle_num_threads(void) { return omp_get_max_threads(); }

/* ---- Philox4x32-10 -------------------------------------------------------- */

static void philox_round(uint32_t c[4], const uint32_t k[2])
{
    uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c[0];
    uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c[2];
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c[1] ^ k[0];
    uint32_t n1 = lo1;
    uint32_t n2 = hi0 ^ c[3] ^ k[1];
    uint32_t n3 = lo0;
    c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
}

void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
    uint32_t k[2] = {key[0], key[1]};
    for (int r = 0; r < 10; ++r) {
        philox_round(c, k);
        k[0] += 0x9E3779B9u;
        k[1] += 0xBB67AE85u;
    }
    memcpy(out, c, sizeof(c));
}

/* ---- correctly rounded binary32 of a binary128 value ---------------------- */

/* Returns RN32(q) and sets *hard when q lies within 2^-100 |q| of a binary32
 * rounding boundary (the midpoint between two neighbouring binary32 values). */
static float round32_checked(__float128 q, int *hard)
{
    float f = (float)q; /* libgcc's binary128 -> binary32 conversion rounds to nearest even */
    __float128 up = (__float128)nextafterf(f, INFINITY);
    __float128 dn = (__float128)nextafterf(f, -INFINITY);
    __float128 mid_up = ((__float128)f + up) / 2;
    __float128 mid_dn = ((__float128)f + dn) / 2;
    __float128 d1 = fabsq(q - mid_up), d2 = fabsq(q - mid_dn);
    __float128 d = d1 < d2 ? d1 : d2;
    if (d <= fabsq(q) * 0x1p-100Q) *hard = 1;
    return f;
}

static __float128 word_to_u(uint32_t w) { return ((__float128)w + 0.5Q) * 0x1p-32Q; }

/* Inverse CDF of the standard Laplace law at u(w). */
float oracle_laplace_t(uint32_t w, int *hard)
{
    __float128 t;
    if (w < 0x80000000u) {
        __float128 a = (2.0Q * (__float128)w + 1.0Q) * 0x1p-32Q; /* = 2u, exact */
        t = logq(a);
    } else {
        __float128 a = (0x1p33Q - 2.0Q * (__float128)w - 1.0Q) * 0x1p-32Q; /* = 2 - 2u, exact */
        t = -logq(a);
    }
    return round32_checked(t, hard);
}

/* Box-Muller radius sqrt(-2 ln u(w)). */
float oracle_gauss_r(uint32_t w, int *hard)
{
    __float128 u = word_to_u(w);
    return round32_checked(sqrtq(-2.0Q * logq(u)), hard);
}

/* sin and cos of 2 pi u(w).  The argument is reduced exactly to an octant
 * before the binary128 library call, so no accuracy is lost near the zeros. */
static void sincos2pi_q(uint32_t w, __float128 *s_out, __float128 *c_out)
{
    uint64_t j = 2ull * (uint64_t)w + 1ull; /* u = j / 2^33, j odd */
    int oct = (int)(j >> 30);               /* floor(8u) */
    uint64_t jf = j - ((uint64_t)oct << 30); /* f = u - oct/8 = jf / 2^33, in (0, 1/8) */
    __float128 twopi = 2.0Q * M_PIq;
    __float128 g = twopi * ((__float128)jf * 0x1p-33Q);
    __float128 h = twopi * ((__float128)((1ull << 30) - jf) * 0x1p-33Q);
    __float128 sg = sinq(g), cg = cosq(g), sh = sinq(h), ch = cosq(h);
    __float128 s, c;
    switch (oct) {
    case 0: s = sg;  c = cg;  break; /* theta = g            */
    case 1: s = ch;  c = sh;  break; /* theta = pi/2 - h     */
    case 2: s = cg;  c = -sg; break; /* theta = pi/2 + g     */
    case 3: s = sh;  c = -ch; break; /* theta = pi - h       */
    case 4: s = -sg; c = -cg; break; /* theta = pi + g       */
    case 5: s = -ch; c = -sh; break; /* theta = 3pi/2 - h    */
    case 6: s = -cg; c = sg;  break; /* theta = 3pi/2 + g    */
    default: s = -sh; c = ch; break; /* theta = 2pi - h      */
    }
    *s_out = s;
    *c_out = c;
}

float oracle_cos2pi(uint32_t w, int *hard)
{
    __float128 s, c;
    sincos2pi_q(w, &s, &c);
    return round32_checked(c, hard);
}

float oracle_sin2pi(uint32_t w, int *hard)
{
    __float128 s, c;
    sincos2pi_q(w, &s, &c);
    return round32_checked(s, hard);
}

/* fn: 0 Laplace t, 1 Gaussian radius, 2 cos 2 pi u, 3 sin 2 pi u.
 * Returns the number of words whose value was too close to a rounding boundary. */
int64_t oracle_transform_batch(int fn, const uint32_t *w, int64_t n, float *out)
{
    int64_t nhard = 0;
#pragma omp parallel for schedule(static) reduction(+ : nhard)
    for (int64_t i = 0; i < n; ++i) {
        int hard = 0;
        float v;
        switch (fn) {
        case 0: v = oracle_laplace_t(w[i], &hard); break;
        case 1: v = oracle_gauss_r(w[i], &hard); break;
        case 2: v = oracle_cos2pi(w[i], &hard); break;
        default: v = oracle_sin2pi(w[i], &hard); break;
        }
        out[i] = v;
        nhard += hard;
    }
    return nhard;
}

void oracle_philox_batch(const uint64_t *blocks, int64_t n, uint64_t seed, uint64_t sid,
                         uint32_t *out /* n x 4 */)
{
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        uint32_t ctr[4] = {(uint32_t)blocks[i], (uint32_t)(blocks[i] >> 32), (uint32_t)sid,
                           (uint32_t)(sid >> 32)};
        oracle_philox4x32_10(ctr, key, out + 4 * i);
    }
}

/* ---- the noise block ------------------------------------------------------ */

enum { MECH_LAPLACE = 0, MECH_GAUSSIAN = 1, MECH_NONE = 2 };

/* eta is M x K, row-major with leading dimension ld (elements). */
int oracle_noise(float *eta, int64_t ld, int64_t M, int64_t K, int mech, double delta,
                 double eps, uint64_t seed, uint64_t sid, uint64_t row0)
{
    if (M < 0 || K < 0 || ld < K) return ORC_ERR_SHAPE;
    if (K % 4 != 0) return ORC_ERR_SHAPE;
    if (mech < 0 || mech > 2) return ORC_ERR_ARG;
    if (!(eps > 0.0) || !isfinite(eps) || !(delta >= 0.0) || !isfinite(delta)) return ORC_ERR_ARG;
    const double s = delta / eps;
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    int64_t nhard = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(+ : nhard)
    for (int64_t i = 0; i < M; ++i) {
        for (int64_t k = 0; k < K; k += 4) {
            uint64_t e = (row0 + (uint64_t)i) * (uint64_t)K + (uint64_t)k;
            uint64_t b = e >> 2;
            uint32_t ctr[4] = {(uint32_t)b, (uint32_t)(b >> 32), (uint32_t)sid,
                               (uint32_t)(sid >> 32)};
            uint32_t w[4];
            oracle_philox4x32_10(ctr, key, w);
            for (int lane = 0; lane < 4; ++lane) {
                float v;
                int hard = 0;
                if (mech == MECH_NONE) {
                    v = 0.0f;
                } else if (mech == MECH_LAPLACE) {
                    float t = oracle_laplace_t(w[lane], &hard);
                    v = (float)(s * (double)t);
                } else {
                    int p = lane >> 1;
                    float r = oracle_gauss_r(w[2 * p], &hard);
                    float c = (lane & 1) ? oracle_sin2pi(w[2 * p + 1], &hard)
                                         : oracle_cos2pi(w[2 * p + 1], &hard);
                    double rc = (double)r * (double)c; /* exact: 24 + 24 bits */
                    v = (float)(s * rc);
                }
                eta[i * ld + k + lane] = v;
                nhard += hard;
            }
        }
    }
    return nhard ? ORC_ERR_HARD_ROUNDING : ORC_OK;
}
