"""Rounding of the matrix-core instructions the GEMM kernels issue.

The tolerances of the GEMM tests rest on the dot-product bound gamma_n (Def. 6) and
on Theorem 4, which assume that every floating-point operation rounds to nearest
with unit roundoff u (2^-24 for binary32, 2^-53 for binary64).  An MFMA instruction
adds kb products to an accumulator in one step, in an order and at an internal
precision the ISA does not state, so the assumption is checked here on crafted
operands (splitee_mfma_probe, include/splitee_probe.h): every output element of the
tile receives the same value c + sum_k a_k b_k, and the cases are chosen so that
round to nearest even of the exact sum differs from truncation, from rounding each
product or each partial sum separately, from ties away from zero and from keeping
extra precision across a chain of instructions.

Model checked (M1): each instruction returns RN_even(c + sum_k a_k b_k), the exact
sum rounded once.  Under M1 an instruction's error is at most u |c + sum a b| <=
u (|c| + sum |a b|), so a chain of n instructions obeys the dot-product bound with
gamma_n; the kernels issue K / kb instructions per plane (three planes for BF16X3)
plus one addition per extra split, fewer than K roundings per output, so the
gamma_K of the tests' bounds covers them.

Expected values come from exact rational arithmetic here, never from the device.
"""
from fractions import Fraction as F

import pytest
import torch

import paper_2609_15039_amd as sp

pytestmark = pytest.mark.gpu

OPS = {  # op: (name, kb, tile elements, significand bits of the accumulator)
    0: ("v_mfma_f32_32x32x16_bf16", 16, 1024, 24),
    1: ("v_mfma_f32_16x16x32_bf16", 32, 256, 24),
    2: ("v_mfma_f32_16x16x4_f32", 4, 256, 24),
    3: ("v_mfma_f64_16x16x4_f64", 4, 256, 53),
}


def _exp2_floor(q):
    """e with 2^e <= q < 2^(e+1) for a positive rational q."""
    e = q.numerator.bit_length() - q.denominator.bit_length()
    while F(2) ** e > q:
        e -= 1
    while F(2) ** (e + 1) <= q:
        e += 1
    return e


def round_bin(q, p, mode="rne"):
    """q rounded to a binary format with p significand bits (normal range):
    'rne' to nearest, ties to even; 'rna' to nearest, ties away; 'rz' toward zero."""
    if q == 0:
        return F(0)
    s = -1 if q < 0 else 1
    a = abs(q)
    ulp = F(2) ** (_exp2_floor(a) - p + 1)
    m = a / ulp
    fl = m.numerator // m.denominator
    rem = m - fl
    if mode == "rne" and (rem > F(1, 2) or (rem == F(1, 2) and fl % 2 == 1)):
        fl += 1
    elif mode == "rna" and rem >= F(1, 2):
        fl += 1
    return s * fl * ulp


def model_chain(c, a, b, kb, p, mode="rne"):
    """M1 (mode 'rne') and its rivals 'rz' / 'rna': per instruction, the exact sum of
    the accumulator and the kb products rounded once."""
    acc = round_bin(F(c), p)
    for i in range(len(a) // kb):
        acc = round_bin(acc + sum(F(x) * F(y) for x, y in zip(a[i * kb:(i + 1) * kb], b[i * kb:(i + 1) * kb])),
                        p, mode)
    return acc


def sequential_chain(c, a, b, kb, p):
    """Rival: every product and every partial sum rounded, in k order."""
    acc = round_bin(F(c), p)
    for x, y in zip(a, b):
        acc = round_bin(acc + round_bin(F(x) * F(y), p), p)
    return acc


def exact_chain(c, a, b):
    """Rival: the whole chain kept exact (rounded only when read)."""
    return F(c) + sum(F(x) * F(y) for x, y in zip(a, b))


def cases(kb, p):
    """(name, c, a, b) with len(a) a multiple of kb; b is 1 unless stated."""
    u = 2.0 ** -p
    out = []

    def one(name, c, a_head, n=1, b_head=None):
        a = list(a_head) + [0.0] * (n * kb - len(a_head))
        b = list(b_head) + [1.0] * (n * kb - len(b_head)) if b_head else [1.0] * (n * kb)
        out.append((name, c, a, b))

    one("up: 1 + 1.5u", 1.0, [1.5 * u])                       # RN 1 + 2u, RZ 1
    one("down: 1 - u/4", 1.0, [-0.25 * u])                    # RN 1, RZ 1 - u
    one("tie to even below: 1 + u", 1.0, [u])                 # RNE 1, RNA 1 + 2u
    one("tie to even above: (1 + 2u) + u", 1.0 + 2 * u, [u])  # RNE 1 + 4u
    one("one rounding of the products: 1 + (kb - 1) 0.75u", 0.0, [1.0] + [0.75 * u] * (kb - 1))
    one("small terms first: (kb - 1) 0.75u + 1", 0.0, [0.75 * u] * (kb - 1) + [1.0])
    one("accumulator in the same rounding: 0.75u + 1 + 0.75u", 0.75 * u, [1.0, 0.75 * u])
    one("cancellation: 1 - 1 + 2^-40", 0.0, [1.0, -1.0, 2.0 ** -40])
    one("cancellation into the accumulator: 2^-40 + 1 - 1", 2.0 ** -40, [1.0, -1.0])
    one("exponent spread: 2^20 + 1 + 2^-20", 0.0, [2.0 ** 20, 1.0, 2.0 ** -20])
    one("negative: -1 - 1.5u", -1.0, [-1.5 * u])
    one("chain rounds per instruction: 1 + 8 x 0.75u", 1.0, [0.75 * u], n=8)
    if p == 53 or kb == 4:  # binary32 / binary64 operands: a product may need 2p bits
        e = 2.0 ** -(p - 1)
        one("product wider than p bits: (1 + 2^(1-p))^2 - 1", -1.0, [1.0 + e], b_head=[1.0 + e])
        one("product tail kept: (1 + 2^(1-p))^2 - 1 - 2^(2-p)", -1.0 - 2 * e, [1.0 + e], b_head=[1.0 + e])
    return out


@pytest.mark.parametrize("op", sorted(OPS))
def test_mfma_rounds_once_to_nearest_even(op):
    name, kb, tile, p = OPS[op]
    report, bad = [], []
    for cname, c, a, b in cases(kb, p):
        n = len(a) // kb
        ad = torch.tensor(a, dtype=torch.float64, device="cuda")
        bd = torch.tensor(b, dtype=torch.float64, device="cuda")
        d = torch.full((1024,), float("nan"), dtype=torch.float64, device="cuda")
        sp.splitee_mfma_probe(op, n, ad, bd, c, d)
        torch.cuda.synchronize()
        got = d[:tile].cpu()
        uniform = bool(torch.all(got == got[0]))
        g = F(float(got[0]))
        want = model_chain(c, a, b, kb, p)
        rivals = {"rz": model_chain(c, a, b, kb, p, "rz"), "rna": model_chain(c, a, b, kb, p, "rna"),
                  "sequential": sequential_chain(c, a, b, kb, p),
                  "exact chain": round_bin(exact_chain(c, a, b), p)}
        line = "%-55s got %r  M1 %r  %s" % (cname, float(g), float(want),
                                              "  ".join("%s %r" % (k, float(v)) for k, v in rivals.items()))
        report.append(line)
        if not uniform or g != want:
            bad.append(line + ("" if uniform else "  (tile not uniform)"))
    print("\n%s\n" % name + "\n".join(report))
    assert not bad, "%s departs from one round-to-nearest-even per instruction:\n%s" % (name, "\n".join(bad))
