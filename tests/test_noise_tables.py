"""The constant tables of the noise kernels' binary64 fast paths (noise_tables.hpp).

The header is what its generator writes, and the entries have the properties the
fast paths rely on, checked here by other means than the generator's: exact
rational arithmetic for the log reduction's reciprocals, exp of the stored
logarithms against the reciprocals, and identities of sin and cos.  (The fast paths
themselves are checked against the double-double slow paths on every 32-bit word by
the GPU suite.)
"""
import contextlib
import io
import math
import re
import runpy
from decimal import Decimal, localcontext
from fractions import Fraction
from pathlib import Path

CSRC = Path(__file__).resolve().parents[1] / "paper_2609_15039_amd" / "csrc"


def _tables():
    text = (CSRC / "noise_tables.hpp").read_text()
    log_part, sc_part = text.split("NOISE_SINCOS_TABLE")
    log = [tuple(float.fromhex(v) for v in row)
           for row in re.findall(r"\{(\S+), (\S+), (\S+), 0\.0\},", log_part)]
    sc = [tuple(float.fromhex(v) for v in row) for row in re.findall(r"\{(\S+), (\S+)\},", sc_part)]
    return text, log, sc


def test_header_is_the_generator_output():
    text, _, _ = _tables()
    out = io.StringIO()
    with contextlib.redirect_stdout(out), localcontext():
        runpy.run_path(str(CSRC / "gen_noise_tables.py"), run_name="__main__")
    assert out.getvalue() == text


def test_log_reduction_entries():
    _, log, _ = _tables()
    assert len(log) == 128
    for i, (rc, hi, lo) in enumerate(log):
        m0, m1 = Fraction(128 + i, 128), Fraction(129 + i, 128)
        if i >= 53:
            m0, m1 = m0 / 2, m1 / 2
        q = Fraction(rc)
        # 20 significant bits: m' (33 bits at most) times rc is exact in binary64
        n = q.numerator
        while n % 2 == 0:
            n //= 2
        assert n.bit_length() <= 20 and q.denominator & (q.denominator - 1) == 0, i
        # |m' rc - 1| <= 2^-7 over the entry's half-open interval of m'
        assert max(abs(m0 * q - 1), abs(m1 * q - 1)) <= Fraction(1, 128), i
        if i in (0, 127):
            assert rc == 1.0 and hi == 0.0 and lo == 0.0
            continue
        # hi + lo = -log rc to about 2^-100: exp(hi + lo) rc = 1
        with localcontext() as ctx:
            ctx.prec = 60
            L = Decimal(hi) + Decimal(lo)
            assert abs(L.exp() * Decimal(rc) - 1) < Decimal(2) ** -100, i
        assert abs(lo) <= math.ulp(hi) / 2, i


def test_sincos_entries():
    _, _, sc = _tables()
    assert len(sc) == 129
    # the zeros and units of the whole circle exactly
    for j, v in ((0, (0.0, 1.0)), (32, (1.0, 0.0)), (64, (0.0, -1.0)), (96, (-1.0, 0.0)), (128, (0.0, 1.0))):
        assert sc[j] == v, j
    assert sc[16][0] == sc[16][1]
    for j, (s, c) in enumerate(sc):
        # math.sin / math.cos of the binary64 angle: within a few units of 2^-53 of the entry
        assert abs(s - math.sin(math.pi * j / 64)) <= 2.0 ** -50
        assert abs(c - math.cos(math.pi * j / 64)) <= 2.0 ** -50
        assert abs(s * s + c * c - 1.0) < 2.0 ** -51
    for j in range(1, 65):  # sin 2a = 2 sin a cos a, cos 2a = c^2 - s^2
        s, c = sc[j]
        assert abs(sc[2 * j][0] - 2 * s * c) < 2.0 ** -51
        assert abs(sc[2 * j][1] - (c * c - s * s)) < 2.0 ** -51
    for j in range(65):  # symmetries: sin(pi - a) = sin a, cos(pi - a) = -cos a, and the half turn
        assert sc[64 - j][0] == sc[j][0] and sc[64 - j][1] == -sc[j][1], j
        assert sc[64 + j][0] == -sc[j][0] and sc[64 + j][1] == -sc[j][1], j
