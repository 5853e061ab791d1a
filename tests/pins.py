"""Independent references used to pin the oracle (no oracle code in here).

* rocRAND's header-only Philox4x32-10 engine, compiled with g++ as a host program.
* mpmath at 200 bits for the transforms, rounded to binary32 by comparing the two
  neighbouring binary32 candidates in mpmath precision.
"""
import functools
import os
import subprocess
import tempfile

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROCRAND_HDR = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"


@functools.lru_cache(maxsize=1)
def rocrand_words_exe():
    out_dir = tempfile.mkdtemp(prefix="rocrand_words_")
    exe = os.path.join(out_dir, "rocrand_words")
    subprocess.run(["g++", "-O2", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    os.path.join(HERE, "helpers", "rocrand_words.cpp"), "-o", exe],
                   check=True)
    return exe


def rocrand_words(seed, sid, offset, count):
    """Philox words number offset .. offset+count-1 of subsequence sid (rocRAND)."""
    res = subprocess.run([rocrand_words_exe(), str(seed), str(sid), str(offset), str(count)],
                         check=True, capture_output=True, text=True)
    return np.array([int(x, 16) for x in res.stdout.split()], dtype=np.uint32)


def _mp():
    import mpmath
    mpmath.mp.prec = 200
    return mpmath


def cr32(v):
    """Correctly rounded binary32 value of the mpmath number v."""
    mpmath = _mp()
    f = np.float32(float(v))
    cands = [f, np.nextafter(f, np.float32(np.inf)), np.nextafter(f, np.float32(-np.inf))]
    return min(cands, key=lambda c: abs(mpmath.mpf(float(c)) - v))


def mp_u(w):
    mpmath = _mp()
    return (mpmath.mpf(int(w)) + mpmath.mpf(0.5)) / mpmath.mpf(2) ** 32


def mp_laplace_t(w):
    """Standard Laplace inverse CDF at u(w)."""
    mpmath = _mp()
    u = mp_u(w)
    if u < mpmath.mpf(0.5):
        return mpmath.log(2 * u)
    return -mpmath.log(2 - 2 * u)


def mp_gauss_r(w):
    mpmath = _mp()
    return mpmath.sqrt(-2 * mpmath.log(mp_u(w)))


def mp_cos2pi(w):
    return _mp().cospi(2 * mp_u(w))


def mp_sin2pi(w):
    return _mp().sinpi(2 * mp_u(w))


MP_FUNCS = [mp_laplace_t, mp_gauss_r, mp_cos2pi, mp_sin2pi]


def edge_words():
    """Words at the ends of (0, 1), at u = 1/2 and at the octant ends of 2 pi u."""
    w = {0, 1, 2, 3, 2**32 - 1, 2**32 - 2, 2**31 - 1, 2**31, 2**31 + 1, 2**31 - 2}
    for k in range(1, 8):
        c = k * 2**29
        w.update({c - 2, c - 1, c, c + 1})
    return np.array(sorted(x for x in w if 0 <= x < 2**32), dtype=np.uint32)
