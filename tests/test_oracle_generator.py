"""Pins for the oracle's counter-based normal generator (CPU only).

The generator is Philox4x32-10 (Salmon et al., SC 2011) feeding Box-Muller
(Box & Muller, 1958) with series-based ln/sin/cos.  It is pinned against
things other than itself:
  * Philox: rocRAND's independent Philox4x32-10 engine (a library routine,
    compiled here from its public header) on random counters and keys;
  * ln / sin / cos (fp32 series): the platform libm, within a few fp32 ulp,
    and the exact quarter-turn rotation of the sin / cos pair;
  * the normals: moments and a Kolmogorov-Smirnov test against N(0,1).
"""
import math
import os
import shutil
import subprocess

import numpy as np
import pytest
from scipy import stats

ROCRAND_HDR = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"

_PROBE = r"""
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
struct Expose : rocrand_device::philox4x32_10_engine {
  uint4 run(uint4 c, uint2 k) { return this->ten_rounds(c, k); }
};
int main() {
  Expose e; unsigned a[6];
  while (scanf("%x %x %x %x %x %x", &a[0], &a[1], &a[2], &a[3], &a[4], &a[5]) == 6) {
    uint4 r = e.run(make_uint4(a[0], a[1], a[2], a[3]), make_uint2(a[4], a[5]));
    printf("%08x %08x %08x %08x\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
"""


@pytest.fixture(scope="module")
def rocrand_probe(tmp_path_factory):
    if not os.path.exists(ROCRAND_HDR) or shutil.which("g++") is None:
        pytest.skip("rocRAND header or g++ not available")
    d = tmp_path_factory.mktemp("philox")
    src = d / "probe.cpp"
    src.write_text(_PROBE)
    exe = d / "probe"
    subprocess.run(["g++", "-std=c++17", "-O1", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    str(src), "-o", str(exe)], check=True, capture_output=True)
    return str(exe)


def test_philox_matches_rocrand(oracle_lib, rocrand_probe):
    rng = np.random.default_rng(123)
    rows = rng.integers(0, 2**32, size=(300, 6), dtype=np.uint64).astype(np.uint32)
    rows[0] = 0
    rows[1] = 0xFFFFFFFF
    inp = "\n".join(" ".join("%x" % v for v in r) for r in rows) + "\n"
    out = subprocess.run([rocrand_probe], input=inp, capture_output=True, text=True, check=True).stdout
    ref = np.array([[int(x, 16) for x in line.split()] for line in out.strip().splitlines()],
                   dtype=np.uint32)
    got = np.stack([oracle_lib.philox4x32_10(r[:4], r[4:]) for r in rows])
    assert np.array_equal(got, ref)


def test_uniform_exact_open_interval(oracle_lib):
    assert oracle_lib.uniform(0) == 2.0 ** -24
    assert oracle_lib.uniform(0xFFFFFFFF) == 1.0 - 2.0 ** -24
    for x in [1, 511, 512, 0x80000000, 0x12345678]:
        assert oracle_lib.uniform(x) == (2 * (x >> 9) + 1) * 2.0 ** -24


def _ulp32(x):
    """Spacing of fp32 values at |x|."""
    return float(np.spacing(np.float32(abs(x))))


def test_ln_series_accuracy(oracle_lib):
    # fp32 series ln against libm's double log, in fp32 ulps of the result
    rng = np.random.default_rng(7)
    xs = (2 * (rng.integers(0, 2**32, 4000, dtype=np.uint64) >> 9) + 1) * 2.0 ** -24
    xs = np.concatenate([xs, [2.0 ** -24, 0.5, 0.70710677, 0.70710683, 1 - 2.0 ** -24]])
    worst = 0.0
    for u in xs:
        u32 = float(np.float32(u))
        got, ref = oracle_lib.ln(u32), math.log(u32)
        worst = max(worst, abs(got - ref) / _ulp32(ref))
    assert worst <= 4.0, worst
    # the split point m in [r, 2r): both sides of it agree with libm
    for u in [0.70710677, 0.70710683, 0.35355338, 0.35355341]:
        u32 = float(np.float32(u))
        assert abs(oracle_lib.ln(u32) - math.log(u32)) <= 3 * _ulp32(math.log(u32))


def _word_of(n):
    """A word whose uniform is n * 2^-24 (n odd)."""
    return ((n - 1) // 2) << 9


def test_sincos_series_accuracy(oracle_lib):
    rng = np.random.default_rng(8)
    words = rng.integers(0, 2**32, 4000, dtype=np.uint64)
    worst = 0.0
    for x in words:
        u = (2 * (int(x) >> 9) + 1) * 2.0 ** -24
        s, c = oracle_lib.sincos_2pi(int(x))
        worst = max(worst, abs(s - math.sin(2 * math.pi * u)), abs(c - math.cos(2 * math.pi * u)))
    # fp32: the rounding of 2 pi and of phi, plus a few roundings in the series
    assert worst < 2e-7, worst
    # a quarter turn later (n + 2^22) the pair rotates exactly:
    # sin(a + pi/2) = cos a, cos(a + pi/2) = -sin a, bit for bit
    for n in [1, 12345, 2**21 - 1, 2**21 + 1, 3 * 2**21 + 7, 2**24 - 2**22 - 1]:
        s0, c0 = oracle_lib.sincos_2pi(_word_of(n))
        s1, c1 = oracle_lib.sincos_2pi(_word_of(n + 2**22))
        assert (s1, c1) == (c0, -s0), n
    # the smallest angle: sin 2 pi u = 2 pi u to fp32 precision, cos = 1
    s, c = oracle_lib.sincos_2pi(0)
    assert c == 1.0 and abs(s - 2 * math.pi * 2.0 ** -24) <= _ulp32(s)


def test_normals_distribution(oracle_lib):
    z = np.concatenate([oracle_lib.normal4(0x1234, 0, 3, h, i, jq)
                        for h in range(2) for i in range(200) for jq in range(16)])
    assert z.size == 2 * 200 * 16 * 4
    assert abs(z.mean()) < 4.0 / math.sqrt(z.size)
    assert abs(z.var() - 1.0) < 0.05
    assert stats.kstest(z, "norm").pvalue > 1e-3
    # Box-Muller pairs: (z0, z1) = r (cos, sin) with the same radius
    q = oracle_lib.normal4(9, 1, 2, 3, 4, 5)
    ua = oracle_lib.uniform(oracle_lib.philox4x32_10([5, 4, 3, (1 << 16) | 2], [9, 0])[0])
    r = math.sqrt(-2.0 * math.log(ua))
    assert math.isclose(math.hypot(q[0], q[1]), r, rel_tol=2e-6)


def test_normals_counter_fields_independent(oracle_lib):
    base = oracle_lib.normal4(5, 0, 0, 0, 0, 0)
    for args in [(5, 1, 0, 0, 0, 0), (5, 0, 1, 0, 0, 0), (5, 0, 0, 1, 0, 0), (5, 0, 0, 0, 1, 0),
                 (5, 0, 0, 0, 0, 1), (6, 0, 0, 0, 0, 0), (5 + (1 << 32), 0, 0, 0, 0, 0)]:
        assert not np.array_equal(oracle_lib.normal4(*args), base), args
