"""Pins for the oracle's random streams (Philox4x32-10, index map, Box-Muller, init).

The Philox block is checked against an independent implementation: PyTorch's
header-only `at::Philox4_32` engine, compiled here with g++. Its counter layout is
(offset lo, offset hi, subsequence lo, subsequence hi) with key = seed, so block
(c0, c1, c2, c3; k) is engine(seed=k, subsequence=c2|c3<<32, offset=c0|c1<<32).
"""
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest
from scipy import stats

from oracle import philox

TORCH_INC = None
try:
    import torch  # noqa: F401  (only to locate its headers)
    TORCH_INC = os.path.join(os.path.dirname(torch.__file__), "include")
except Exception:  # pragma: no cover
    pass

_PROBE = r"""
#include <ATen/core/PhiloxRNGEngine.h>
#include <cstdio>
int main() {
  unsigned long long seed, sub, off;
  while (scanf("%llu %llu %llu", &seed, &sub, &off) == 3) {
    at::Philox4_32 e(seed, sub, off);
    unsigned a = e(), b = e(), c = e(), d = e();
    printf("%u %u %u %u\n", a, b, c, d);
  }
}
"""


@pytest.fixture(scope="module")
def torch_philox():
    hdr = os.path.join(TORCH_INC or "", "ATen", "core", "PhiloxRNGEngine.h")
    if not (TORCH_INC and os.path.exists(hdr) and shutil.which("g++")):
        pytest.skip("independent Philox header or g++ not available")
    d = tempfile.mkdtemp()
    src, exe = os.path.join(d, "p.cpp"), os.path.join(d, "p")
    open(src, "w").write(_PROBE)
    subprocess.check_call(["g++", "-std=c++17", "-O1", "-I" + TORCH_INC, src, "-o", exe])

    def run(triples):
        inp = "".join("%d %d %d\n" % t for t in triples)
        out = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True).stdout
        return np.array([[int(x) for x in l.split()] for l in out.strip().splitlines()], dtype=np.uint64)
    return run


def test_block_matches_independent_implementation(torch_philox):
    rng = np.random.default_rng(123)
    cases = [(0, 0, 0, 0, 0, 0), (2**32 - 1,) * 6, (7, 3, 1, 0, 1, 0)]
    cases += [tuple(int(x) for x in rng.integers(0, 2**32, 6)) for _ in range(200)]
    triples = [((k1 << 32) | k0, (c3 << 32) | c2, (c1 << 32) | c0) for c0, c1, c2, c3, k0, k1 in cases]
    ref = torch_philox(triples)
    for (c0, c1, c2, c3, k0, k1), r in zip(cases, ref):
        got = np.array([int(x) for x in philox.block(c0, c1, c2, c3, k0, k1)], dtype=np.uint64)
        assert np.array_equal(got, r), (c0, c1, c2, c3, k0, k1)


def test_stream_counter_layout(torch_philox):
    """words(seed, n, step, purpose, tid)[i] is word i&3 of block (i>>2, step, purpose, tid)."""
    seed, step, purpose, tid = 0x1234_5678_9ABC, 77, philox.PURPOSE_IDX, 5
    w = philox.words(seed, 40, step, purpose, tid)
    ref = torch_philox([(seed, (tid << 32) | purpose, (step << 32) | blk) for blk in range(10)])
    assert np.array_equal(w, ref.reshape(-1))


def test_index_closed_forms():
    w = philox.words(9, 4096, 3, philox.PURPOSE_IDX)
    assert np.all(philox.indices(9, 3, 4096, 1) == 0)
    for k in (1, 5, 20, 31):
        assert np.array_equal(philox.indices(9, 3, 4096, 2 ** k), (w >> np.uint64(32 - k)).astype(np.int64))
    idx = philox.indices(9, 3, 4096, 1000)
    assert idx.min() >= 0 and idx.max() < 1000


def test_index_uniformity_chi2():
    size, n = 1000, 1_000_000
    idx = philox.indices(1, 1, n, size)
    counts = np.bincount(idx, minlength=size)
    chi2, p = stats.chisquare(counts)
    assert p > 1e-4, (chi2, p)
    # different steps give different draws
    assert not np.array_equal(idx[:100], philox.indices(1, 2, 100, size))


def test_box_muller_special_values():
    # words crafted so that u1 = 1 (radius 0) or u2 = 0 (angle 0) inside one block
    assert philox.normals(0, 1, 2, 4).shape == (4,)
    # Reach the transform directly through a stream whose words we know: use the
    # identity R cos, R sin with (u1, u2) recovered from the words.
    w = philox.words(5, 8, 2, philox.PURPOSE_NOISE_POL)
    n = philox.normals(5, 2, philox.PURPOSE_NOISE_POL, 8)
    for blk in range(2):
        for pair in range(2):
            wa, wb = int(w[4 * blk + 2 * pair]), int(w[4 * blk + 2 * pair + 1])
            u1 = ((wa >> 8) + 1) / 2.0 ** 24
            u2 = (wb >> 8) / 2.0 ** 24
            r = n[4 * blk + 2 * pair: 4 * blk + 2 * pair + 2]
            # radius^2 = -2 ln u1 and angle = 2 pi u2 (textbook Box-Muller)
            assert np.isclose(r[0] ** 2 + r[1] ** 2, -2.0 * np.log(u1), rtol=1e-12, atol=1e-12)
            if abs(r[0]) + abs(r[1]) > 1e-6:
                ang = np.arctan2(r[1], r[0]) % (2 * np.pi)
                assert np.isclose(ang, (2 * np.pi * u2) % (2 * np.pi), atol=1e-9) or \
                    np.isclose(abs(ang - 2 * np.pi * u2), 2 * np.pi, atol=1e-9)


def test_normal_moments_and_ks():
    n = philox.normals(3, 11, philox.PURPOSE_NOISE_TGT, 1_000_000)
    assert abs(n.mean()) < 5e-3 and abs(n.var() - 1.0) < 5e-3
    assert stats.kstest(n, "norm").pvalue > 1e-4
    # odd lengths are prefixes of longer draws
    assert np.array_equal(philox.normals(3, 11, 2, 7), n[:7])


def test_init_uniform_range_and_variance():
    fan_in = 376
    k = np.float32(1.0 / np.sqrt(fan_in))
    v = philox.init_uniform(1, 16, 200_000, fan_in)
    assert v.dtype == np.float32
    assert np.all(np.abs(v) <= k)
    assert abs(v.var() / (float(k) ** 2 / 3.0) - 1.0) < 0.02
    assert abs(v.mean()) < 3e-3 * float(k)
    # distinct tensors draw distinct streams
    assert not np.array_equal(v[:64], philox.init_uniform(1, 17, 64, fan_in))
