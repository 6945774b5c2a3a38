"""Pins for the oracle's Philox4x32-10 and the two random streams built on it.

The generator is pinned to the published known-answer vectors and to a second,
independent implementation (PyTorch's C++ Philox engine, compiled from its
shipped source header). The stream layouts are checked for the statistical
properties the method relies on: a uniform sign vector that depends only on the
high seed word, and uniform, independent 16-bit dithering noise.
"""

import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest

import oracle
from oracle.philox import philox4x32_10, philox4x32_10_scalar, sign_vector, noise16

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat():
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        lhs, rhs = line.split(":")
        ins = [int(v, 16) for v in lhs.split()]
        outs = [int(v, 16) for v in rhs.split()]
        yield ins[:4], ins[4:], outs


def test_known_answer_vectors_scalar_and_vectorised():
    cases = list(_kat())
    assert len(cases) == 3
    for ctr, key, expect in cases:
        assert list(philox4x32_10_scalar(ctr, key)) == expect
        got = philox4x32_10(*[np.array([c]) for c in ctr], key[0], key[1])
        assert [int(v[0]) for v in got] == expect


def test_vectorised_matches_scalar_on_random_inputs():
    rng = np.random.default_rng(1)
    ctr = rng.integers(0, 2 ** 32, size=(4, 64), dtype=np.uint64)
    key = rng.integers(0, 2 ** 32, size=(2, 64), dtype=np.uint64)
    vec = philox4x32_10(*ctr, *key)
    for i in range(64):
        s = philox4x32_10_scalar(ctr[:, i], key[:, i])
        assert tuple(int(v[i]) for v in vec) == s


def _torch_header():
    try:
        import torch
    except ImportError:
        return None
    inc = os.path.join(os.path.dirname(torch.__file__), "include")
    return inc if os.path.exists(os.path.join(inc, "ATen", "core", "PhiloxRNGEngine.h")) else None


TORCH_PROBE = r"""
#include <ATen/core/PhiloxRNGEngine.h>
#include <cstdio>
int main() {
  unsigned long long seed, sub, off;
  while (std::scanf("%llu %llu %llu", &seed, &sub, &off) == 3) {
    at::philox_engine e(seed, sub, off);
    unsigned a = e(), b = e(), c = e(), d = e();
    std::printf("%u %u %u %u\n", a, b, c, d);
  }
  return 0;
}
"""


@pytest.mark.skipif(shutil.which("g++") is None or _torch_header() is None,
                    reason="needs g++ and PyTorch's C++ headers")
def test_matches_pytorch_philox_engine():
    """PyTorch's engine keys Philox with the 64-bit seed and counts with
    (offset lo, offset hi, subsequence lo, subsequence hi): the same layout the
    noise stream uses (subsequence 0) and the sign stream uses (subsequence
    2^32, key (0, hi32(seed)))."""
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "p.cpp")
        exe = os.path.join(d, "p")
        open(src, "w").write(TORCH_PROBE)
        subprocess.run(["g++", "-O1", "-std=c++17", "-I" + _torch_header(), src, "-o", exe],
                       check=True, capture_output=True)
        rng = np.random.default_rng(7)
        seeds = [0, 1, 0xFFFFFFFFFFFFFFFF, 0x0123456789ABCDEF] + [int(v) for v in rng.integers(0, 2 ** 63, 8)]
        lines, expect = [], []
        for s in seeds:
            for sub in (0, 1 << 32):
                for off in (0, 1, 12345, (1 << 32) + 3):
                    lines.append(f"{s} {sub} {off}")
                    ctr = (off & 0xFFFFFFFF, off >> 32, sub & 0xFFFFFFFF, sub >> 32)
                    expect.append(philox4x32_10_scalar(ctr, (s & 0xFFFFFFFF, s >> 32)))
        out = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True,
                             check=True).stdout.split("\n")
        for got, exp in zip(out, expect):
            assert tuple(int(v) for v in got.split()) == exp


@pytest.mark.skipif(shutil.which("g++") is None or _torch_header() is None,
                    reason="needs g++ and PyTorch's C++ headers")
def test_noise_stream_equals_pytorch_engine_sequence():
    """Element 8q + 2i (+1) of a row-major stream is the low (high) half of the
    i-th output of the engine at offset q: checked through the engine itself."""
    seed = 0x00C0FFEE12345678
    rows, cols = 3, 64
    r16 = noise16(seed, rows, cols)
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "p.cpp")
        exe = os.path.join(d, "p")
        open(src, "w").write(TORCH_PROBE)
        subprocess.run(["g++", "-O1", "-std=c++17", "-I" + _torch_header(), src, "-o", exe],
                       check=True, capture_output=True)
        lines = [f"{seed} 0 {q}" for q in range(rows * cols // 8)]
        out = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True,
                             check=True).stdout.split()
    words = np.array([int(v) for v in out], dtype=np.uint64)
    halves = np.stack([words & np.uint64(0xFFFF), words >> np.uint64(16)], axis=1).reshape(-1)
    assert np.array_equal(halves.reshape(rows, cols), r16.astype(np.uint64))


@pytest.mark.skipif(shutil.which("g++") is None or _torch_header() is None,
                    reason="needs g++ and PyTorch's C++ headers")
def test_sign_vector_bits_from_pytorch_engine():
    """Every position of S, bit by bit, from the independent engine: S_j = -1
    iff bit j % 32 of output word (j / 32) % 4 of the engine at offset j / 128,
    subsequence 2^32, seeded with hi32(seed) << 32 (the layout the library's
    header documents). A swapped word, a shifted bit or a counter in the wrong
    slot fails here even though it would stay balanced."""
    seeds = [0xABCDEF0100000000, 0x00000001DEADBEEF, 0xFFFFFFFF00000000, 0x8000000000000007]
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "p.cpp")
        exe = os.path.join(d, "p")
        open(src, "w").write(TORCH_PROBE)
        subprocess.run(["g++", "-O1", "-std=c++17", "-I" + _torch_header(), src, "-o", exe],
                       check=True, capture_output=True)
        lines = [f"{(s >> 32) << 32} {1 << 32} {off}" for s in seeds for off in (0, 1)]
        out = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True,
                             check=True).stdout.split("\n")
    for i, s in enumerate(seeds):
        words = [int(v) for line in out[2 * i:2 * i + 2] for v in line.split()]   # 8 words: offsets 0, 1
        expect = np.array([-1.0 if (words[j // 32] >> (j % 32)) & 1 else 1.0 for j in range(256)])
        for g in (32, 64, 128, 256):
            assert np.array_equal(sign_vector(s, g), expect[:g]), (hex(s), g)


def test_sign_vector_depends_only_on_high_word_and_is_balanced():
    for g in (32, 64, 128, 256):
        s = sign_vector(0xABCDEF0100000000, g)
        assert s.shape == (g,) and set(np.unique(s)) <= {-1.0, 1.0}
        assert np.array_equal(s, sign_vector(0xABCDEF01FFFFFFFF, g))
        assert np.array_equal(s[:32], sign_vector(0xABCDEF0100000000, 32))  # prefix-consistent
    # Over many seeds each position is -1 about half the time.
    acc = np.zeros(256)
    n = 2000
    for hi in range(n):
        acc += sign_vector(hi << 32, 256) < 0
    frac = acc / n
    assert np.all(np.abs(frac - 0.5) < 5 * np.sqrt(0.25 / n))
    # Different high words give different vectors.
    assert not np.array_equal(sign_vector(1 << 32, 64), sign_vector(2 << 32, 64))


def test_noise_is_uniform_16_bit_and_independent_of_position():
    r = noise16(12345, 512, 512).astype(np.int64)
    assert r.min() >= 0 and r.max() < 65536
    n = r.size
    # Each of the 16 bits is a fair coin.
    for b in range(16):
        p = np.mean((r >> b) & 1)
        assert abs(p - 0.5) < 5 * np.sqrt(0.25 / n)
    # Histogram over 256 bins of the top byte is flat (chi-square, 255 dof).
    hist = np.bincount((r >> 8).ravel(), minlength=256)
    chi2 = np.sum((hist - n / 256) ** 2 / (n / 256))
    assert chi2 < 255 + 6 * np.sqrt(2 * 255)
    # Neighbouring elements (same generator call) are uncorrelated.
    u = (r - 32767.5) / 65536
    assert abs(np.mean(u[:, 0::2] * u[:, 1::2])) < 5 / np.sqrt(n / 2) / 12
    # Changing the low seed word changes the noise.
    assert np.mean(noise16(12345, 8, 64) == noise16(12346, 8, 64)) < 0.01


def test_noise_row_sampling_matches_full_matrix():
    full = noise16(99, 40, 96)
    ids = np.array([0, 7, 39, 13])
    assert np.array_equal(noise16(99, 4, 96, row_ids=ids), full[ids])


def test_public_exports():
    for name in oracle.__all__:
        assert hasattr(oracle, name)
