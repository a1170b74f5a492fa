"""Pins of the oracle's Philox4x32-10 and its uniform map against an
independent implementation (rocRAND's host-callable engine) and against
statistics."""

import os
import shutil
import subprocess

import numpy as np
import pytest
import scipy.stats

from oracle.philox import open_unit, philox4x32_10, token_words

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def rocrand_ref(tmp_path_factory):
    gxx = shutil.which("g++")
    inc = "/opt/rocm/include"
    if gxx is None or not os.path.exists(os.path.join(inc, "rocrand", "rocrand_philox4x32_10.h")):
        pytest.skip("g++ or rocRAND headers not available")
    exe = str(tmp_path_factory.mktemp("philox") / "ref")
    subprocess.check_call([gxx, "-O1", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I" + inc,
                           os.path.join(HERE, "philox_rocrand_ref.cpp"), "-o", exe])
    return exe


def test_matches_rocrand(rocrand_ref):
    rng = np.random.default_rng(0)
    n = 3000
    seeds = rng.integers(0, 2 ** 63, size=n, dtype=np.uint64) * np.uint64(2) + rng.integers(0, 2, size=n).astype(np.uint64)
    ctr = rng.integers(0, 2 ** 32, size=(n, 4), dtype=np.uint64)
    ctr[:50] = 0
    ctr[50:100] = 0xFFFFFFFF
    seeds[:10] = 0
    lines = "".join("%x %x %x %x %x\n" % (int(s), *map(int, c)) for s, c in zip(seeds, ctr))
    out = subprocess.run([rocrand_ref], input=lines, capture_output=True, text=True, check=True).stdout
    ref = np.array([[int(x, 16) for x in line.split()] for line in out.strip().split("\n")], dtype=np.uint64)
    k0 = (seeds & np.uint64(0xFFFFFFFF)).astype(np.uint32)
    k1 = (seeds >> np.uint64(32)).astype(np.uint32)
    got = philox4x32_10(ctr[:, 0].astype(np.uint32), ctr[:, 1].astype(np.uint32),
                        ctr[:, 2].astype(np.uint32), ctr[:, 3].astype(np.uint32), k0, k1)
    got = np.stack(got, axis=1).astype(np.uint64)
    assert np.array_equal(got, ref)


def test_uniform_map_is_open_and_exact():
    w = np.array([0, 1, 2 ** 31, 2 ** 32 - 1], dtype=np.uint32)
    u = open_unit(w)
    assert (u > 0).all() and (u < 1).all()
    assert u[0] == 2.0 ** -33 and u[-1] == 1 - 2.0 ** -33
    assert u[2] == 0.5 + 2.0 ** -33


def test_token_words_uniform_and_distinct():
    L = 200000
    u = open_unit(token_words(12345, 7, 1, 3, L))
    assert abs(u.mean() - 0.5) < 5 * (1 / np.sqrt(12 * L))
    assert scipy.stats.kstest(u, "uniform").pvalue > 1e-3
    a = token_words(1, 0, 0, 0, 4096)
    for other in (token_words(1, 0, 0, 1, 4096), token_words(1, 0, 1, 0, 4096),
                  token_words(1, 1, 0, 0, 4096), token_words(2, 0, 0, 0, 4096)):
        assert (a != other).mean() > 0.99


def test_token_words_layout():
    """Token j takes word j mod 4 of the block at counter (j // 4, h, b, layer)."""
    seed, layer, b, h = 0xDEADBEEF12345678, 5, 2, 9
    w = token_words(seed, layer, b, h, 11)
    for j in range(11):
        blk = philox4x32_10(j // 4, h, b, layer, seed & 0xFFFFFFFF, seed >> 32)
        assert w[j] == blk[j % 4]
