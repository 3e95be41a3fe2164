"""Pin the oracle's Philox4x32-10 stream against rocRAND's engine.

rocRAND's philox4x32_10_engine(seed, subsequence, offset) uses key = seed,
counter = (offset / 4 as 64 bits, subsequence as 64 bits) and returns word
offset % 4 first, which is exactly the oracle's SR word layout with
subsequence = tensor id (see oracle.philox)."""

import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import philox

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def rocrand_ref(tmp_path_factory):
    cxx = shutil.which("g++")
    inc = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"
    if cxx is None or not os.path.exists(inc):
        pytest.skip("g++ or the rocRAND header is not available")
    exe = str(tmp_path_factory.mktemp("philox") / "ref")
    subprocess.check_call([cxx, "-O1", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                           os.path.join(HERE, "philox_rocrand_ref.cpp"), "-o", exe])

    def run(seed, sub, off, n):
        out = subprocess.check_output([exe, str(seed), str(sub), str(off), str(n)])
        return np.array([int(t) for t in out.split()], dtype=np.uint64)
    return run


@pytest.mark.parametrize("seed,tid,off", [(0, 0, 0), (1, 2, 0), (1, 1, 7),
                                          (0xDEADBEEFCAFEF00D, 0xFFFFFFFF, 12345),
                                          (42, 3, (1 << 34) + 3)])
def test_sr_words_match_rocrand(rocrand_ref, seed, tid, off):
    n = 37
    ref = rocrand_ref(seed, tid, off, n)
    mine = philox.sr_words(seed, tid, np.arange(off, off + n, dtype=np.int64))
    assert np.array_equal(ref, mine.astype(np.uint64))


def test_block_function_zero_key(rocrand_ref):
    # Counter (0,0,0,0), key (0,0): the first four engine outputs.
    mine = philox.philox4x32_10(np.zeros((1, 4), np.uint32), (0, 0))[0]
    assert np.array_equal(rocrand_ref(0, 0, 0, 4), mine.astype(np.uint64))


def test_words_look_uniform():
    w = philox.sr_words(7, 1, np.arange(1 << 18)).astype(np.float64)
    mean = w.mean() / 2.0 ** 32
    assert abs(mean - 0.5) < 5 * (1 / np.sqrt(12)) / np.sqrt(w.size)
