"""Pins of the oracle's Philox4x32-10 and dither stream (CPU).

* against rocRAND's philox4x32_10 engine (an independent, published
  implementation compiled here from its open-source header) on random and
  extreme counters/keys;
* counter uniqueness over (layer, kv head, slot, channel group);
* byte uniformity (chi-square) and the dither lattice.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import philox

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def rocrand_dump(tmp_path_factory):
    gxx = shutil.which("g++")
    hdr = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"
    if gxx is None or not os.path.exists(hdr):
        pytest.skip("g++ or rocRAND headers not available")
    exe = str(tmp_path_factory.mktemp("rr") / "rocrand_dump")
    subprocess.run([gxx, "-O1", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    os.path.join(HERE, "philox_ref", "rocrand_dump.cpp"), "-o", exe],
                   check=True, capture_output=True)

    def run(keys, ctrs):
        lines = "".join("%x %x %x %x %x %x\n" % (k[0], k[1], *c) for k, c in zip(keys, ctrs))
        res = subprocess.run([exe], input=lines, capture_output=True, text=True, check=True)
        return np.array([[int(w, 16) for w in ln.split()] for ln in res.stdout.splitlines()],
                        dtype=np.uint64)
    return run


def test_philox_matches_rocrand(rocrand_dump):
    rng = np.random.default_rng(7)
    n = 400
    keys = rng.integers(0, 2**32, size=(n, 2), dtype=np.uint64)
    ctrs = rng.integers(0, 2**32, size=(n, 4), dtype=np.uint64)
    # extremes: all-zero, all-ones, single bits, and each word alone
    ext_c = [[0, 0, 0, 0], [0xFFFFFFFF] * 4, [1, 0, 0, 0], [0, 1, 0, 0], [0, 0, 1, 0],
             [0, 0, 0, 1], [0x80000000, 0, 0, 0x80000000]]
    ext_k = [[0, 0], [0xFFFFFFFF, 0xFFFFFFFF], [1, 0], [0, 1], [0x9E3779B9, 0xBB67AE85],
             [0, 0], [0xFFFFFFFF, 0]]
    keys = np.concatenate([keys, np.array(ext_k, dtype=np.uint64)])
    ctrs = np.concatenate([ctrs, np.array(ext_c, dtype=np.uint64)])
    ref = rocrand_dump(keys.tolist(), ctrs.tolist())
    got = np.stack([philox.philox4x32_10(c, (int(k[0]), int(k[1]))) for k, c in zip(keys, ctrs)])
    assert np.array_equal(got.astype(np.uint64), ref)


def test_dither_counters_are_unique():
    seen = set()
    for layer in (0, 1, 27):
        for kv in range(4):
            ctr = philox.dither_counter(np.arange(300)[:, None], np.arange(8)[None, :], layer, kv)
            for row in ctr.reshape(-1, 4):
                seen.add(tuple(int(x) for x in row))
    assert len(seen) == 3 * 4 * 300 * 8
    # high slot words land in word 2
    c = philox.dither_counter(np.int64(5 << 32 | 9), 3, 2, 1)
    assert [int(x) for x in c] == [3, 9, 5, (2 << 16) | 1]


def test_dither_bytes_uniform_and_lattice():
    by = philox.dither_bytes(np.arange(20000), 128, 3, 1, 0x5EED000000000003).ravel()
    counts = np.bincount(by, minlength=256)
    expected = by.size / 256
    chi2 = float(np.sum((counts - expected) ** 2 / expected))
    # 255 dof: mean 255, sd ~22.6; 400 is > 6 sigma
    assert chi2 < 400, chi2
    xi = philox.dither_values(np.arange(64), 128, 0, 0, 1)
    assert np.all(np.abs(xi) < 0.5)
    assert np.all(np.abs(xi * 512 - np.rint(xi * 512)) == 0)          # odd multiples of 1/512
    assert np.all(np.rint(xi * 512).astype(np.int64) % 2 != 0)
    assert abs(float(np.mean(xi))) < 5e-3


def test_keys_and_values_share_the_counter_but_layers_do_not():
    a = philox.dither_bytes([7, 8], 128, 4, 2, 11)
    assert np.array_equal(a, philox.dither_bytes([7, 8], 128, 4, 2, 11))
    assert not np.array_equal(a, philox.dither_bytes([7, 8], 128, 5, 2, 11))
    assert not np.array_equal(a, philox.dither_bytes([7, 8], 128, 4, 3, 11))
    assert not np.array_equal(a, philox.dither_bytes([7, 8], 128, 4, 2, 12))
