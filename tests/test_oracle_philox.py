"""Pins for the oracle's counter-based dropout generator (oracle/philox.py).

* Every output word agrees with rocRAND's philox4x32_10 engine, an
  independent implementation of the same published generator (Salmon et al.,
  SC'11), on random and edge-case counters and keys.
* Keep rates match 1 - p within 6 sigma; p = 0 is the identity.
"""
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest

from oracle import philox

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def rocrand_ref():
    gxx = shutil.which("g++")
    inc = "/opt/rocm/include"
    if gxx is None or not os.path.exists(os.path.join(inc, "rocrand", "rocrand_philox4x32_10.h")):
        pytest.skip("g++ or rocRAND headers not available")
    d = tempfile.mkdtemp()
    exe = os.path.join(d, "philox_ref")
    subprocess.check_call([gxx, "-O1", "-std=c++17", f"-I{inc}", "-D__HIP_PLATFORM_AMD__",
                           os.path.join(HERE, "rocrand_philox_ref.cpp"), "-o", exe])

    def run(rows):
        txt = "\n".join(" ".join(str(int(v)) for v in r) for r in rows) + "\n"
        out = subprocess.run([exe], input=txt, capture_output=True, text=True, check=True).stdout
        return np.array([[int(t) for t in ln.split()] for ln in out.strip().splitlines()],
                        dtype=np.uint64)
    yield run
    shutil.rmtree(d, ignore_errors=True)


def test_matches_rocrand(rocrand_ref):
    rng = np.random.default_rng(7)
    n = 3000
    rows = rng.integers(0, 2**32, size=(n, 6), dtype=np.uint64)
    rows[:, 1] &= np.uint64(0x3FFFFFFF)            # rocRAND offset = 4*block must fit 64 bits
    edge = np.array([[0, 0, 0, 0, 0, 0],
                     [0xFFFFFFFF, 0x3FFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF],
                     [1, 0, 0, 0, 0, 0], [0, 0, 1, 0, 0, 0], [0, 0, 0, 0, 1, 0],
                     [0, 0, 0, 0, 0, 1], [12345, 0, 2, 7, 0, 0]], dtype=np.uint64)
    rows = np.concatenate([edge, rows])
    ref = rocrand_ref(rows)
    got = philox.philox4x32_10(rows[:, 0], rows[:, 1], rows[:, 2], rows[:, 3], 0, 0)
    # key varies per row: evaluate row by row groups with identical keys
    out = np.zeros((len(rows), 4), dtype=np.uint64)
    for idx in range(len(rows)):
        w = philox.philox4x32_10(rows[idx, 0], rows[idx, 1], rows[idx, 2], rows[idx, 3],
                                 int(rows[idx, 4]), int(rows[idx, 5]))
        out[idx] = [int(v) for v in w]
    assert got[0].shape == (len(rows),)
    np.testing.assert_array_equal(out, ref)


def test_random_words_follow_counter_definition(rocrand_ref):
    # element e -> counter (lo(e>>2), hi(e>>2), site, layer), word e & 3
    seed = 0x1234_5678_9ABC_DEF0
    e = np.array([0, 1, 2, 3, 4, 5, 6, 7, 1 << 33 | 5, 33554431, 123456789], dtype=np.uint64)
    site, layer = 2, 17
    rows = [[int(x >> 2) & 0xFFFFFFFF, int(x >> 2) >> 32, site, layer,
             seed & 0xFFFFFFFF, seed >> 32] for x in e]
    ref = rocrand_ref(rows)
    want = np.array([ref[i, int(x) & 3] for i, x in enumerate(e)], dtype=np.uint64)
    got = philox.random_words(seed, site, layer, e).astype(np.uint64)
    np.testing.assert_array_equal(got, want)


def test_threshold():
    assert philox.keep_threshold(0.1) == 3865470566
    assert philox.keep_threshold(0.0) == 2**32
    assert philox.keep_threshold(0.5) == 2**31
    with pytest.raises(ValueError):
        philox.keep_threshold(1.0)


@pytest.mark.parametrize("p", [0.1, 0.3, 0.5])
def test_keep_rate(p):
    n = 1 << 20
    m = philox.keep_mask(0, philox.SITE_ATTN, 0, p, n)
    sigma = np.sqrt(p * (1 - p) / n)
    assert abs(m.mean() - (1 - p)) < 6 * sigma


def test_identity_at_p0():
    f = philox.dropout_factor(3, 1, 0, 0.0, (4, 5))
    assert np.all(f == 1.0)


def test_sites_and_layers_decorrelated():
    n = 1 << 16
    a = philox.keep_mask(0, 0, 0, 0.5, n)
    b = philox.keep_mask(0, 1, 0, 0.5, n)
    c = philox.keep_mask(0, 0, 1, 0.5, n)
    d = philox.keep_mask(1, 0, 0, 0.5, n)
    for other in (b, c, d):
        agree = (a == other).mean()
        assert abs(agree - 0.5) < 6 * 0.5 / np.sqrt(n)


def test_offset_consistency():
    full = philox.keep_mask(5, 2, 3, 0.2, 1000)
    part = philox.keep_mask(5, 2, 3, 0.2, 300, offset=401)
    np.testing.assert_array_equal(full[401:701], part)
