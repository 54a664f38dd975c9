"""Pins of the oracle's counter-based generator (oracle/philox.py).

* Published known-answer vectors of Philox4x32-10 (tests/golden).
* An independent implementation: rocRAND's header-only Philox engine,
  compiled for the host, on random counters and keys.
* The uniform map u24 hits its closed-form extremes and is uniform (chi^2).
* Counter fields are independent streams (no equal words across fields).
"""
import os
import shutil
import subprocess

import numpy as np
import pytest
from scipy import stats

from oracle import philox

HERE = os.path.dirname(os.path.abspath(__file__))


def _kat_rows():
    rows = []
    with open(os.path.join(HERE, "golden", "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            rows.append([int(w, 16) for w in line.split()])
    return rows


def test_known_answer_vectors():
    rows = _kat_rows()
    assert len(rows) == 3
    for r in rows:
        out = philox.philox4x32_10(tuple(r[0:4]), tuple(r[4:6]))
        assert [int(o) for o in out] == r[6:10]


@pytest.fixture(scope="module")
def rocrand_ref(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("philox") / "ref")
    r = subprocess.run([hipcc, "-O1", "--offload-arch=gfx950", os.path.join(HERE, "philox_rocrand_ref.cpp"),
                        "-o", exe], capture_output=True, text=True)
    if r.returncode != 0:
        pytest.skip("could not build the rocRAND reference: " + r.stderr[-400:])
    return exe


def test_matches_independent_implementation(rocrand_ref):
    rng = np.random.default_rng(11)
    n = 4000
    words = rng.integers(0, 2 ** 32, size=(n, 6), dtype=np.uint64)
    words[:50, 0] = np.arange(50)  # small counters too
    inp = "\n".join(" ".join(str(int(x)) for x in row) for row in words) + "\n"
    r = subprocess.run([rocrand_ref], input=inp, capture_output=True, text=True, check=True)
    ref = np.array([[int(x) for x in line.split()] for line in r.stdout.strip().splitlines()], dtype=np.uint64)
    out = philox.philox4x32_10(tuple(words[:, i] for i in range(4)), (words[:, 4], words[:, 5]))
    got = np.stack(out, axis=1)
    assert np.array_equal(got, ref)


def test_draw_words_layout():
    # word (draw & 3) of the block (draw >> 2); node | stream << 16 in word 1
    seed = 0x0123456789ABCDEF
    draws = np.arange(16, dtype=np.uint64)
    w = philox.draw_words(seed, 7, 3, 5, philox.STREAM_BONUS, draws)
    for d in range(16):
        blk = philox.philox4x32_10((d >> 2, 5 | (2 << 16), 3, 7), (seed & 0xFFFFFFFF, seed >> 32))
        assert int(w[d]) == int(blk[d & 3])


def test_u24_closed_form_extremes():
    assert philox.u24(0) == 2.0 ** -24
    assert philox.u24(0xFFFFFFFF) == 1.0 - 2.0 ** -24
    assert philox.u24(1 << 31) == 0.5 + 2.0 ** -24
    # exactly representable in binary32
    w = np.random.default_rng(0).integers(0, 2 ** 32, 1000, dtype=np.uint64)
    u = philox.u24(w)
    assert np.array_equal(u.astype(np.float32).astype(np.float64), u)
    assert philox.G_MAX == pytest.approx(-np.log(-np.log1p(-2.0 ** -24)), rel=1e-15)
    assert philox.G_MIN == pytest.approx(-np.log(24 * np.log(2.0)), rel=1e-15)


def test_uniformity_chi2():
    u = philox.uniforms(42, 0, 0, 0, philox.STREAM_REPLAY, np.arange(200000, dtype=np.uint64))
    counts, _ = np.histogram(u, bins=64, range=(0, 1))
    assert stats.chisquare(counts).pvalue > 1e-4
    # Gumbel noise has mean Euler-Mascheroni and variance pi^2/6
    g = philox.gumbel(u)
    assert abs(g.mean() - np.euler_gamma) < 5 * np.sqrt(np.pi ** 2 / 6 / g.size)
    assert abs(g.var() - np.pi ** 2 / 6) < 0.05


def test_counter_fields_are_distinct_streams():
    base = philox.draw_words(9, 1, 1, 1, 0, np.arange(4096, dtype=np.uint64))
    for args in [(9, 2, 1, 1, 0), (9, 1, 2, 1, 0), (9, 1, 1, 2, 0), (9, 1, 1, 1, 1), (10, 1, 1, 1, 0)]:
        other = philox.draw_words(*args, np.arange(4096, dtype=np.uint64))
        assert (base == other).mean() < 0.01
        # no linear correlation of the uniforms
        assert abs(np.corrcoef(philox.u24(base), philox.u24(other))[0, 1]) < 0.06
