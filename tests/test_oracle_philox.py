"""Pins of the oracle's random words.

* Philox4x32-10 against the known-answer vectors published with Random123
  (tests/golden/philox4x32_10_kat.txt).
* The counter layout (key = seed, counter = (g_lo, g_hi, tensor_id,
  4*step + stream), element e -> word e & 3 of group e >> 2) against an
  independent Philox: PyTorch's header-only engine, compiled here from source.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def _kat_rows():
    rows = []
    with open(os.path.join(HERE, "golden", "philox4x32_10_kat.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            rows.append([int(x, 16) for x in line.split()])
    return rows


@pytest.mark.parametrize("row", _kat_rows())
def test_philox_known_answers(row):
    c, k, want = row[0:4], row[4:6], row[6:10]
    got = oracle.philox4x32([c[0]], [c[1]], [c[2]], [c[3]], k[0], k[1], rounds=10)
    assert [int(x[0]) for x in got] == want


def test_philox_vectorised_matches_scalar():
    rng = np.random.default_rng(1)
    c = rng.integers(0, 2 ** 32, size=(4, 257), dtype=np.uint64)
    k0, k1 = 0x12345678, 0x9ABCDEF0
    vec = oracle.philox4x32(c[0], c[1], c[2], c[3], k0, k1)
    for j in (0, 1, 100, 256):
        one = oracle.philox4x32([c[0, j]], [c[1, j]], [c[2, j]], [c[3, j]], k0, k1)
        assert [int(x[0]) for x in one] == [int(v[j]) for v in vec]


@pytest.fixture(scope="module")
def torch_philox(tmp_path_factory):
    gxx = shutil.which("g++")
    try:
        import torch
        inc = os.path.join(os.path.dirname(torch.__file__), "include")
    except Exception:  # pragma: no cover
        inc = None
    if gxx is None or inc is None or not os.path.exists(os.path.join(inc, "ATen", "core", "PhiloxRNGEngine.h")):
        pytest.skip("g++ or PyTorch's PhiloxRNGEngine.h not available")
    out = tmp_path_factory.mktemp("philox") / "philox_torch_ref"
    subprocess.run([gxx, "-std=c++17", "-O1", "-I", inc, os.path.join(HERE, "philox_torch_ref.cpp"),
                    "-o", str(out)], check=True, capture_output=True)

    def run(triples):
        text = "".join(f"{s} {sub} {off}\n" for s, sub, off in triples)
        res = subprocess.run([str(out)], input=text, capture_output=True, text=True, check=True)
        return [[int(x, 16) for x in line.split()] for line in res.stdout.strip().splitlines()]

    return run


def test_group_words_match_torch_engine(torch_philox):
    rng = np.random.default_rng(2)
    cases = []
    for _ in range(64):
        seed = int(rng.integers(0, 2 ** 63)) * 2 + int(rng.integers(0, 2))
        step = int(rng.integers(0, 2 ** 30))
        tid = int(rng.integers(0, 2 ** 32))
        g = int(rng.integers(0, 2 ** 62))
        stream = int(rng.integers(0, 4))
        cases.append((seed, step, tid, g, stream))
    cases.append((0, 0, 0, 0, 0))
    cases.append((2 ** 64 - 1, 2 ** 30 - 1, 2 ** 32 - 1, 2 ** 64 - 1, 3))
    triples = [(seed, tid | (((step << 2) | stream) << 32), g) for seed, step, tid, g, stream in cases]
    want = torch_philox(triples)
    for (seed, step, tid, g, stream), w in zip(cases, want):
        got = oracle.group_words(seed, step, tid, [g], stream)
        assert [int(x[0]) for x in got] == w


def test_element_words_lane_layout(torch_philox):
    seed, step, tid = 0x5EED0003, 17, 41
    off, n = 4 * 1000 + 3, 37  # starts in the middle of a group
    got = oracle.element_words(seed, step, tid, off, n, oracle.STREAM_MASK)
    e = np.arange(off, off + n)
    groups = sorted(set((e >> 2).tolist()))
    ref = dict(zip(groups, torch_philox([(seed, tid | ((step << 2) << 32), g) for g in groups])))
    for i, ei in enumerate(e):
        assert int(got[i]) == ref[ei >> 2][ei & 3]


def test_streams_steps_tensors_differ():
    base = oracle.element_words(7, 3, 5, 0, 4096, 0)
    for other in (oracle.element_words(7, 3, 5, 0, 4096, 1),
                  oracle.element_words(7, 4, 5, 0, 4096, 0),
                  oracle.element_words(7, 3, 6, 0, 4096, 0),
                  oracle.element_words(8, 3, 5, 0, 4096, 0)):
        assert np.mean(base == other) < 0.01


def test_key_range_errors():
    with pytest.raises(ValueError):
        oracle.element_words(0, 2 ** 30, 0, 0, 4, 0)
    with pytest.raises(ValueError):
        oracle.element_words(-1, 0, 0, 0, 4, 0)
    with pytest.raises(ValueError):
        oracle.element_words(0, 0, 2 ** 32, 0, 4, 0)
