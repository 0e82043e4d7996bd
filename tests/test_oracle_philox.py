"""Pins the oracle's Philox4x32-10 against PyTorch ATen's independent
implementation (built from its open-source header with g++), bit for bit."""
import os
import shutil
import subprocess
import sysconfig

import numpy as np
import pytest

from oracle import event_words, philox4x32_10, uniform_from_words

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def aten_philox(tmp_path_factory):
    import torch
    inc = os.path.join(os.path.dirname(torch.__file__), "include")
    if shutil.which("g++") is None or not os.path.exists(os.path.join(inc, "ATen/core/PhiloxRNGEngine.h")):
        pytest.skip("g++ or ATen header unavailable")
    exe = str(tmp_path_factory.mktemp("aten") / "aten_philox")
    subprocess.check_call(["g++", "-O1", "-std=c++17", "-I", inc, os.path.join(HERE, "aten_philox_ref.cpp"), "-o", exe])

    def run(triples):
        inp = "".join(f"{s} {st} {o}\n" for s, st, o in triples)
        out = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True).stdout
        return np.array([[int(v) for v in line.split()] for line in out.strip().splitlines()], dtype=np.uint64).astype(np.uint32)
    return run


def test_event_words_match_aten(aten_philox):
    rng = np.random.default_rng(123)
    triples = [(0, 0, 0), (1, 0, 0), (0, 0, 1), (2**64 - 1, 0, 2**64 - 1), (0xDEADBEEFCAFEF00D, 3, 2**32 - 1),
               (5, 1, 2**32), (7, 2, 2**40 + 12345)]
    for _ in range(200):
        triples.append((int(rng.integers(0, 2**63)) * 2 + int(rng.integers(0, 2)),
                        int(rng.integers(0, 4)), int(rng.integers(0, 2**62))))
    ref = aten_philox(triples)
    for (seed, stream, off), r in zip(triples, ref):
        got = event_words(seed, np.array([off], dtype=np.uint64), stream)[0]
        assert np.array_equal(got, r), (seed, stream, off, got, r)


def test_counter_layout_matches_aten_for_consecutive_ids(aten_philox):
    ids = np.arange(1000, dtype=np.uint64) + np.uint64(2**32 - 500)   # crosses the lo/hi carry
    ref = aten_philox([(42, 0, int(i)) for i in ids])
    assert np.array_equal(event_words(42, ids, 0), ref)


def test_raw_block_function_vs_aten_fields(aten_philox):
    # counter (c0,c1,c2,c3) = (offset lo, offset hi, stream lo, stream hi) in ATen
    off, stream, seed = 0x0123456789ABCDEF, 0x00000007, 0xFEDCBA9876543210
    ctr = np.array([[off & 0xFFFFFFFF, off >> 32, stream, 0]], dtype=np.uint64)
    got = philox4x32_10(ctr, (seed & 0xFFFFFFFF, seed >> 32))[0]
    assert np.array_equal(got, aten_philox([(seed, stream, off)])[0])


def test_uniform_grid_exact_in_fp32():
    w = np.array([0, 1, 511, 512, 2**31, 2**32 - 1, 2**32 - 512, 0x80000200], dtype=np.uint64).astype(np.uint32)
    u = uniform_from_words(w)
    u32 = u.astype(np.float32)
    assert np.array_equal(u32.astype(np.float64), u)                    # exact in fp32
    assert np.array_equal((np.float32(1) - u32).astype(np.float64), 1.0 - u)  # 1-u exact
    assert u.min() == 2.0 ** -24 and u.max() == 1.0 - 2.0 ** -24
    assert u[1] == u[0] and u[3] == u[0] + 2.0 ** -23                    # cells of width 2^-23
    m = np.arange(0, 2**23, 4099, dtype=np.uint64)
    uu = uniform_from_words((m << np.uint64(9)).astype(np.uint32))
    assert np.all(np.diff(uu) > 0) and np.all((uu > 0) & (uu < 1))
