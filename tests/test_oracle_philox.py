"""Pin the oracle's Philox4x32-10 against an independent implementation: PyTorch's
header-only engine (ATen/core/PhiloxRNGEngine.h), compiled here with g++ and
driven only through its public interface (seed, subsequence, offset)."""
import os
import subprocess

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def torch_philox(tmp_path_factory):
    import torch

    inc = os.path.join(os.path.dirname(torch.__file__), "include")
    exe = str(tmp_path_factory.mktemp("philox") / "torch_philox_stream")
    src = os.path.join(HERE, "philox_ref", "torch_philox_stream.cpp")
    subprocess.run(["g++", "-std=c++17", "-O1", "-I", inc, src, "-o", exe], check=True)

    def run(triples):
        text = "".join(f"{s} {sub} {off}\n" for s, sub, off in triples)
        out = subprocess.run([exe], input=text, capture_output=True, text=True, check=True).stdout
        return [tuple(int(v) for v in line.split()) for line in out.strip().splitlines()]

    return run


def _oracle_words(seed, sub, off):
    # torch's engine: key = seed halves, counter = (offset lo, offset hi, subsequence lo, hi)
    ctr = (off & 0xFFFFFFFF, off >> 32, sub & 0xFFFFFFFF, sub >> 32)
    key = (seed & 0xFFFFFFFF, seed >> 32)
    return tuple(int(v) for v in oracle.philox4x32_10(ctr, key))


def test_philox_matches_torch_engine(torch_philox):
    rng = np.random.default_rng(7)
    M64 = (1 << 64) - 1
    triples = [(0, 0, 0), (M64, M64, M64), (1, 0, 0), (0, 1, 0), (0, 0, 1),
               (0xA4093822299F31D0, 0x13198A2E03707344, 0x243F6A8885A308D3)]
    for _ in range(300):
        w = [int(v) for v in rng.integers(0, 2**32, size=6, dtype=np.uint64)]
        triples.append((w[0] | w[1] << 32, w[2] | w[3] << 32, w[4] | w[5] << 32))
    ref = torch_philox(triples)
    got = [_oracle_words(*t) for t in triples]
    assert got == ref


def test_uniform_u64_counter_layout(torch_philox):
    # draw k of token j, batch row b, seed s -> counter (k, j, b, 0), key (s_lo, s_hi)
    seed, b, j = 0x0123456789ABCDEF, 5, 77
    ks = [0, 1, 2, 1000]
    trip = [(seed, b, (j << 32) | k) for k in ks]
    ref = torch_philox(trip)
    got = oracle.uniform_u64(seed, b, j, ks)
    assert got == [w[0] | (w[1] << 32) for w in ref]


def test_vectorised_equals_scalar():
    ks = np.arange(64, dtype=np.uint64)
    vec = oracle.philox4x32_10((ks, ks * 3, ks + 9, ks ^ 5), (11, 12))
    for i in range(64):
        one = oracle.philox4x32_10((int(ks[i]), int(ks[i]) * 3, int(ks[i]) + 9, int(ks[i]) ^ 5), (11, 12))
        assert tuple(int(v[i]) for v in vec) == tuple(int(v) for v in one)
