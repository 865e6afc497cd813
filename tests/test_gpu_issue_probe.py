"""The issue-cost probe library (libmca_probe.so, include/mca_probe.h) on the GPU: every
kind runs, every wave leaves its clock stamps, and the stamps advance. Timing-independent:
the measured costs themselves are reported by `bench.py --issue-probe`, not asserted."""
import ctypes
import os

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROBE = os.path.join(ROOT, "paper_2201_12854_amd", "libmca_probe.so")


@pytest.fixture(scope="module")
def probe():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    if not os.path.exists(PROBE):
        raise RuntimeError(f"{PROBE} is not built")
    torch.cuda.init()
    lib = ctypes.CDLL(PROBE)
    f = lib.mca_issue_probe
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_longlong), ctypes.c_int,
                  ctypes.POINTER(ctypes.c_int)]
    return f, torch.cuda.get_device_properties(0).multi_processor_count


@pytest.mark.parametrize("kind,w", [(0, 1), (1, 2), (2, 4), (3, 1), (4, 2), (5, 2), (6, 2), (7, 1), (8, 4)])
def test_issue_probe_stamps(probe, kind, w):
    f, ncu = probe
    cap = 8192
    buf = (ctypes.c_longlong * (4 * cap))()
    nw = ctypes.c_int(0)
    rounds = 64
    assert f(kind, w, rounds, buf, cap, ctypes.byref(nw)) == 0
    assert nw.value == ncu * 4 * w
    st = np.frombuffer(buf, dtype=np.int64, count=4 * nw.value).reshape(-1, 4)
    assert np.all(st[:, 1] > st[:, 0])   # shader clock advanced over the rounds
    assert np.all(st[:, 3] >= st[:, 2])  # 100 MHz clock did not run backwards
    # a round is at least one instruction of a few cycles per wave
    assert np.median(st[:, 1] - st[:, 0]) >= rounds
    # too small a stamp buffer is rejected after the wave count is known
    assert f(kind, w, rounds, buf, nw.value - 1, ctypes.byref(nw)) == -1
