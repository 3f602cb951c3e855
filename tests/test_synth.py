"""Input generator: published Philox4x32-10 answers, its own log, distributions, random access."""
import ctypes
import math

import numpy as np
import pytest

import synth


def _philox(ctr, key):
    lib = synth.host_lib()
    c = (ctypes.c_uint32 * 4)(*ctr)
    k = (ctypes.c_uint32 * 2)(*key)
    o = (ctypes.c_uint32 * 4)()
    lib.synth_philox_host(c, k, o)
    return list(o)


def test_philox_known_answers():
    # Known-answer vectors of Philox4x32-10 (Salmon et al., SC'11, Random123 distribution).
    assert _philox([0, 0, 0, 0], [0, 0]) == [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]
    assert _philox([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2) == [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]
    assert _philox([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0]) == \
        [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]


def test_own_log_accuracy():
    lib = synth.host_lib()
    lib.synth_log_host.restype = ctypes.c_double
    lib.synth_log_host.argtypes = [ctypes.c_double]
    rng = np.random.default_rng(1)
    for x in np.concatenate([rng.random(2000), [1e-300, 2.0 ** -53, 0.5, 1.0, 0.70710678, 0.9999999]]):
        ref = math.log(x)
        got = lib.synth_log_host(float(x))
        assert abs(got - ref) <= 4e-16 * max(1.0, abs(ref)), (x, got, ref)


def test_fill_and_gather_agree():
    wl = synth.layer()
    a = synth.fill_host(wl, 4, 1, first=1000, n=5000)
    idx = np.arange(1000, 6000)
    b = synth.gather_host(wl, 4, 1, idx)
    assert np.array_equal(a, b)


def test_distributions():
    wl = synth.stack_7b()
    base = synth.fill_host(wl, 0, 0, n=400000)
    d = synth.fill_host(wl, 0, 1, n=400000)
    bf = (base.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    df = (d.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert abs(bf.mean()) < 1e-4 and abs(bf.std() - 0.02) < 3e-4
    nz = df[df != 0]
    assert abs(nz.size / df.size - 0.2) < 0.005
    assert abs(nz.std() - 5e-5) < 1e-6
    lap = synth.stack_1p5b()
    l = synth.fill_host(lap, 0, 1, n=400000)
    lf = (l.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    nz = lf[lf != 0]
    assert abs(nz.size / lf.size - 0.3) < 0.005
    assert abs(np.mean(np.abs(nz)) - 5e-5) < 1.5e-6       # E|X| = b for Laplace(0, b)
    t = synth.tiny()
    x = synth.fill_host(t, 0, 2)
    assert x.dtype == np.float32 and abs(np.count_nonzero(x) / x.size - 0.3) < 0.01


def test_streams_differ():
    wl = synth.layer()
    a = synth.fill_host(wl, 0, 1, n=1000)
    b = synth.fill_host(wl, 0, 2, n=1000)
    c = synth.fill_host(wl, 1, 1, n=1000)
    assert not np.array_equal(a, b) and not np.array_equal(a, c)


@pytest.mark.parametrize("name,n", [("tiny", 65536), ("layer", 51380224), ("1.5b", 1543569408),
                                    ("7b", 7615283200)])
def test_workload_sizes(name, n):
    assert synth.workload(name).numel == n


def test_threaded_fill_is_the_sequential_fill():
    wl = synth.layer()
    a = synth.fill_host(wl, 1, 2, first=77, n=(3 << 20) + 5)
    b = synth.fill_host(wl, 1, 2, first=77, n=(3 << 20) + 5, threads=3)
    assert np.array_equal(a, b)
