"""The oracle's Philox4x32-10 (the generator of the stochastic rounding)
against a library implementation: rocRAND's Philox4x32-10 host generator
produces, for seed s, the words of counters (n, 0, 0, 0) under key
(s mod 2^32, s / 2^32) in order.  rocRAND's host generator needs the HIP
runtime with a device, hence a GPU test; it runs no kernel of this library."""
import ctypes
import os

import numpy as np
import pytest

from oracle import oracle as O

ROCRAND = "/opt/rocm/lib/librocrand.so"
PHILOX4_32_10 = 404


@pytest.mark.gpu
@pytest.mark.parametrize("seed", [0, 1, 0x123456789ABCDEF0, 2 ** 64 - 1])
def test_philox_matches_rocrand(seed):
    assert os.path.exists(ROCRAND), "rocRAND is part of the ROCm image"
    L = ctypes.CDLL(ROCRAND)
    g = ctypes.c_void_p()
    assert L.rocrand_create_generator_host_blocking(ctypes.byref(g), PHILOX4_32_10) == 0
    try:
        assert L.rocrand_set_seed(g, ctypes.c_ulonglong(seed)) == 0
        n = 256
        out = np.zeros(4 * n, dtype=np.uint32)
        assert L.rocrand_generate(g, out.ctypes.data_as(ctypes.c_void_p), ctypes.c_size_t(out.size)) == 0
    finally:
        L.rocrand_destroy_generator(g)
    key = [seed & 0xFFFFFFFF, seed >> 32]
    want = np.concatenate([O.philox4x32_10([i, 0, 0, 0], key) for i in range(n)])
    assert np.array_equal(out, want)
