"""Pin: the oracle's Philox4x32-10 against an independent implementation.

The generator is the counter-based Philox4x32-10 of Salmon, Moraes, Dror and
Shaw (SC'11).  rocRAND ships an open-source, host-callable implementation of
the same bijection; a tiny test-only shim exposes it so that the two can be
compared on many (counter, key) pairs, including extreme words.
"""
import ctypes
import os
import shutil
import subprocess

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def rocrand_philox(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc) or not os.path.exists("/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"):
        pytest.skip("hipcc or the rocRAND headers are not installed")
    out = str(tmp_path_factory.mktemp("shim") / "shim.so")
    subprocess.check_call([hipcc, "-O1", "-fPIC", "-shared", "--offload-arch=gfx950", "-o", out,
                           os.path.join(HERE, "rocrand_philox_shim.cpp")], cwd="/tmp")
    lib = ctypes.CDLL(out)
    fn = lib.shim_philox4x32_10
    u32p = ctypes.POINTER(ctypes.c_uint32)
    fn.argtypes = [u32p, u32p, u32p, ctypes.c_int]
    fn.restype = None

    def run(ctr, key):
        ctr = np.ascontiguousarray(ctr, dtype=np.uint32)
        key = np.ascontiguousarray(key, dtype=np.uint32)
        out = np.zeros_like(ctr)
        n = ctr.shape[0]
        fn(ctr.ctypes.data_as(u32p), key.ctypes.data_as(u32p), out.ctypes.data_as(u32p), n)
        return out

    return run


def test_philox_matches_rocrand(oracle_mod, rocrand_philox):
    rng = np.random.default_rng(123)
    n = 2000
    ctr = rng.integers(0, 2**32, size=(n, 4), dtype=np.uint64).astype(np.uint32)
    key = rng.integers(0, 2**32, size=(n, 2), dtype=np.uint64).astype(np.uint32)
    # extreme words
    ctr[0] = 0; key[0] = 0
    ctr[1] = 0xFFFFFFFF; key[1] = 0xFFFFFFFF
    ctr[2] = [0, 1, 2, 3]; key[2] = [0x50A10000, 0]
    ref = rocrand_philox(ctr, key)
    ours = np.stack([oracle_mod.philox(ctr[i], key[i]) for i in range(n)])
    assert np.array_equal(ours, ref)


def test_philox_is_not_identity_and_depends_on_every_word(oracle_mod):
    base_c = np.array([1, 2, 3, 4], np.uint32)
    base_k = np.array([5, 6], np.uint32)
    y = oracle_mod.philox(base_c, base_k)
    for i in range(4):
        c = base_c.copy(); c[i] ^= 1
        assert not np.array_equal(oracle_mod.philox(c, base_k), y)
    for i in range(2):
        k = base_k.copy(); k[i] ^= 1
        assert not np.array_equal(oracle_mod.philox(base_c, k), y)
