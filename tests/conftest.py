import ctypes
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


@pytest.fixture(scope="session")
def orc():
    import oracle
    oracle.build()
    return oracle


@pytest.fixture(scope="session")
def dg():
    import datagen
    datagen.build()
    return datagen


@pytest.fixture(scope="session")
def pins(orc, tmp_path_factory):
    """The native pin loops (tests/native/pins.c), linked against the oracle."""
    src = os.path.join(ROOT, "tests", "native", "pins.c")
    out = str(tmp_path_factory.mktemp("pins") / "libpins.so")
    odir = os.path.dirname(orc._LIB)
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-pthread", src, "-o", out,
                           "-L" + odir, "-loracle", "-Wl,-rpath," + odir])
    L = ctypes.CDLL(out)
    vp, u32, u64 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64
    L.pin_bounded_exhaustive.restype = ctypes.c_int
    L.pin_bounded_exhaustive.argtypes = [u32, vp, ctypes.POINTER(u64), ctypes.c_int]
    for name in ("pin_subset_hist", "pin_subset_hist_nodes", "pin_marginals"):
        fn = getattr(L, name)
        fn.restype = ctypes.c_int
        fn.argtypes = [u32, u32, u32, u32, u64, u64, vp]
    return L
