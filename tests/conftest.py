import ctypes
import os
import subprocess
import sys
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parent.parent
if str(ROOT) not in sys.path:
    sys.path.insert(0, str(ROOT))


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP path)")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session")
def oracle_mod():
    import oracle
    if not oracle.LIB.exists():
        oracle.build()
    return oracle


@pytest.fixture(scope="session")
def brute(tmp_path_factory):
    """The exhaustive checker (tests/brute/brute.c), compiled for this session."""
    out = tmp_path_factory.mktemp("brute") / "brute.so"
    subprocess.run(["gcc", "-O2", "-shared", "-fPIC", "-o", str(out),
                    str(ROOT / "tests" / "brute" / "brute.c")], check=True)
    lib = ctypes.CDLL(str(out))
    lib.brute_run.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                              ctypes.c_void_p, ctypes.c_void_p]
    lib.brute_alphabet.restype = ctypes.c_char_p
    lib.brute_alphabet.argtypes = [ctypes.c_int]
    lib.brute_member.argtypes = [ctypes.c_int, ctypes.c_char_p, ctypes.c_int]
    return lib
