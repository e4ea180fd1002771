import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(ROOT, "tests", "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


@pytest.fixture(scope="session", autouse=True)
def _host_libs():
    """The oracle and the host-side input generator are plain C/C++ that
    build in about a second; build them if they are missing."""
    from oracle import oracle
    from paper_2606_01387_amd.synth import content

    if not os.path.exists(oracle.LIBRARY):
        oracle.build()
    if not os.path.exists(content.HOST_LIB):
        import subprocess

        subprocess.run(["gcc", "-O2", "-std=c99", "-shared", "-fPIC", content.HOST_SRC,
                        "-o", content.HOST_LIB], check=True)


@pytest.fixture(scope="session")
def torch():
    """torch, on a machine with a GPU (the GPU tests' fixture)."""
    import torch as t

    assert t.cuda.is_available(), "GPU tests need a GPU"
    return t


@pytest.fixture(scope="session")
def ck():
    """The library's binding, with the library loaded (it fails loudly when
    the library has not been built: there is no fallback)."""
    from paper_2606_01387_amd import claimkv

    claimkv.lib()
    return claimkv
