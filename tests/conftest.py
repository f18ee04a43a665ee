"""Shared test setup: repo root on sys.path, the `gpu` marker, native builds.

CPU tests (-m "not gpu") build the generator and the oracle libraries when
they are missing; GPU tests load the in-tree HIP library and never build it."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long CPU test")


def _ensure_host_libs():
    import oracle
    from paper_2302_11665_amd import build
    if not os.path.exists(build.GEN_LIB):
        build.build_gen()
    if not os.path.exists(oracle.LIB_PATH):
        oracle.build()


_ensure_host_libs()


@pytest.fixture(scope="session")
def olib():
    import oracle
    return oracle.lib()
