import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the C ABI on a GPU)")
    config.addinivalue_line("markers", "slow: large host-side work")


def _built():
    libs = [
        os.path.join(ROOT, "oracle", "liboracle.so"),
        os.path.join(ROOT, "kvsynth", "libkvsynth_host.so"),
        os.path.join(ROOT, "kvsynth", "libkvsynth_dev.so"),
        os.path.join(ROOT, "paper_2609_11744_amd", "libkvx.so"),
    ]
    return all(os.path.exists(p) for p in libs)


def pytest_sessionstart(session):
    # KVX_TEST_LIB: run the tests against another build of libkvx (the
    # sanitizer tests' host-only build); nothing outside tests/ reads it.
    if os.environ.get("KVX_TEST_LIB"):
        from paper_2609_11744_amd import _native

        _native.LIB_PATH = os.environ["KVX_TEST_LIB"]
    # Build only when nothing is built; after a source change run
    # __graft_entry__.build() before pytest.
    if not _built() and not os.environ.get("KVX_NO_AUTOBUILD"):
        import __graft_entry__

        __graft_entry__.build()
