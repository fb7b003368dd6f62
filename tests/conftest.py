import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


# Tests that must run at one end of a session, whatever the selection (-k,
# file order, plugins): the cross-process replay needs the device free of
# this process's own context, so it goes first; the entry point that keeps
# its scratch in a static device array shares that array with nothing else
# if it runs last.
_FIRST = ("test_gpu_a_va_replay.py",)
_LAST = ("test_zz_no_alloc.py",)


def pytest_collection_modifyitems(session, config, items):
    def rank(item):
        name = item.nodeid.split("::")[0].rsplit("/", 1)[-1]
        return 0 if name in _FIRST else 2 if name in _LAST else 1
    items.sort(key=rank)            # stable: the order within each group is kept
