"""Shared pytest set-up: the ``gpu`` marker and the native test helpers.

The seeded generator (``synth``) and the CPU oracle (``oracle``) are small
host libraries; they are compiled here on first use if the tree has no built
copy yet.  The GPU library is never built by the tests: build it first
(``python -c "import __graft_entry__ as g; g.build()"``).
"""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


def _ensure_host_libs():
    import oracle
    import synth
    if not os.path.exists(synth._LIB_PATH):
        synth.build()
    if not os.path.exists(oracle._LIB_PATH):
        oracle.build()


_ensure_host_libs()
