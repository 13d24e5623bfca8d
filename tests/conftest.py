"""Shared pytest setup: the ``gpu`` marker and paths.

Tests marked ``gpu`` need an MI355X and the built HIP library; everything else runs on the
CPU. The CPU-side helper libraries (oracle, generators) are compiled with gcc on first use
if they are missing; the HIP library is never built from inside a test.
"""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(ROOT, "tests", "golden")

# Selections without an estimate vector estimate every coordinate when the sketch is small
# (d*r at most 2,000,000) and prune otherwise. The GPU tests run most shapes small, so they
# fix the pruned form, which has the most machinery (sampled bound, heavy-cell maps,
# survivors, fallback); test_gpu_parity.test_selection_path_by_size covers the automatic
# choice. Read by gs_create.
os.environ.setdefault("GS_SELECT_PATH", "pruned")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X GPU and the built HIP library")


@pytest.fixture(scope="session")
def golden_dir():
    return GOLDEN
