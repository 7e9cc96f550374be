import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP library)")
    config.addinivalue_line("markers", "slow: long CPU test")
    # A checkout without the built libraries: on a machine with no GPU (where the
    # CPU tests run) compile them with hipcc for gfx950 first, as
    # __graft_entry__.build() does.  On a GPU machine nothing is built here: a
    # missing library fails the import loudly.
    pkg = os.path.join(ROOT, "paper_2207_07736_amd")
    libs = [os.path.join(pkg, "librlsim.so"), os.path.join(pkg, "librlsim_probe.so")]
    if not all(os.path.exists(x) for x in libs) and not os.path.exists("/dev/kfd"):
        import importlib.util
        spec = importlib.util.spec_from_file_location("rlsim_build", os.path.join(pkg, "build.py"))
        mod = importlib.util.module_from_spec(spec)
        spec.loader.exec_module(mod)
        mod.build()
