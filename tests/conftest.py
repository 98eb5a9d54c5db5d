import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")
    # W2V_TEST_LIB: run the tests against another build of libw2v (the sanitizer build of the host code)
    if os.environ.get("W2V_TEST_LIB"):
        import paper_1606_07822_amd
        paper_1606_07822_amd.LIB_PATH = os.environ["W2V_TEST_LIB"]


@pytest.fixture(scope="session", autouse=True)
def _built_c_helpers():
    """The oracle and the input generator are plain C; build them if missing (gcc, seconds)."""
    import oracle
    oracle.build()
    import subprocess
    so = os.path.join(ROOT, "synth", "libsynth.so")
    src = os.path.join(ROOT, "synth", "synth.c")
    if not os.path.exists(so) or os.path.getmtime(so) < os.path.getmtime(src):
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-std=c11", "-fPIC", "-shared", src, "-o", so, "-lm"])
