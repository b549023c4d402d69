import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: larger CPU cases")
    # host-only libraries are cheap to build; build them if absent
    for sub, lib in (("synth", "libsynth.so"), ("oracle", "liboracle.so")):
        if not os.path.exists(os.path.join(ROOT, sub, lib)):
            subprocess.check_call(["make", "-s", "-C", os.path.join(ROOT, sub)])
