import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU statistics test")


@pytest.fixture(scope="session")
def torch_philox(tmp_path_factory):
    """Philox4x32-10 words computed by PyTorch's own open-source engine
    (ATen/core/PhiloxRNGEngine.h), compiled into a tiny helper and called --
    an implementation independent of the oracle's."""
    import torch
    inc = os.path.join(os.path.dirname(torch.__file__), "include")
    src = os.path.join(os.path.dirname(os.path.abspath(__file__)), "philox_ref.cpp")
    exe = str(tmp_path_factory.mktemp("philox") / "philox_ref")
    subprocess.run(["g++", "-std=c++17", "-O1", "-I" + inc, "-o", exe, src], check=True)

    def run(rows):
        """rows: iterable of (c0, c1, c2, c3, k0, k1) -> array [n, 4] uint32."""
        rows = [tuple(int(x) & 0xFFFFFFFF for x in r) for r in rows]
        txt = "\n".join(" ".join(str(x) for x in r) for r in rows) + "\n"
        out = subprocess.run([exe], input=txt, capture_output=True, text=True, check=True).stdout
        return np.array([[int(x) for x in line.split()] for line in out.strip().splitlines()], dtype=np.uint64)

    return run
