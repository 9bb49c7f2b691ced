import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


@pytest.fixture(scope="session")
def ref():
    """The CPU oracle, rebuilt from source once per session."""
    import oracle
    from oracle import build as obuild
    obuild.build()
    return oracle


@pytest.fixture(scope="session")
def rocrand_philox(tmp_path_factory):
    """Philox4x32-10 words computed by rocRAND's host-callable engine.

    Returns f(rows) where rows is an int array [M, 5] of (seed, c0, c1, c2, c3);
    the result is a uint32 array [M, 4].
    """
    src = os.path.join(ROOT, "tests", "rocrand_philox_probe.cpp")
    exe = str(tmp_path_factory.mktemp("rocrand") / "probe")
    subprocess.run(["g++", "-O1", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", src, "-o",
                    exe], check=True)

    def run(rows):
        rows = [tuple(int(v) for v in r) for r in rows]
        text = "".join(f"{s} {a} {b} {c} {d}\n" for s, a, b, c, d in rows)
        out = subprocess.run([exe], input=text, capture_output=True, text=True,
                             check=True).stdout.split()
        return np.array([int(v) for v in out], dtype=np.uint64).astype(np.uint32).reshape(-1, 4)

    return run


def u01_exact(words):
    """The top 24 bits of each word divided by 2^24 (exact in fp32)."""
    w = np.asarray(words, dtype=np.uint64)
    return ((w >> np.uint64(8)).astype(np.float64) / float(1 << 24)).astype(np.float32)


@pytest.fixture(scope="session")
def evox_gpu():
    """The HIP library on cuda:0.  Fails (does not skip) without a GPU or library."""
    import torch
    import paper_2301_12457_amd as m
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a GPU")
    if not os.path.exists(m.LIB_PATH):
        pytest.fail(f"{m.LIB_PATH} is not built")
    m.lib()
    torch.cuda.init()
    return m
