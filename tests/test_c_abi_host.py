"""The plain C caller of the library (tests/c_abi/jorge_c_driver.c), on the CPU:
it compiles as strict C11 with gcc against include/jorge.h, and without a GPU
it stops at its first HIP call with a message and exit status 1. Its input
generator's Python twin (tests/c_abi_inputs.py) is pinned to splitmix64's
published first outputs."""
import os
import subprocess
import sys

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "c_abi"))
from build_driver import build_driver, command  # noqa: E402
from c_abi_inputs import splitmix64, uniform  # noqa: E402

LIB = os.path.join(os.path.dirname(HERE), "paper_2310_12298_amd", "libjorge.so")


def test_splitmix64_matches_its_published_sequence():
    # The generator with state 1234567: the state advances by the golden gamma
    # before each output (reference values of the published algorithm).
    state = np.uint64(1234567)
    out = []
    for _ in range(3):
        out.append(int(splitmix64(state)))
        with np.errstate(over="ignore"):
            state = state + np.uint64(0x9E3779B97F4A7C15)
    assert out == [6457827717110365317, 3203168211198807973, 9817491932198370423]


def test_uniform_inputs_are_exact_and_in_range():
    u = uniform(3, 2, 1, 100000)
    assert u.dtype == np.float32 and u.min() >= -1.0 and u.max() < 1.0
    q = (u.astype(np.float64) + 1.0) * 2**23
    assert np.array_equal(q, np.round(q))          # 24-bit integers over 2^23, exact in fp32
    assert abs(u.mean()) < 0.01 and abs(u.std() - 1 / np.sqrt(3)) < 0.01


@pytest.mark.skipif(not os.path.exists(LIB), reason="libjorge.so is not built")
def test_driver_compiles_as_c11_and_fails_cleanly_without_a_gpu(tmp_path):
    out = str(tmp_path / "drv")
    build_driver(out)
    assert "-std=c11" in command(out) and "-Werror" in command(out)
    if os.path.exists("/dev/kfd"):
        pytest.skip("a GPU is present: the run is the GPU test's")
    # Built outside the tree, the binary finds the library through the loader's path.
    env = dict(os.environ, LD_LIBRARY_PATH=os.path.dirname(LIB))
    res = subprocess.run([out, str(tmp_path / "o.bin"), "1", "1", "8", "8"], capture_output=True, text=True,
                         timeout=60, env=env)
    assert res.returncode == 1, res.stdout + res.stderr
    assert "jorge_c_driver: hipMalloc" in res.stderr and "failed" in res.stderr, res.stderr
    res = subprocess.run([out], capture_output=True, text=True, timeout=60, env=env)
    assert res.returncode == 2 and "usage" in res.stderr
