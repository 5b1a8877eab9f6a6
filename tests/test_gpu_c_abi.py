"""The C ABI from plain C: tests/c_abi/jorge_c_driver (gcc, C11, no Python or
PyTorch in the process) takes Jorge steps on seeded inputs, and its
parameters, L_hat, R_hat, m and m_SGD must equal bitwise those of the same
steps taken through the Python binding on torch's stream. The library's
results do not depend on the caller or the stream (fixed-order reductions, no
atomics)."""
import os
import subprocess
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)
from c_abi_inputs import uniform  # noqa: E402
from paper_2310_12298_amd.jorge import Jorge  # noqa: E402

pytestmark = pytest.mark.gpu
DRIVER = os.path.join(HERE, "c_abi", "jorge_c_driver")
HP = dict(lr=0.1, beta2=0.9, beta1=0.9, weight_decay=5e-4)


def python_run(shapes, seed, steps):
    params = [torch.from_numpy(uniform(seed, 0, l, m * n).reshape(m, n)).cuda() for l, (m, n) in enumerate(shapes)]
    opt = Jorge(shapes)
    for t in range(1, steps + 1):
        G = [torch.from_numpy(uniform(seed, t, l, m * n, 1e-2).reshape(m, n)).cuda()
             for l, (m, n) in enumerate(shapes)]
        opt.step(params, G, **HP)
    out = []
    for l, p in enumerate(params):
        out.append(p.cpu().numpy())
        for k in ("L", "R", "mom", "mom_sgd"):
            out.append(opt.get_state(l, k).cpu().numpy())
    return out


@pytest.mark.parametrize("shapes,steps", [
    ([(64, 96), (200, 300), (512, 1152)], 4),     # grouped levels, split tiles, both orders
    ([(48, 40), (100, 70), (128, 128)], 3),       # an all-small context: the LDS chains
])
def test_c_driver_matches_the_python_binding_bitwise(tmp_path, shapes, steps):
    if not os.path.exists(DRIVER):
        pytest.fail(f"{DRIVER} is not built: run __graft_entry__.build() first")
    seed = 5
    out = tmp_path / "c_out.bin"
    args = [DRIVER, str(out), str(seed), str(steps)] + [str(v) for s in shapes for v in s]
    print("running", " ".join(args[1:]), flush=True)
    res = subprocess.run(args, capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert f"steps {steps} nonfinite 0" in res.stdout, res.stdout
    raw = np.fromfile(out, dtype=np.float32)
    ref = python_run(shapes, seed, steps)
    assert raw.size == sum(r.size for r in ref)
    off = 0
    for i, r in enumerate(ref):
        got = raw[off:off + r.size].reshape(r.shape)
        off += r.size
        assert np.array_equal(got, r), (i // 5, ("theta", "L", "R", "mom", "mom_sgd")[i % 5])
