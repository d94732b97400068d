"""Arithmetic identities the quantizer kernels use in place of the
straightforward forms, checked on the CPU in binary32
(tests/arith/kernel_identities.c, built here with gcc -ffp-contract=off):

- stochastic rounding as ceil(t - u) of the exact ratio, against
  "floor + 1 iff u * step < m - floor" on the E2M1, E2M3, E3M2 and E2M0
  grids and the INT candidates, every sampled fp32 magnitude of each range
  with the draws at, below and above its fraction;
- the group-scale quotient by Markstein's correction, against the correctly
  rounded division, as the E4M3 encoder consumes it.

The sampled strides keep this to a few seconds; stride 1 (every value) was
run too and found no difference."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "arith", "kernel_identities.c")


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path_factory.mktemp("arith") / "kernel_identities")
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-o", exe, SRC, "-lm"], check=True)
    return exe


@pytest.mark.parametrize("what, stride", [("sr", 97), ("div", 61)])
def test_kernel_identity(checker, what, stride):
    out = subprocess.run([checker, what, str(stride)], capture_output=True, text=True)
    assert out.returncode == 0, out.stdout + out.stderr
    n, bad = (int(w) for w in out.stdout.split()[1::2][:2])
    assert bad == 0 and n > 10 ** 8, out.stdout
