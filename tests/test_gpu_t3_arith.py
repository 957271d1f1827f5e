"""The Student-t draw's square root and division (Eq. 2's heavy-tailed
noise z0 / sqrt(z1^2 + z2^2 + z3^2)): the kernels use short forms of the
correctly rounded sequences, valid on the draw's ranges.  The device check
tests/device_checks/t3_arith compares them with the compiler's sqrtf and
fp32 division bit for bit: every float in [2^-96, 2^7) for the square root,
every divisor in [2^-17, 2^4) against 256 Irwin-Hall dividends for the
division (the draw reaches q in [6.9e-10, 36], s in [2.6e-5, 6] and
|z0| <= 3.47).  The uncorrected forms must differ on some of the same
inputs, so the comparison is not vacuous."""
import os
import subprocess

import pytest

from tests.conftest import ROOT
from tests.gpu_util import announce

pytestmark = pytest.mark.gpu

EXE = os.path.join(ROOT, "tests", "device_checks", "t3_arith")


def test_t3_sqrt_and_division_are_correctly_rounded():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    if not os.path.exists(EXE):
        pytest.fail("tests/device_checks/t3_arith is not built; run __graft_entry__.build()")
    announce("t3 sqrt / division device check")
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    got = dict(line.split() for line in r.stdout.strip().splitlines())
    assert int(got["sqrt_inputs"]) == 0x43000000 - 0x0F800000
    assert int(got["sqrt_differ"]) == 0
    assert int(got["div_pairs"]) == (0x41800000 - 0x37000000) * 256
    assert int(got["div_differ"]) == 0
    assert int(got["sqrt_raw_differ"]) > 0 and int(got["div_raw_differ"]) > 0
