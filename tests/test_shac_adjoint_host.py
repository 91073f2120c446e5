"""The SHAC window kernel's reverse-mode physics (csrc/shac_adjoint.hpp) checked on the CPU:
the header's templates instantiated in double by tests/shac_adjoint_check.cpp (g++), every
vector-Jacobian product (Fossen right side, RK4 substep with renormalisation, observation
in its general, small-angle and negative-scalar branches, reward) against central
differences of the forward it differentiates."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2512_13359_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_adjoint_products_match_finite_differences(tmp_path):
    exe = str(tmp_path / "adjoint_check")
    subprocess.run(["g++", "-O2", "-std=c++17", "-Wall", "-Werror", f"-I{CSRC}",
                    os.path.join(HERE, "shac_adjoint_check.cpp"), "-o", exe], check=True)
    out = subprocess.run([exe], capture_output=True, text=True)
    print(out.stdout)
    assert out.returncode == 0, out.stdout
    assert out.stdout.strip().endswith("OK")
    assert out.stdout.count("max rel err") == 6
