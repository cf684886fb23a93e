"""The posterior's row plans (which row blocks of V each wave owns, and the
order in which the packed inverse factor streams them; 16-row blocks in both
precisions), checked on the host
for every observation count the library accepts: tests/row_plan_check.cpp,
built here with the host compiler against the library's internal header."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_row_plans_every_size(tmp_path):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    exe = str(tmp_path / "row_plan_check")
    subprocess.run([cxx, "-O1", "-std=c++17", "-I", os.path.join(ROOT, "include"), "-I",
                    os.path.join(ROOT, "paper_2408_04323_amd", "csrc"),
                    os.path.join(ROOT, "tests", "row_plan_check.cpp"), "-o", exe], check=True)
    r = subprocess.run([exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout
    lines = r.stdout.splitlines()
    assert len(lines) == 18 and not any("BAD" in line for line in lines)
