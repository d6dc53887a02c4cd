"""Host-side check of the attention kernel's score-operand bit-field plans:
compiles tests/kplan_check.cpp against the package header with g++ and runs it.
The identity it checks is plain arithmetic (a dot product of integer codes
recovered from masked, scaled bit fields); no oracle is involved."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_07915_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_score_field_plans_reproduce_code_dot_products():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "kplan_check")
        subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", f"-I{CSRC}",
                        os.path.join(ROOT, "tests", "kplan_check.cpp"), "-o", exe], check=True)
        r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
        assert r.returncode == 0 and r.stdout.strip() == "OK", r.stdout + r.stderr
