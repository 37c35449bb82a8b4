"""Host logic of the fused recouple tables (no GPU): the per-degree tables of
the alpha / D^f variant (Alg. 1's alpha^(k) = alpha / D^k per filter degree)
partition the plain layer's terms, and the passes that stack several degrees
in the K rows hold exactly the per-degree tables at their segments' rows.
tests/fuse_tables_check.cpp is built with g++ against the library's
tables.cpp and run; see its header for the checks."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2501_19216_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_fuse_tables_stacked_and_per_degree(tmp_path):
    exe = str(tmp_path / "fuse_tables_check")
    cmd = ["g++", "-O2", "-std=c++17", "-I", CSRC, "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "fuse_tables_check.cpp"), os.path.join(CSRC, "tables.cpp"), "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True, timeout=300)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    print(r.stdout)
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert r.returncode == 0, r.stdout + r.stderr
    # per L: the per-degree check, the cover check and one line per pass (two at L = 4)
    assert len(lines) == 5 * 2 + 6 and all(": ok" in l for l in lines), r.stdout
