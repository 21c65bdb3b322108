"""Host check of the matrix-core kernels' data layouts (mfma_layout.h,
mfma_layout_wide.h): compiled with g++ from the same headers the kernels
include, it emulates on the CPU the direct-to-LDS stream and both operand
reads of the 16-row tiling, the tiled-copy loads of the register-fed passes,
and the wide tiling's operand-register writes and transposing reads."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_layouts_deliver_every_operand(tmp_path):
    exe = tmp_path / "mfma_layout_check"
    src = os.path.join(ROOT, "tests", "native", "mfma_layout_check.cpp")
    inc = os.path.join(ROOT, "paper_2609_35440_amd", "csrc")
    subprocess.run(["g++", "-std=c++17", "-O1", f"-I{inc}", src, "-o", str(exe)], check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True)
    print(r.stdout)
    assert r.returncode == 0, r.stdout
    rows = {(int(m.group(1)), int(m.group(2))): m for m in re.finditer(
        r"DS=(\d+) waves=(\d+) padded=(\d) slice=\d+ errors=(\d+) row_conflicts=(\d+) tr_conflicts=(\d+) "
        r"tiled_errors=(\d+)", r.stdout)}
    assert sorted(rows) == [(32, 8), (64, 8), (96, 8), (128, 8), (160, 8), (192, 8), (224, 8), (256, 8)]
    for key, m in rows.items():
        assert int(m.group(4)) == 0, key
        assert int(m.group(7)) == 0, key
        if m.group(3) == "1":  # padded layouts (DS = 128, 256): both read patterns conflict-free
            assert int(m.group(5)) == 0, key
            assert int(m.group(6)) == 0, key
    # the wide layout: every write lands once and every read returns its operand;
    # at the shipped width (320 columns per wave) both access patterns are conflict-free
    wide = {int(m.group(1)): m for m in re.finditer(
        r"WIDE DS=(\d+) slice=\d+ errors=(\d+) write_conflicts=(\d+) tr_conflicts=(\d+)", r.stdout)}
    assert sorted(wide) == [320, 384]
    for ds, m in wide.items():
        assert int(m.group(2)) == 0, ds
    assert [int(wide[320].group(i)) for i in (3, 4)] == [0, 0]
