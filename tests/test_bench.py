"""Host-side contract of bench.py (no GPU): the multi-GPU refusal, the source
stamp of counter-derived traffic, and the oracle's CPU baseline record."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_source_stamp_ignores_comments_and_whitespace_only():
    csrc = os.path.join(ROOT, "paper_2609_35440_amd", "csrc")
    names = sorted(f for f in os.listdir(csrc) if f.endswith((".hip", ".h")))
    # every library source is stamped, the wide tiling and the small kernels included
    assert {"k_mfma.hip", "k_mfma_wide.hip", "mfma_layout_wide.h", "k_small.hip", "solo_api.hip"} <= set(names)
    files = {f: open(os.path.join(csrc, f)).read() for f in names}
    base = bench.kernel_sources_hash(lambda f: files[f])
    assert base == bench.kernel_sources_hash()
    changed_wide = dict(files)
    changed_wide["k_mfma_wide.hip"] = files["k_mfma_wide.hip"] + "\nstatic int extra_symbol;\n"
    assert bench.kernel_sources_hash(lambda f: changed_wide[f]) != base
    edited = dict(files)
    edited["k_mfma.hip"] = "// a new comment\n/* and a block\n comment */\n" + files["k_mfma.hip"].replace(
        "\n", "\n  ", 5)
    assert bench.kernel_sources_hash(lambda f: edited[f]) == base
    changed = dict(files)
    changed["mfma_layout.h"] = files["mfma_layout.h"].replace("constexpr int YC = 16;", "constexpr int YC = 32;")
    assert changed["mfma_layout.h"] != files["mfma_layout.h"]
    assert bench.kernel_sources_hash(lambda f: changed[f]) != base


def test_committed_traffic_record_is_stamped():
    rec = json.load(open(os.path.join(ROOT, "profiles", "traffic_local_loss_1b.json")))
    for key in ("kernel_sources_sha256_16", "bytes_per_launch", "fetch_bytes", "write_bytes", "fetch_scale",
                "write_scale", "commands"):
        assert key in rec, key
    assert abs(rec["fetch_bytes"] + rec["write_bytes"] - rec["bytes_per_launch"]) <= 1e-6 * rec["bytes_per_launch"]


def test_cpu_baseline_record():
    r = bench.cpu_baseline("tiny", 16)
    for key in ("value", "unit", "cores", "cpu_model", "gflops_algorithmic", "kind", "sample", "seconds"):
        assert key in r, key
    assert r["kind"] == "oracle" and r["unit"] == "tokens/s"
    assert r["value"] > 0 and r["cores"] >= 1 and r["gflops_algorithmic"] > 0
    assert "T=16" in r["sample"]
