"""Host logic of bench.py (CPU only): the one-GPU contract, and the lookup
of the committed counter summaries that roofline.traffic comes from."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_recorded_traffic_follows_the_kernel_sources(tmp_path, monkeypatch):
    # a counter summary recorded for the current sources is found by its keys
    prof = tmp_path / "profiles"
    prof.mkdir()
    keys = {"workload": "qwen2.5-7b->qwen2.5-1.5b", "precision": "bf16x2", "src_tokens": "4096",
            "batch": "1", "target_layout": "contiguous",
            "kernel_source_sha256": bench.kernel_source_hash(),
            "traffic_bytes_per_launch": "370097794"}
    (prof / "fused_kernel_x.md").write_text(
        "# summary\n\n" + "".join(f"- `{k}`: `{v}`\n" for k, v in keys.items()))
    look = lambda *a: bench.recorded_traffic(*a, profiles=str(prof))  # noqa: E731
    assert look("qwen2.5-7b->qwen2.5-1.5b", "bf16x2", 4096, 1, "contiguous") == 370097794
    # another precision, size or layout has no summary
    assert look("qwen2.5-7b->qwen2.5-1.5b", "f16", 4096, 1, "contiguous") is None
    assert look("qwen2.5-7b->qwen2.5-1.5b", "bf16x2", 2048, 1, "contiguous") is None
    assert look("qwen2.5-7b->qwen2.5-1.5b", "bf16x2", 4096, 1, "paged16") is None
    # a changed fused-kernel source invalidates it; the fit's and the staged
    # path's sources do not
    src = tmp_path / "csrc"
    shutil.copytree(bench.KERNEL_SOURCES, src)
    monkeypatch.setattr(bench, "KERNEL_SOURCES", str(src))
    h0 = bench.kernel_source_hash()
    for other in ("fit.hip", "staged.hip", "staged.h"):
        with open(src / other, "a") as fh:
            fh.write("\n// edit\n")
    assert bench.kernel_source_hash() == h0
    with open(src / "kernel_mfma.h", "a") as fh:
        fh.write("\n// edit\n")
    assert bench.kernel_source_hash() != h0
    assert look("qwen2.5-7b->qwen2.5-1.5b", "bf16x2", 4096, 1, "contiguous") is None


def test_committed_summaries_are_parsable():
    """Every committed fused-kernel summary carries the keys the lookup reads."""
    import glob
    for path in glob.glob(os.path.join(ROOT, "profiles", "fused_kernel_*.md")):
        text = open(path).read()
        for k in ("workload", "precision", "src_tokens", "kernel_source_sha256"):
            assert f"- {k}: " in text, (path, k)
