"""Host logic of bench.py, on the CPU: the refusal of more than one GPU, and
the rule that the HBM traffic figure comes from the committed counter summary
only while the profiled sources are unchanged."""
import json
import os
import shutil
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120)
    assert out.returncode == 2
    rec = json.loads(out.stdout.strip().splitlines()[-1])
    assert rec["requested_gpus"] == 2 and "one GPU" in rec["error"]


def _tree(tmp_path):
    """A copy of the files pmc_traffic reads."""
    for rel in ("profiles/diff_kernel_sweep_pmc.md",
                *("paper_2608_20711_amd/csrc/" + f for f in bench.PROFILED_SOURCES)):
        dst = tmp_path / rel
        dst.parent.mkdir(parents=True, exist_ok=True)
        shutil.copy(os.path.join(ROOT, rel), dst)
    return tmp_path


def test_traffic_only_while_the_profiled_sources_are_unchanged(tmp_path, monkeypatch):
    root = _tree(tmp_path)
    monkeypatch.setattr(bench, "ROOT", str(root))
    line = next(l for l in open(root / "profiles/diff_kernel_sweep_pmc.md") if l.strip().startswith("PMC_TRAFFIC "))
    rec = json.loads(line.strip()[len("PMC_TRAFFIC "):])
    got = bench.pmc_traffic()
    if got is not None:                           # the committed summary matches the committed sources
        assert got == rec["bytes_per_launch"]
        # the recorded bytes are the calibrated counters of one launch
        want = rec["fetch_kib"] * 1024 * rec["fetch_scale"] + rec["write_kib"] * 1024 * rec["write_scale"]
        assert abs(got - want) <= 5e-6 * got      # the scale factors are recorded to 5 decimals
    with open(root / "paper_2608_20711_amd/csrc/diff.hip", "a") as f:
        f.write("\n// changed\n")
    assert bench.pmc_traffic() is None            # a changed kernel source voids the figure
    os.remove(root / "paper_2608_20711_amd/csrc/diff.hip")
    assert bench.pmc_traffic() is None            # so does a missing one
    (root / "profiles/diff_kernel_sweep_pmc.md").write_text("no summary here\n")
    assert bench.pmc_traffic() is None
