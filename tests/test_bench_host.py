"""Host-side pieces of bench.py (no GPU): the one-GPU guard and the measured-traffic record."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

PROFILE = os.path.join("profiles", "mix_resnet50_stage1_hbm_bytes.md")
SOURCES = ("paper_2608_23794_amd/csrc/mfmamix.hip", "paper_2608_23794_amd/csrc/moce_internal.h")


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def _tree(tmp_path, edit=None):
    """A copy of the sources with a counter record taken for exactly these sources, then `edit` appended to."""
    import hashlib
    h = hashlib.sha256()
    for f in SOURCES:
        dst = tmp_path / f
        dst.parent.mkdir(parents=True, exist_ok=True)
        shutil.copy(os.path.join(ROOT, f), dst)
        h.update(open(dst, "rb").read())
    lines = []
    for ln in open(os.path.join(ROOT, PROFILE)):
        if ln.startswith("sources_sha256:"):
            ln = f"sources_sha256: {h.hexdigest()}\n"
        lines.append(ln)
    (tmp_path / PROFILE).parent.mkdir(parents=True, exist_ok=True)
    (tmp_path / PROFILE).write_text("".join(lines))
    if edit:
        with open(tmp_path / edit, "a") as fh:
            fh.write("\n// edited\n")
    return str(tmp_path)


def _record_kernel():
    for ln in open(os.path.join(ROOT, PROFILE)):
        if ln.startswith("kernel:"):
            return ln.partition(":")[2].strip()
    raise AssertionError("no kernel line in the counter record")


def test_traffic_record_is_the_calibrated_counters():
    """The reported figure is the record's calibrated sum while the sources hash to its value (null after a
    change to the kernel, until the counters are taken again)."""
    import hashlib
    rec = {}
    for ln in open(os.path.join(ROOT, PROFILE)):
        k, sep, v = ln.partition(":")
        if sep:
            rec[k.strip()] = v.strip()
    h = hashlib.sha256()
    for f in rec["sources"].split():
        h.update(open(os.path.join(ROOT, f), "rb").read())
    t = bench.measured_traffic(rec["kernel"])
    if h.hexdigest() != rec["sources_sha256"]:
        assert t is None
        return
    assert t == int(rec["traffic_bytes"])
    # the record is the calibrated sum of the two counters
    fetch = float(rec["fetch_kib_per_dispatch"]) * 1024 * float(rec["fetch_scale"])
    write = float(rec["write_kib_per_dispatch"]) * 1024 * float(rec["write_scale"])
    assert t == pytest.approx(fetch + write, rel=1e-6)
    assert bench.measured_traffic("another_kernel") is None


@pytest.mark.parametrize("edit", SOURCES)
def test_traffic_is_null_once_the_kernel_changed(tmp_path, monkeypatch, edit):
    kernel = _record_kernel()
    monkeypatch.setattr(bench, "ROOT", _tree(tmp_path))
    assert bench.measured_traffic(kernel) is not None
    monkeypatch.setattr(bench, "ROOT", _tree(tmp_path / "edited", edit))
    assert bench.measured_traffic(kernel) is None
