"""bench.py's contract pieces that need no GPU: the one-GPU guard, the
algorithmic byte counts it reports, and the memory-counter summary it
reads."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_algorithmic_bytes_of_the_workloads():
    import bench
    import synth
    wl = synth.workload("resnet50")
    ab = bench.algorithmic_bytes(wl, 25558, detach=False)
    K, d = 16, 25557032
    # read g, e and write e per worker-element; w_t, w_prev, then w read and written; messages
    assert ab["step"] == 12 * K * d + 16 * d + 16 * K * 25558 == 5322405504
    assert ab["fused"] == 12 * K * d + 8 * d
    rb = synth.workload("rbgs")
    m = 63 * 4096
    ab = bench.algorithmic_bytes(rb, m, detach=True)
    assert ab["step"] == 12 * 8 * d + 16 * d + 8 * 8 * m + 4 * 8 * d
    assert ab["fused"] == 12 * 8 * d + 8 * d + 4 * 8 * m + 4 * 8 * d
    # sparse momentum term: the bitmap and the changed components instead of w_t, w_prev;
    # the server pass reads the old bitmap, writes the new one, and moves w only at the
    # old and the new entries
    ab = bench.algorithmic_bytes(wl, 25558, detach=False, sparse_w=True)
    assert ab["fused"] == 12 * K * d + d // 8 + 8 * K * 25558
    assert ab["step"] == (12 * K * d + d // 8 + 8 * K * 25558 + 2 * (d // 8) + 16 * K * 25558
                          + 16 * K * 25558)


def test_pmc_summary_matches_the_sources_or_is_ignored(tmp_path, monkeypatch):
    import bench
    if not os.path.exists(bench.PMC_SUMMARY):
        pytest.skip("no counter summary committed")
    t = bench.read_pmc_summary()
    kv = {}
    with open(bench.PMC_SUMMARY) as f:
        for line in f:
            if "=" in line and not line.lstrip().startswith("#"):
                k, v = line.split("=", 1)
                kv[k.strip()] = v.strip()
    if kv["kernel_source_sha256"] == bench.kernel_source_hash() and kv.get("sparse_momentum", "0") == "1":
        fs = float(kv["copy_bytes"]) / (float(kv["copy_fetch_kib"]) * 1024)
        ws = float(kv["copy_bytes"]) / (float(kv["copy_write_kib"]) * 1024)
        want = float(kv["fused_fetch_kib"]) * 1024 * fs + float(kv["fused_write_kib"]) * 1024 * ws
        assert t == pytest.approx(want)
    else:
        assert t is None
    # a summary taken on other sources is never used
    stale = tmp_path / "pmc.txt"
    stale.write_text(open(bench.PMC_SUMMARY).read().replace(kv["kernel_source_sha256"], "0" * 64))
    monkeypatch.setattr(bench, "PMC_SUMMARY", str(stale))
    assert bench.read_pmc_summary() is None


def test_survey_bytes_of_the_workloads():
    """The bench's headline fraction takes the dense byte definition: for
    the ResNet-50-sized step 5,322,405,504 B (12 K d + 16 d + 16 K k)."""
    import bench
    import synth
    wl = synth.workload("resnet50")
    assert bench.survey_bytes(wl, 25558, detach=False) == 5322405504
    rb = synth.workload("rbgs")
    d = 25557032
    assert bench.survey_bytes(rb, 63 * 4096, detach=False) == 12 * 8 * d + 16 * d + 8 * 8 * 63 * 4096
    assert bench.survey_bytes(rb, 63 * 4096, detach=True) == 12 * 8 * d + 16 * d + 8 * 8 * 63 * 4096 + 4 * 8 * d
    h = bench.host_cpu()
    assert h["nproc"] >= 1
