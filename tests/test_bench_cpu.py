"""Host-side checks of the benchmark: the algorithmic byte counts behind its roofline figures, the
one-GPU guard, and the source hashes that decide whether a committed traffic record applies."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2609_30738_amd import workloads  # noqa: E402


def test_algorithmic_bytes_of_the_benchmark_workload():
    wl = workloads.mistral_pass_32k()
    ab = bench.algorithmic_bytes(wl)
    units = 32 * 8  # layers x kv heads
    L, d, e, G, W, B = 32768, 128, 2, 4, 32, 64
    # pass 1: K once, the unit's queries once, (max, sum) per window row of every head
    pass1 = units * (L * d * e + G * W * d * e + G * W * 8)
    # pass 2: the same reads plus mu and sigma of every key
    pass2 = pass1 + units * L * 8
    assert ab["stats_pass"] == pass1 == 2_156_134_400
    assert ab["mu_sigma_pass"] == pass2 == 2_223_243_264
    kept = units * 2 * 2 * (B + W) * d * e  # K and V rows kept, read and written
    assert ab["total"] == units * (L * d * e + G * W * d * e) + kept + units * B * 4
    assert ab["scoring"] == units * (L * d * e + G * W * d * e) == 2_155_872_256
    assert bench.mfma_flops(wl) == 2.0 * 32 * L * 32 * W * d


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 2 and "one GPU" in line["error"]


@pytest.mark.parametrize("kernel", sorted(bench.KERNEL_SOURCES))
def test_traffic_record_is_keyed_to_the_kernel_sources(kernel, tmp_path, monkeypatch):
    sha = bench.source_sha(kernel)
    assert len(sha) == 16
    # a record taken on other sources is ignored; one taken on these is used
    prof = tmp_path / "profiles"
    prof.mkdir()
    path = prof / f"{kernel}_wl_traffic.json"
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "source_sha", lambda k: sha)
    path.write_text(json.dumps({"source_sha": "0" * 16, "hbm_bytes_per_launch": 5}))
    assert bench.measured_traffic(kernel, "wl") is None
    path.write_text(json.dumps({"source_sha": sha, "hbm_bytes_per_launch": 5}))
    assert bench.measured_traffic(kernel, "wl") == 5


def test_committed_traffic_records_name_their_kernel():
    for kernel in bench.KERNEL_SOURCES:
        path = os.path.join(ROOT, "profiles", f"{kernel}_mistral32_L32768_W32_B64_traffic.json")
        if not os.path.exists(path):
            continue
        with open(path) as f:
            rec = json.load(f)
        assert rec["kernel"].startswith(kernel)
        assert rec["source_files"] == list(bench.KERNEL_SOURCES[kernel])
        # the one launch of the whole pass moves what the pass must move; a scoring kernel, K and
        # Q_W once
        ab = bench.algorithmic_bytes(workloads.mistral_pass_32k())
        assert rec["algorithmic_bytes_per_launch"] == ab[
            "total" if kernel == "window_prune" else "scoring"]


def test_source_hash_ignores_comments_only():
    code = bench._code_only('int a; // note\n/* block\n note */ int b;\nconst char* s = "a // b";\n\n')
    assert code == 'int a;\n int b;\nconst char* s = "a // b";'
    assert bench._code_only("x = 1;  // one\n") == bench._code_only("// header\nx = 1;\n")
    assert bench._code_only("x = 1;\n") != bench._code_only("x = 2;\n")
