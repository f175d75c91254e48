"""Host-side behaviour of bench.py (no GPU): the single-GPU guard, the traffic figure read from a
rocprofv3 counter summary (dropped once the kernel source differs from the one the counters were
taken on), and the overlap sweep's merge of its two contexts."""
import hashlib
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=60)
    assert r.returncode != 0
    assert "one GPU" in r.stderr and r.stdout == ""


def _summary(path, sha, fetch_kib=1000.0, write_kib=100.0, ff=0.5, wf=1.0):
    with open(path, "w") as f:
        f.write("# counters\n")
        f.write(f"kernels_source_sha256: {sha}\n")
        f.write(f"fetch_kib_per_dispatch: {fetch_kib}\nwrite_kib_per_dispatch: {write_kib}\n")
        f.write(f"fetch_copy_factor: {ff}\nwrite_copy_factor: {wf}\n")


def test_traffic_from_counter_summary(tmp_path, monkeypatch):
    import bench
    src_dir = tmp_path / "paper_2608_22704_amd" / "csrc"
    src_dir.mkdir(parents=True)
    (tmp_path / "profiles").mkdir()
    src = src_dir / "wnw_kernels.hip"
    src.write_bytes(b"kernel source v1\n")
    sha = hashlib.sha256(src.read_bytes()).hexdigest()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    path = tmp_path / "profiles" / "attention_w_pmc.txt"
    # each counter scaled by what it reads for a copy of known size: fetch 1000 KiB at factor 0.5
    # is 2000 KiB of HBM reads, write 100 KiB at factor 1 is 100 KiB
    _summary(path, sha)
    assert bench.measured_traffic("attention", "w") == (2000 + 100) * 1024
    # no summary for another workload
    assert bench.measured_traffic("attention", "other") is None
    # the kernel source changed since the counters were taken
    src.write_bytes(b"kernel source v2\n")
    assert bench.measured_traffic("attention", "w") is None
    # a summary missing a field
    src.write_bytes(b"kernel source v1\n")
    path.write_text(f"kernels_source_sha256: {sha}\nfetch_kib_per_dispatch: 1\n")
    assert bench.measured_traffic("attention", "w") is None


def test_merge_sweep_takes_steps_from_the_plain_context_and_recall_from_the_timed_one():
    import bench
    plain = [{"new_per_step": 1, "ms_per_step": 0.15, "copied_per_step": 0.25, "revived_per_step": 0.75, "recall_ms": None},
             {"new_per_step": 4, "ms_per_step": 0.20, "copied_per_step": 2.0, "revived_per_step": 2.0, "recall_ms": None}]
    timed = [{"new_per_step": 1, "ms_per_step": 0.16, "copied_per_step": 0.25, "revived_per_step": 0.75, "recall_ms": 0.05},
             {"new_per_step": 4, "ms_per_step": 0.21, "copied_per_step": 2.0, "revived_per_step": 2.0, "recall_ms": 0.12}]
    out = bench.merge_sweep(plain, timed, 0.145)
    assert [r["new_per_step"] for r in out] == [1, 4]
    assert abs(out[0]["steps_per_s"] - 1e3 / 0.15) < 1e-9 and out[0]["ms_per_step"] == 0.15
    assert out[0]["recall_ms"] == 0.05 and out[1]["recall_ms"] == 0.12
    # overlap = 1 - (T_step - T_no_recall) / T_recall, clamped to [0, 1]
    assert abs(out[0]["overlap"] - (1 - (0.15 - 0.145) / 0.05)) < 1e-12
    assert abs(out[1]["overlap"] - (1 - (0.20 - 0.145) / 0.12)) < 1e-12
    # without the timed context there is no recall time and no overlap
    bare = bench.merge_sweep(plain, [], 0.145)
    assert all(r["recall_ms"] is None and r["overlap"] is None for r in bare)
    assert bench.merge_sweep(plain, [dict(timed[0], recall_ms=0.001)], 0.145)[0]["overlap"] == 0.0
