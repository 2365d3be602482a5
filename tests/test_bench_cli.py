"""CPU tests of the benchmark's contract that need no GPU: it measures one GPU
only and says so for more; a traffic record counts only for the kernel source
it was taken on."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_exits_with_a_message():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr


def test_traffic_record_of_another_source_is_ignored(tmp_path):
    import bench
    rec = tmp_path / "rec.txt"
    rec.write_text("kernel_source_sha256_16 = 0000000000000000\nhbm_bytes_per_launch = 123\n")
    assert bench.traffic_for_current_kernel(str(rec)) is None
    rec.write_text(f"kernel_source_sha256_16 = {bench.kernel_source_hash()}\nhbm_bytes_per_launch = 123\n")
    assert bench.traffic_for_current_kernel(str(rec)) == 123
