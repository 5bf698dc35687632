"""Host-side logic of bench.py that needs no GPU."""
import subprocess
import sys
import os

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_counter_traffic_lookup():
    # no summary covers an unknown kernel class or workload
    assert bench.counter_traffic("no_such_class", "switch_base_8e") == (None, None, None)
    assert bench.counter_traffic("exit", "no_such_workload") == (None, None, None)
    # a covered class gives bytes, the summary's path and the kernel measured,
    # or nothing once the kernel source no longer matches the recorded hash
    val, src, kern = bench.counter_traffic("exit", "switch_base_8e")
    assert (val is None and src is None and kern is None) or \
        (val > 0 and src.startswith("profiles/") and kern.startswith("k_exit"))


def test_counter_traffic_blocks(tmp_path, monkeypatch):
    # several machine-readable blocks in one summary, each found by class;
    # a block whose source hash differs gives nothing
    import hashlib
    src = tmp_path / "k.hip"
    src.write_text("kernel source")
    sha = hashlib.sha256(src.read_bytes()).hexdigest()
    (tmp_path / "profiles").mkdir()
    (tmp_path / "profiles" / "w.md").write_text(
        "# summary\n\n```\nclass: exit\nkernel: k_exit_x\nworkload: w\n"
        "traffic_bytes_per_launch: 123\nsource: k.hip\nsource_sha256: " + sha + "\n```\n\n"
        "```\nclass: down\nkernel: k_down_x\nworkload: w\n"
        "traffic_bytes_per_launch: 456\nsource: k.hip\nsource_sha256: 00\n```\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.counter_traffic("exit", "w") == (123.0, "profiles/w.md", "k_exit_x")
    assert bench.counter_traffic("down", "w") == (None, None, None)
    assert bench.counter_traffic("up", "w") == (None, None, None)


def test_step_statistics():
    st = bench.step_stats([5.0, 1.0, 2.0, 4.0, 3.0])
    assert st["median"] == 3.0 and st["mean"] == 3.0
    assert st["min"] == 1.0 and st["max"] == 5.0
    assert 1.0 <= st["p10"] <= st["median"] <= st["p90"] <= 5.0


def test_host_cpu_description():
    h = bench.host_cpu()
    assert h["nproc"] == os.cpu_count() and h["nproc"] >= 1
    assert h["usable"] is None or 1 <= h["usable"] <= h["nproc"]


def test_kernel_names_follow_the_tile_selection():
    from synthgen import workload
    assert bench.class_kernel("up", workload("mixtral_8x7b_prefill")).startswith("k_ffn_big<0>")
    assert bench.class_kernel("down", workload("mixtral_8x7b_prefill")).startswith("k_ffn_big<2>")
    assert bench.class_kernel("exit", workload("qwen_moe_a2_7b")).startswith("k_exit_big")
    assert bench.class_kernel("exit", workload("switch_base_8e")).startswith("k_exit_mma")
    assert bench.class_kernel("up", workload("mixtral_8x7b_decode")).startswith("k_ffn_mma")
