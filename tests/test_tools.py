"""Host-side tools, on the CPU: the profile summaries' source hash (comments do
not count, code does), the counter traffic that bench.py reports only while a
summary matches the current kernel source, and bench.py's refusal of more
than one GPU."""
import os
import subprocess
import sys

from paper_2609_30656_amd import profiling

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_code_only_ignores_comments_and_blank_lines():
    a = "int f(int x) {\n  return x + 1;  // add one\n}\n"
    b = "/* a block\n   comment */\nint f(int x) {\n\n  return x + 1;\n}  // trailing\n"
    assert profiling._code_only(a) == profiling._code_only(b)
    assert profiling._code_only(a) != profiling._code_only(a.replace("+ 1", "+ 2"))


def test_source_hash_follows_code_not_comments(tmp_path, monkeypatch):
    for f in ("eb_device.h", "eb_forward.hip"):
        (tmp_path / f).write_text(open(os.path.join(profiling.CSRC, f)).read())
    monkeypatch.setattr(profiling, "CSRC", str(tmp_path))
    h0 = profiling.kernel_source_hash("forward")
    assert h0 == profiling.kernel_source_hash("forward")
    src = tmp_path / "eb_forward.hip"
    src.write_text(src.read_text() + "\n// a note\n/* another */\n")
    assert profiling.kernel_source_hash("forward") == h0
    src.write_text(src.read_text() + "\nstatic int eb_extra_symbol;\n")
    assert profiling.kernel_source_hash("forward") != h0


def test_counter_traffic_only_for_the_current_source(tmp_path, monkeypatch):
    monkeypatch.setattr(profiling, "PROFILES", str(tmp_path))
    assert profiling.counter_traffic("c2", "zipf", "forward") is None  # no summary
    path = profiling.summary_path("forward", "c2", "zipf", "pmc")
    current = profiling.kernel_source_hash("forward")
    with open(path, "w") as f:
        f.write("# header = ignored\n")
        f.write(f"kernel_source_sha256_16 = {current}\n")
        f.write("hbm_bytes_per_launch = 123456   (scaled)\n")
    assert profiling.counter_traffic("c2", "zipf", "forward") == 123456.0
    with open(path, "w") as f:
        f.write("kernel_source_sha256_16 = 0000000000000000\n")
        f.write("hbm_bytes_per_launch = 123456\n")
    assert profiling.counter_traffic("c2", "zipf", "forward") is None  # taken on other code


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""
