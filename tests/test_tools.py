"""Host-side tools, on the CPU: the profile summaries' source hash (comments do
not count, code does), the counter traffic that bench.py reports only while a
summary matches the current kernel source, that every committed summary does,
and bench.py's refusal of more than one GPU."""
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


def test_counter_calibration_uses_the_last_copies(tmp_path):
    # set-up copies (c5 builds its tables by copies) come before the lookup;
    # only the run's last three copies, the 1 GiB calibration, scale the counters
    path = tmp_path / "pmc_counter_collection.csv"
    rows = []
    d = 0

    def add(kernel, value):
        nonlocal d
        d += 1
        rows.append(f'{d},{d},"Agent 1",1,1,1,64,1,"{kernel}",256,0,0,8,0,16,"FETCH_SIZE",{value},0,1')

    for _ in range(64):
        add("__amd_rocclr_copyBuffer", 390000.0)  # table set-up
    for _ in range(5):
        add("void eb::(anonymous namespace)::eb_pool_kernel<2, 3, false, false>(eb::FwdArgs)", 1000.0)
    for _ in range(3):
        add("__amd_rocclr_copyBuffer", 524288.0)  # calibration
    header = ('"Correlation_Id","Dispatch_Id","Agent_Id","Queue_Id","Process_Id","Thread_Id","Grid_Size",'
              '"Kernel_Id","Kernel_Name","Workgroup_Size","LDS_Block_Size","Scratch_Size","VGPR_Count",'
              '"Accum_VGPR_Count","SGPR_Count","Counter_Name","Counter_Value","Start_Timestamp","End_Timestamp"')
    path.write_text(header + "\n" + "\n".join(rows) + "\n")
    acc = profiling.read_counters(str(path), "eb_pool_kernel")
    assert acc["FETCH_SIZE"] == [1000.0] * 5
    assert acc["copy:FETCH_SIZE"] == [524288.0] * 3


def test_committed_summaries_match_the_current_sources():
    # every summary under profiles/ that names a kernel source hash was taken
    # on the kernel as it is now: a kernel change without new summaries fails
    checked, stale = 0, []
    for name in sorted(os.listdir(profiling.PROFILES)):
        path = os.path.join(profiling.PROFILES, name)
        with open(path) as f:
            hashes = [ln.split("=", 1)[1].split()[0] for ln in f if ln.startswith("kernel_source_sha256_16")]
        if not hashes:
            continue
        modes = [m for m, (k, _) in profiling.KERNELS.items() if name.startswith(k + "_")]
        assert len(modes) == 1, name
        checked += 1
        if hashes[0] != profiling.kernel_source_hash(modes[0]):
            stale.append(name)
    assert checked > 0
    assert not stale, f"summaries taken on other kernel code: {stale}"
