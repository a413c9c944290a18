"""Host-side checks of the benchmark's reporting (no GPU): the committed
HBM-counter summary of the fused step was taken on the current kernel source
(otherwise bench.py reports the traffic as unknown), the summaries name the
commands that produced them, and --gpus above 1 is refused with a message."""
import importlib.util
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
WORKLOAD = "stress_torusknot_12v_128x16_b8"


def load_bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_counter_summary_matches_kernel_source():
    bench = load_bench()
    traffic = bench.read_traffic(WORKLOAD)
    assert traffic is not None, ("profiles/fused_transport_reconstruct_*_counters.txt was taken on another kernel "
                                 "source: retake the FETCH_SIZE / WRITE_SIZE passes")
    algo = None
    for line in open(os.path.join(ROOT, "profiles", f"fused_transport_reconstruct_{WORKLOAD}_counters.txt")):
        if line.startswith("algorithmic_bytes_per_launch:"):
            algo = float(line.split(":")[1])
    assert algo and 0.95 <= traffic / algo <= 1.2


def test_summaries_name_their_commands():
    pdir = os.path.join(ROOT, "profiles")
    for name in os.listdir(pdir):
        text = open(os.path.join(pdir, name)).read()
        assert "rocprofv3" in text, name
        assert "bench.py" in text, name


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
