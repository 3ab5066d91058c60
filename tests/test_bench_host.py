"""Host-side logic of bench.py (no GPU): the one-GPU guard and the gate
that reports counter-measured HBM traffic only for the kernel source the
counters were taken on."""
import hashlib
import importlib.util
import json
import os
import subprocess
import sys

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def load_bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(REPO, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(REPO, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_gate_follows_the_source_hash(tmp_path):
    bench = load_bench()
    src = tmp_path / "kernel.hip"
    src.write_bytes(b"// a kernel\n")
    (tmp_path / "profiles").mkdir()
    prof = {"source": "kernel.hip", "source_sha256": hashlib.sha256(src.read_bytes()).hexdigest(),
            "traffic_bytes_per_call": 123456}
    (tmp_path / "profiles" / "attn_fwd_window_s10920_h12_d128.json").write_text(json.dumps(prof))
    bench.REPO = str(tmp_path)
    assert bench.measured_traffic() == 123456
    src.write_bytes(b"// a kernel, changed\n")
    assert bench.measured_traffic() is None
    (tmp_path / "profiles" / "attn_fwd_window_s10920_h12_d128.json").write_text("{not json")
    assert bench.measured_traffic() is None


def test_committed_profile_was_taken_on_the_shipped_kernel_source():
    """profiles/attn_fwd_window_s10920_h12_d128.json carries the sha256 of the
    attention source its counters were taken on (written by a script from
    the file); after a change to that source the counters must be taken
    again before this passes."""
    prof = json.load(open(os.path.join(REPO, "profiles", "attn_fwd_window_s10920_h12_d128.json")))
    src = open(os.path.join(REPO, prof["source"]), "rb").read()
    assert hashlib.sha256(src).hexdigest() == prof["source_sha256"]
    assert prof["traffic_bytes_per_call"] > 0
