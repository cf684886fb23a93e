"""CPU tests of bench.py's contract that need no GPU: the refusal of more than
one GPU, the options of the default run's other workloads, and the binding of
the stored posterior traffic figure to the kernel source it was measured on."""
import hashlib
import importlib.util
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_options_parse(monkeypatch):
    b = _bench()
    for argv in (["--only", "pass"], ["--no-secondary"], ["--only", "forest", "--kernel-loops", "5"]):
        monkeypatch.setattr(sys, "argv", ["bench.py"] + argv)
        b.parse()
    # every child command of the default run is a valid command line of its own
    for _, extra in b.SECONDARY:
        monkeypatch.setattr(sys, "argv", ["bench.py"] + extra)
        a = b.parse()
        assert a.gpus == 1


def test_stored_posterior_traffic_matches_the_kernel_source():
    """The roofline's traffic figure is reported only for the kernel source its
    counters were taken on; a change to the kernel without new counters would
    turn it into null, which this catches before a GPU run."""
    b = _bench()
    with open(os.path.join(ROOT, "paper_2408_04323_amd", "csrc", "k_posterior.hip"), "rb") as fh:
        digest = hashlib.sha1(fh.read()).hexdigest()
    assert digest == b.POSTERIOR_TRAFFIC["source_sha1"]
    assert set(b.POSTERIOR_TRAFFIC["bytes"]) == {"f32", "f64"}
