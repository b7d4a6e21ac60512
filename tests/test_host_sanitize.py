"""The host half of the library (planner, flow export, traffic, model, lower
bounds, timeline) run under AddressSanitizer and UndefinedBehaviorSanitizer
over one-GPU and several-GPUs-per-server profiles and the error paths
(tests/host_sanitize.cpp, built by the package build with g++)."""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BIN = os.path.join(ROOT, "tests", "host_sanitize")


def test_host_code_under_sanitizers():
    assert os.path.exists(BIN), "tests/host_sanitize is not built: run the package build"
    # verify_asan_link_order=0: a preloaded library must not stop the run
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([BIN], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "host_sanitize: ok" in r.stdout
