"""Host builds under sanitizers (CPU only):
  * the CPU oracle, every entry point on random small inputs with the edge
    cases of the tests, under AddressSanitizer and UndefinedBehaviorSanitizer;
  * the staging planner driven by a worker thread and a round thread under
    the library's locking protocol, under ThreadSanitizer and under
    AddressSanitizer + UndefinedBehaviorSanitizer.
Each program exits non-zero on the first report (or on a broken planner
invariant)."""
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2206_00470_amd", "csrc")


def build_and_run(tmp_path, compiler, src, flags, args=()):
    exe = str(tmp_path / "prog")
    subprocess.check_call([compiler, *flags, "-o", exe, os.path.join(HERE, src)])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               TSAN_OPTIONS="halt_on_error=1", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    res = subprocess.run([exe, *args], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "ERROR" not in res.stderr and "WARNING: ThreadSanitizer" not in res.stderr, res.stderr
    return res.stdout


def test_oracle_under_address_and_undefined_sanitizers(tmp_path):
    out = build_and_run(tmp_path, "gcc", "oracle_sanitize.c",
                        ["-std=c11", "-O1", "-g", "-ffp-contract=off", "-fsanitize=address,undefined",
                         "-fno-sanitize-recover=all", "-lm"])
    assert out.startswith("checksum")


@pytest.mark.parametrize("san", ["thread", "address,undefined"])
def test_staging_planner_threads_under_sanitizers(tmp_path, san):
    out = build_and_run(tmp_path, "g++", "planner_stress.cpp",
                        ["-std=c++20", "-O1", "-g", f"-fsanitize={san}", "-fno-sanitize-recover=all",
                         "-I", CSRC, "-pthread"], args=("300",))
    fields = dict(zip(out.split()[0::2], map(int, out.split()[1::2])))
    assert fields["bad"] == 0 and fields["staged"] > 0 and fields["evicted"] > 0, out
