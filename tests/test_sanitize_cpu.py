"""The host-side queue and continuous-batching engine under AddressSanitizer
and UndefinedBehaviorSanitizer: queue.cpp and serve.cpp are compiled with
g++ -fsanitize=address,undefined together with a stress driver
(tests/sanitize_serve.cpp) that runs random workloads under every policy,
the dynamic rule, deferred first tokens and pool pressure, checking the
schedule's invariants; any sanitizer report fails the run."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2603_11273_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_queue_and_serve_under_asan_ubsan():
    with tempfile.TemporaryDirectory() as tmp:
        exe = os.path.join(tmp, "serve_stress")
        cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
               "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
               os.path.join(ROOT, "tests", "sanitize_serve.cpp"),
               os.path.join(CSRC, "queue.cpp"), os.path.join(CSRC, "serve.cpp"), "-o", exe]
        r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
        assert r.returncode == 0, r.stdout
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
                   UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
        r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                           env=env, timeout=300)
        print(r.stdout[-2000:])
        assert r.returncode == 0, r.stdout[-4000:]
        assert "sanitized queue/serve stress: ok" in r.stdout
