"""The host planner (Sec. 3.3 DP / Algorithm 1, Sec. 3.4 batch split and
joint plan), the Eq. 9 cost model and the C oracle, built for the CPU with
AddressSanitizer + UndefinedBehaviorSanitizer and, separately, with
ThreadSanitizer (the DP solves thresholds on several threads), then driven by
tests/native/sanitize_driver.cpp on seeded tables: the DP equals the oracle's
DP on every table, error paths, the batch split, the joint plan, the exact
recovery of a linear overhead model (also through tp_profile_cost_model with a
synthetic profiler), and the oracle's slicing invariance.  Any sanitizer
report aborts the driver and fails the test.

CPU only: the GPU library is not involved (gcc/g++ builds of the host sources).
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2102_07988_amd", "csrc")
SANITIZERS = {
    "address_undefined": ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                          "-fno-omit-frame-pointer"],
    "thread": ["-fsanitize=thread"],
}


@pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None,
                    reason="needs gcc and g++")
@pytest.mark.parametrize("kind", sorted(SANITIZERS))
def test_host_code_under_sanitizers(kind, tmp_path):
    flags = SANITIZERS[kind] + ["-g", "-O1"]
    objs = []
    for src, cc in ((os.path.join(CSRC, "planner.cpp"), ["g++", "-std=c++17"]),
                    (os.path.join(CSRC, "costmodel.cpp"), ["g++", "-std=c++17"]),
                    (os.path.join(ROOT, "oracle", "tp_oracle.c"), ["gcc", "-ffp-contract=off"]),
                    (os.path.join(ROOT, "tests", "native", "sanitize_driver.cpp"),
                     ["g++", "-std=c++17"])):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        subprocess.run(cc + flags + ["-c", src, "-o", obj], check=True, capture_output=True)
        objs.append(obj)
    exe = str(tmp_path / "driver")
    subprocess.run(["g++"] + flags + ["-o", exe] + objs + ["-lpthread", "-lm"], check=True,
                   capture_output=True)
    env = dict(os.environ)
    env.pop("LD_PRELOAD", None)
    env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["TSAN_OPTIONS"] = "halt_on_error=1"
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, f"driver failed ({kind}):\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"
    assert "OK (0 failures)" in r.stdout
