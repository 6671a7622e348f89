"""The host tests again, against a build whose host C++ (stage.cpp in
dry-run mode, tstage.cpp, sched.cpp, partition.cpp) carries
AddressSanitizer and UndefinedBehaviorSanitizer (any report aborts the
process).  CPU only: the kernels of that build are the regular ones and are
never launched."""

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HOST_TESTS = ["test_abi_host.py", "test_schedule_host.py", "test_partition_host.py",
              "test_tuner_host.py", "test_tstage_host.py", "test_uvit_plan_host.py"]


def test_host_tests_under_asan_and_ubsan():
    sys.path.insert(0, ROOT)
    from paper_2606_19163_amd import build as B
    lib = B.build_asan()
    env = dict(os.environ)
    env.update({
        "PULSE_STAGE_LIB": lib,
        "LD_PRELOAD": B.asan_runtime(),
        # the interpreter itself is not instrumented; its arena is not a leak
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
        "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1",
        "HIP_VISIBLE_DEVICES": "",
    })
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
           *[os.path.join(ROOT, "tests", t) for t in HOST_TESTS]]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in tail and "runtime error" not in tail, tail
