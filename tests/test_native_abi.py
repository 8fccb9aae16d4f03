"""The C ABI from a C99 client, with AddressSanitizer and UndefinedBehaviorSanitizer
on the library's host code (and LeakSanitizer on the CPU run) (tests/native: abi_driver.c and the
sanitizer build of the library, made by tests/native/build_native.py, which
__graft_entry__.build() runs). CPU: descriptor, weight-table and error
handling, no HIP call. GPU: rollouts in every mode, the step calls including
the allocation-free candidate call, batched calls and the kernel entry points
of a small model."""
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
DRIVER = os.path.join(HERE, "native", "_out", "abi_driver")


def _run(mode, timeout):
    assert os.path.exists(DRIVER), f"{DRIVER} missing: run tests/native/build_native.py (or __graft_entry__.build())"
    env = dict(os.environ)
    # leak checking on the CPU run only: once a device is in use, the HIP
    # runtime keeps allocations until the process exits
    env["ASAN_OPTIONS"] = f"detect_leaks={int(mode == 'cpu')}:halt_on_error=1:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([DRIVER, mode], capture_output=True, text=True, timeout=timeout, env=env)
    out = r.stdout + r.stderr
    print(out[-4000:])
    assert r.returncode == 0, f"abi_driver {mode} exited with {r.returncode}"
    for marker in ("AddressSanitizer", "LeakSanitizer", "runtime error:"):
        assert marker not in out, marker
    assert f"abi_driver {mode}: ok" in out


def test_c_abi_host_code_under_sanitizers_cpu():
    _run("cpu", 120)


@pytest.mark.gpu
def test_c_abi_host_code_under_sanitizers_gpu():
    _run("gpu", 240)
