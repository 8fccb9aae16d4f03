"""The non-default kernel forms behind the comparison switches, against the
oracle. The library reads a switch once per process, so each case runs
tests/switch_check.py in one child process with the switch set."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("switch,value,kind", [
    ("WDC_GEMM_VARIANT", "2", "gemm"),   # 16 waves of 64 x 64
    ("WDC_GEMM_VARIANT", "0", "gemm"),   # 4 waves of 128 x 128
    ("WDC_ATTN_VARIANT", "4", "attn"),   # two-phase reference-max kernel at hd 64 and 128
])
def test_switch_matches_oracle(switch, value, kind):
    env = dict(os.environ, **{switch: value})
    r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "switch_check.py"), kind], env=env,
                       cwd=ROOT, capture_output=True, text=True, timeout=240)
    print(r.stdout[-2000:], r.stderr[-2000:])
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
