"""The stage on CU-masked streams (dispatch, expert FFN and combine on
disjoint CU partitions), checked against the oracle and bit for bit against
the null stream.  Masked streams need hardware queues of their own, which
the streams of earlier tests in this process have taken, so the check runs in
a fresh child process (tests/cu_masked_child.py)."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))


def test_stage_on_cu_masked_streams():
    r = subprocess.run([sys.executable, "-u", os.path.join(HERE, "cu_masked_child.py")],
                       capture_output=True, text=True, timeout=240)
    print(r.stdout[-3000:], flush=True)
    assert r.returncode == 0, r.stderr[-3000:]
    assert "CU-MASKED OK" in r.stdout
