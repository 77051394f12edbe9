"""The bounds-checked build (libattuner_checked.so): the GPU parity cases of
tests/_checked_run.py rerun through it with no violation reported, and
block-table entries corrupted on purpose (a page id past the pool, rows past
the cache plane, in the gather and in the attention launch's page copy) are
reported and skipped.  The cases run in a process of their own, started with
ATTUNER_LIB_VARIANT=checked so every binding call goes to the checked
library."""

import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.timeout(600)
def test_checked_build_parity_and_planted_entries():
    env = dict(os.environ, ATTUNER_LIB_VARIANT="checked")
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "tests", "_checked_run.py")], cwd=ROOT, env=env,
                       stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=540)
    print(r.stdout[-6000:], flush=True)
    assert r.returncode == 0, f"checked build run failed (exit {r.returncode})"
    assert "[done]" in r.stdout
