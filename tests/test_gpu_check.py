"""GPU: the checking build and run-to-run determinism.

libfgq_check.so is the library compiled with -DFGQ_CHECK: every buffer load
is tested for the case the hardware's range check misses (an in-range
vector offset carried past the end by the scalar offset) and every output,
split-sum and code store against the extent it writes; failures are
suppressed and counted (fgq_check_violations).  A child process loads it
(FGQ_LIBRARY=check), runs the calls of tests/check_cases.py over every
kernel family on ragged and seeded random shapes, and must report no
violation and produce the same bytes as the normal library.  The normal
library then runs the same calls twice in this process: a race through LDS
or between workgroups would show as a difference between the runs.
"""
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

import check_cases

fgq = pytest.importorskip("paper_1705_01462_amd")

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_checking_build_reports_no_violation(tmp_path):
    lib = os.path.join(ROOT, "paper_1705_01462_amd", "libfgq_check.so")
    assert os.path.exists(lib), "libfgq_check.so not built (__graft_entry__.build())"
    env = dict(os.environ, FGQ_LIBRARY="check")
    print("[check] child process on libfgq_check.so", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "tests", "check_cases.py"), str(tmp_path)],
                       env=env, capture_output=True, text=True, timeout=600)
    print(r.stdout[-2000:], flush=True)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "libfgq_check.so" in r.stdout
    n, site, off = (int(v) for v in open(tmp_path / "violations.txt").read().split())
    assert n == 0, f"{n} out-of-bounds accesses, the first at site {site}, offset {off}"
    ref = check_cases.run_cases(fgq, torch)
    assert len(ref) > 100
    for k, v in ref.items():
        got = np.load(tmp_path / (k + ".npy"))
        assert got.dtype == v.dtype and got.shape == v.shape, k
        assert got.tobytes() == v.tobytes(), k


def test_repeated_runs_are_identical():
    a = check_cases.run_cases(fgq, torch)
    b = check_cases.run_cases(fgq, torch)
    assert a.keys() == b.keys()
    for k in a:
        assert a[k].tobytes() == b[k].tobytes(), k
