"""Stream ordering: the same step with every kernel launch serialised (a
child process with HIP_LAUNCH_BLOCKING=1 and AMD_SERIALIZE_KERNEL=3) gives
the same bits as the library run as deployed, whose chunks alternate
between the caller's stream and the handle's second one.  A missing
dependency between the streams, or between a call's kernels, would show as
a difference.  The child also prints the plan (MUON_HIP_LOG=1)."""
import json
import os
import subprocess
import sys

import pytest

from tests.gpu_util import require_gpu

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_serialised_launches_give_the_same_bits():
    require_gpu()
    from tests.gpu_child_step import run
    want = run()
    env = dict(os.environ, HIP_LAUNCH_BLOCKING="1", AMD_SERIALIZE_KERNEL="3", MUON_HIP_LOG="1")
    print("[child] serialised step", flush=True)
    p = subprocess.run([sys.executable, "-m", "tests.gpu_child_step"], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=240)
    assert p.returncode == 0, p.stderr[-3000:]
    got = json.loads(p.stdout.strip().splitlines()[-1])
    plan = [l for l in p.stderr.splitlines() if l.startswith("muon:")]
    print("\n".join(plan), flush=True)
    assert got == want
    assert "two streams" in plan[0] and sum("second stream" in l for l in plan) >= 1
