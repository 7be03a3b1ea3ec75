"""Wavefront-timing independence of the replay (race detection).

The race-detection build delays each wavefront by a pseudo-random amount
after every workgroup barrier, so that the wavefronts of an instance reach
each stretch of code between two barriers in shifted order.  Every result
must still equal the oracle's.  The build runs in a child process (a
process loads one build of the library)."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.timeout(600)
def test_replay_results_independent_of_wavefront_timing():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "jitter_child.py"), ROOT],
                       capture_output=True, text=True, timeout=540)
    assert r.returncode == 0, r.stderr[-4000:]
    done = json.loads(r.stdout.strip().splitlines()[-1])
    assert done["step_boundary"] == 3 * done["step_boundary_dense"] > 0
    assert done["random"] > 0 and done["chat_full_length"] == 15 and done["many_groups"] > 0
    assert all(done[n] > 0 for n in ("selector512x8", "selector4096x32", "attack_onetouch", "attack_lowslow",
                                     "attack_replay", "tiers"))
