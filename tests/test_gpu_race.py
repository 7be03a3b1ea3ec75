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


# The child takes 15-25 s on an MI355X; a run that has not finished well
# after that is ended and reported with the child's progress lines, which
# name the batch it was replaying.
CHILD_TIMEOUT_S = 150


@pytest.mark.timeout(CHILD_TIMEOUT_S + 60)
def test_replay_results_independent_of_wavefront_timing():
    try:
        r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "jitter_child.py"), ROOT],
                           capture_output=True, text=True, timeout=CHILD_TIMEOUT_S)
    except subprocess.TimeoutExpired as e:
        err = e.stderr.decode() if isinstance(e.stderr, bytes) else (e.stderr or "")
        pytest.fail(f"race-detection replay did not finish in {CHILD_TIMEOUT_S} s; its progress:\n{err[-3000:]}")
    assert r.returncode == 0, r.stderr[-4000:]
    done = json.loads(r.stdout.strip().splitlines()[-1])
    assert done["step_boundary"] == 3 * done["step_boundary_dense"] > 0
    assert done["random"] > 0 and done["chat_full_length"] == 15 and done["many_groups"] > 0
    assert all(done[n] > 0 for n in ("selector512x8", "selector4096x32", "attack_onetouch", "attack_lowslow",
                                     "attack_replay", "tiers"))
