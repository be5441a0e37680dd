"""The oracles' pins catch plausible mistakes: each mutation in
tests/oracle_mutations.py is planted in a child process, which runs the pin
tests of that oracle (tests/test_oracle_pins.py, or the pin tests of
tests/test_schedule.py and tests/test_pipeline.py -- not their checks of
the library, which are no pins); they must fail there.  Resharding:
a multi-axis spec token kept to its first axis or read in reverse, a
padding-style split, the remainder on the last shards, minor-major axis
order, column-major devices, shortest-first or heaviest-sender balancing,
the highest-index naive sender, destination cut points dropped, no replica
check, replicas counted once in the traffic, a permuted buffer laid out
with the inverse permutation.  Scheduling: tasks that wait
for their sender host only or for every earlier task, a lower bound
charging every candidate, shortest-first balancing, the randomized search
left out or cut to one random order per iteration, DFS stopped at its first
complete schedule.  Pipeline: one warm-up forward too many, eagerness ignored.
CPU only."""

import concurrent.futures
import os
import subprocess
import sys

import pytest

from tests.oracle_mutations import MUTATIONS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run_pins(mutation):
    pin_file, select = MUTATIONS[mutation][3]
    env = dict(os.environ, RESHARD_ORACLE_MUTATION=mutation)
    env.pop("PYTEST_XDIST_WORKER", None)
    cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", pin_file), "-x", "-q",
           "-p", "no:cacheprovider", "-m", "not gpu"]
    if select:
        cmd += ["-k", select]
    return subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)


@pytest.fixture(scope="module")
def outcomes():
    """Every mutation's child run, four at a time."""
    with concurrent.futures.ThreadPoolExecutor(max_workers=4) as pool:
        return dict(zip(sorted(MUTATIONS), pool.map(_run_pins, sorted(MUTATIONS))))


@pytest.mark.parametrize("mutation", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(mutation, outcomes):
    r = outcomes[mutation]
    # exit status 1: tests ran and at least one failed (2+ would be a broken run)
    assert r.returncode == 1, f"{mutation}: pins passed or the run broke ({r.returncode})\n{r.stdout[-3000:]}"
