"""The oracle's pins catch plausible mistakes: each mutation in
tests/oracle_mutations.py (a padding-style split, the remainder on the last
shards, minor-major axis order, column-major devices, shortest-first or
heaviest-sender balancing, the highest-index naive sender, destination cut
points dropped, no replica check, replicas counted once in the traffic) is
planted in a child process, and tests/test_oracle_pins.py must fail there.
CPU only."""

import os
import subprocess
import sys

import pytest

from tests.oracle_mutations import MUTATIONS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PINS = os.path.join(ROOT, "tests", "test_oracle_pins.py")


def _run_pins(mutation):
    env = dict(os.environ, RESHARD_ORACLE_MUTATION=mutation) if mutation else dict(os.environ)
    env.pop("PYTEST_XDIST_WORKER", None)
    return subprocess.run([sys.executable, "-m", "pytest", PINS, "-x", "-q", "-p", "no:cacheprovider",
                           "-p", "no:randomly", "-m", "not gpu"],
                          cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)


@pytest.mark.parametrize("mutation", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(mutation):
    r = _run_pins(mutation)
    # exit status 1: tests ran and at least one failed (2+ would be a broken run)
    assert r.returncode == 1, f"{mutation}: pins passed or the run broke ({r.returncode})\n{r.stdout[-3000:]}"
