"""Every planted mistake in tests/oracle_mutations.py must make its pin
module fail: the pins of the oracles (closed forms, invariants, library
routines, brute force) are checked against a wrong oracle, one mistake at a
time, each in its own pytest process.  CPU only."""
import concurrent.futures
import os
import subprocess
import sys

import pytest

from tests.oracle_mutations import MUTATIONS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_pins(name):
    pins = MUTATIONS[name][0]
    env = dict(os.environ, ORACLE_MUTATION=name, CUDA_VISIBLE_DEVICES="", HIP_VISIBLE_DEVICES="")
    r = subprocess.run([sys.executable, "-m", "pytest", pins, "-x", "-q", "-m", "not gpu", "-p", "no:cacheprovider",
                        "-p", "tests.oracle_mutations"], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=900)
    return r.returncode, (r.stdout + r.stderr)[-3000:]


@pytest.fixture(scope="module")
def outcomes():
    with concurrent.futures.ThreadPoolExecutor(max_workers=4) as ex:
        return dict(zip(MUTATIONS, ex.map(run_pins, MUTATIONS)))


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_fails_a_pin(name, outcomes):
    rc, log = outcomes[name]
    # 1: some pin failed (the mistake is caught); 0 would mean every pin
    # passed against the wrong oracle; anything else is a broken mutation
    assert rc == 1, f"{name}: pytest exit code {rc}\n{log}"
