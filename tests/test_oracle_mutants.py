"""The oracle's pins catch plausible mistakes: each planted mistake of
tests/oracle_mutants.py (a boundary off by one, a sign, a dropped term, an
operand from the wrong vector, a comparison that is not strict, a summation
order) is installed in a separate pytest process, and some pin of the
oracle function it touches must then fail on an assertion."""
import os
import re
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

import oracle_mutants as OM

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NAMES = sorted(OM.MUTANTS)


def _run(name):
    group = OM.MUTANTS[name][0]
    env = dict(os.environ, ORACLE_MUTANT=name, OMP_NUM_THREADS="1")
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           "-m", "not gpu", *OM.PIN_FILES[group]],
                          cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)


@pytest.fixture(scope="module")
def runs():
    with ThreadPoolExecutor(max_workers=min(6, os.cpu_count() or 1)) as ex:
        return dict(zip(NAMES, ex.map(_run, NAMES)))


@pytest.mark.parametrize("name", NAMES)
def test_pins_catch_planted_mistake(runs, name):
    r = runs[name]
    out = r.stdout + r.stderr
    assert r.returncode == 1, "mutant %s survived (exit %d):\n%s" % (name, r.returncode, out[-2000:])
    # killed by an assertion of a pin, not by an error in the mutant itself
    assert re.search(r"^E\s+(AssertionError|assert |Failed)", out, re.M), out[-3000:]
