import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


# A planted oracle mistake (tests/oracle_mutants.py), for the runs that check
# that the oracle's pins catch it; never set in ordinary runs.
if os.environ.get("ORACLE_MUTANT"):
    import oracle_mutants
    oracle_mutants.install(os.environ["ORACLE_MUTANT"])


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the HIP library)")
    config.addinivalue_line("markers", "slow: full-size workload (minutes of CPU time)")


@pytest.fixture(scope="session")
def golden():
    import json

    def load(name):
        with open(os.path.join(ROOT, "tests", "golden", name)) as f:
            return json.load(f)
    return load
