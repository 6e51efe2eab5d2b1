import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size model shapes; minutes of host work")


# A planted oracle mistake, applied only when a mutation run asks for it
# (see tests/test_oracle_mutations.py); never set in normal runs.
if os.environ.get("ORACLE_MUTATION"):
    from tests import oracle_mutations as _om

    _om.apply(os.environ["ORACLE_MUTATION"])
