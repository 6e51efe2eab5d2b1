"""Every planted oracle mistake must make at least one pin fail (CPU only).

The pins are the oracle suites; each mutation runs them in a fresh process with
ORACLE_MUTATION set, and that process must report a failure."""

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

from tests.oracle_mutations import MUTATIONS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PIN_SUITES = ["tests/test_oracle_primitives.py", "tests/test_oracle_model.py",
              "tests/test_oracle_golden.py", "tests/test_oracle_sampling.py", "tests/test_oracle_draft.py"]


def _run(name):
    env = dict(os.environ, ORACLE_MUTATION=name, OMP_NUM_THREADS="1", OPENBLAS_NUM_THREADS="1")
    p = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:randomly", *PIN_SUITES],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return name, p.returncode, p.stdout[-2000:]


@pytest.fixture(scope="module")
def mutation_results():
    workers = max(1, min(8, (os.cpu_count() or 2)))
    with ThreadPoolExecutor(workers) as ex:
        return {n: (rc, out) for n, rc, out in ex.map(_run, sorted(MUTATIONS))}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(mutation_results, name):
    rc, out = mutation_results[name]
    assert rc == 1, f"mutation {name} survived the pins (rc={rc}):\n{out}"
