"""The oracle's pins fail under every planted mistake (tests/oracle_mutations.py).

For each mutation the oracle pin tests run in a subprocess with the mistake
applied; the run must fail (a test assertion, or an error the mistake causes).
A mutation that no pin catches names a gap in the pins."""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

from oracle_mutations import MUTATIONS

HERE = os.path.dirname(os.path.abspath(__file__))
PINS = sorted(os.path.join(HERE, f) for f in os.listdir(HERE) if f.startswith("test_oracle_") and f.endswith(".py")
              and f != "test_oracle_mutations.py")


def run_pins(mutation):
    env = dict(os.environ, ORACLE_MUTATION=mutation, OMP_NUM_THREADS="2", OPENBLAS_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *PINS],
                       cwd=os.path.dirname(HERE), env=env, capture_output=True, text=True, timeout=300)
    return r.returncode, r.stdout[-2000:]


@pytest.fixture(scope="module")
def outcomes():
    with ThreadPoolExecutor(max_workers=4) as pool:
        return dict(zip(MUTATIONS, pool.map(run_pins, MUTATIONS)))


def test_pins_pass_without_a_mutation():
    rc, out = run_pins("")
    assert rc == 0, out


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_mutation(name, outcomes):
    rc, out = outcomes[name]
    assert rc == 1, "%s (%s) is not caught by any pin (exit %d):\n%s" % (name, MUTATIONS[name][4], rc, out)
