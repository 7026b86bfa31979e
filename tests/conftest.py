import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    # A planted oracle mistake (tests/oracle_mutations.py), applied before any test
    # module imports the oracle; only the mutation check sets this, in a subprocess.
    mutation = os.environ.get("ORACLE_MUTATION")
    if mutation:
        sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
        import oracle_mutations
        oracle_mutations.apply(mutation)
