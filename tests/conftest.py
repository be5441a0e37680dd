import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: CPU test that takes more than a few seconds")


@pytest.fixture(scope="session")
def gpu_lib():
    """The built HIP library on a machine with a GPU; errors loudly when either is missing."""
    import torch

    if not torch.cuda.is_available():
        pytest.fail("GPU test collected on a machine without a GPU; run with -m 'not gpu'")
    from paper_2211_05322_amd import binding

    return binding.load()


# A planted oracle mistake for tests/test_oracle_mutations.py, which runs the
# pin tests in a child process with this variable set; never set otherwise.
_MUTATION = os.environ.get("RESHARD_ORACLE_MUTATION")
if _MUTATION:
    from tests import oracle_mutations

    oracle_mutations.apply(_MUTATION)
