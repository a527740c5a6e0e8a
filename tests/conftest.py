import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")
    # FPDE_TEST_LIBRARY=check: every test runs on the checking build (LDS filled
    # with NaN before each march, other tilings, chunk lengths and algorithms)
    # instead of the product library, so that the parity suite checks those
    # against the oracle too (the checking-build comparisons then compare it
    # with itself)
    if os.environ.get("FPDE_TEST_LIBRARY") == "check":
        from paper_2607_18020_amd import binding  # noqa: PLC0415
        if not os.path.exists(binding.CHECK_LIB_PATH):
            raise pytest.UsageError(f"{binding.CHECK_LIB_PATH} is not built")
        binding.LIB_PATH = binding.CHECK_LIB_PATH
        binding._lib = None


@pytest.fixture(scope="session")
def oracle_mod():
    import oracle  # noqa: PLC0415  (test infrastructure)
    oracle._load()
    return oracle
