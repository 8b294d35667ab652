import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


@pytest.fixture(scope="session", autouse=True)
def library_built_from_sources(request):
    """Before any GPU test runs, load the verifier library; loading refuses a
    library whose embedded source hash differs from the sources beside it."""
    if any(item.get_closest_marker("gpu") for item in request.session.items):
        import paper_2608_03447_amd as asd
        asd._load()
