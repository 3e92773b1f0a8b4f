import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the HIP library")


@pytest.fixture(scope="session")
def golden_maps():
    """Hand-written landmark maps: {(N, m, mode): int list}."""
    path = os.path.join(ROOT, "tests", "golden", "landmark_maps.txt")
    maps, key, rows = {}, None, []
    with open(path) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("map"):
                if key is not None:
                    maps[key] = rows
                _, N, m, mode = line.split()
                key, rows = (int(N), int(m), int(mode)), []
            else:
                rows.extend(int(x) for x in line.split())
    if key is not None:
        maps[key] = rows
    return maps
