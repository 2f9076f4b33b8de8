import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: large CPU work (minutes)")


@pytest.fixture(scope="session")
def model_dir(tmp_path_factory):
    d = os.environ.get("JET_MODEL_CACHE")
    if d:
        os.makedirs(d, exist_ok=True)
        return d
    return str(tmp_path_factory.mktemp("models"))


def record_parity(name, **vals):
    """Append measured parity errors to $JET_PARITY_LOG (JSON lines), if set."""
    import json
    path = os.environ.get("JET_PARITY_LOG")
    if not path:
        return
    with open(path, "a") as f:
        f.write(json.dumps({"case": name, **{k: float(v) for k, v in vals.items()}}) + "\n")
