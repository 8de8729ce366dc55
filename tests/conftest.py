import sys
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parent.parent
if str(ROOT) not in sys.path:
    sys.path.insert(0, str(ROOT))


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU test (full-size oracle runs)")


@pytest.fixture(scope="session")
def oracle_mod():
    import oracle

    oracle._load()
    return oracle


def gpu_available() -> bool:
    try:
        import torch

        return torch.cuda.is_available()
    except Exception:  # pragma: no cover
        return False


@pytest.fixture(scope="session")
def fff_lib():
    """The HIP library through its Python binding; fails loudly if the GPU or library is missing."""
    if not gpu_available():
        pytest.fail("GPU test selected but no GPU is visible")
    import paper_2311_10770_amd as fff

    fff.load_library()
    return fff


def golden_path(name: str) -> Path:
    return ROOT / "tests" / "golden" / name


def read_table(name: str):
    rows = []
    for line in golden_path(name).read_text().splitlines():
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        rows.append(line.split())
    return rows


def flush_print(*a):
    """Name the case before a GPU step, so a crash still leaves it in the log."""
    print(*a, flush=True)
