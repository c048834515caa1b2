import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def _parse_fraction(tok: str):
    from fractions import Fraction

    return Fraction(tok)


def load_golden(name: str) -> dict:
    """Parse a tests/golden fixture: 'key v1 v2 ...' lines, '#' comments.

    Repeated keys whose first value is an integer step index are collected as
    {key: {step: [values]}}; other keys map to their value list.
    """
    path = os.path.join(ROOT, "tests", "golden", name)
    out: dict = {}
    with open(path) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, *vals = line.split()
            out.setdefault(key, []).append([_parse_fraction(v) for v in vals])
    return out


@pytest.fixture
def golden():
    return load_golden


def pytest_collection_modifyitems(config, items):
    try:
        import torch

        has_gpu = torch.cuda.is_available()
    except Exception:  # pragma: no cover
        has_gpu = False
    if has_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)
