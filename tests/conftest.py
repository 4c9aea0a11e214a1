import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through libad.so)")
    config.addinivalue_line("markers", "slow: large CPU oracle work")


@pytest.fixture(scope="session")
def tiny_cfg():
    from paper_2608_12703_amd.configs import Config
    return Config(name="unit_tiny", n_layers=2, d_model=128, n_heads=2, d_ffn=256, vocab=11,
                  dtype="bf16", batch=3, k=3, kv_max=20, geo_p=0.3, seed=7)
