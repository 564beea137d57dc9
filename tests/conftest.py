import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: CPU test that takes > 30 s")


@pytest.fixture(scope="session")
def hf():
    """transformers' Llama, used as an independent library implementation of
    the decoder the paper's target and drafter layers follow."""
    import transformers  # noqa: F401
    from transformers import LlamaConfig, LlamaForCausalLM
    return LlamaConfig, LlamaForCausalLM
