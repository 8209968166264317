import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: large-model case (minutes of CPU oracle work)")


_WEIGHTS = {}


def weights_for(name):
    """Session cache of generated weights (generation of the 1.5B shape takes seconds)."""
    import synth
    if name not in _WEIGHTS:
        _WEIGHTS[name] = synth.generate_weights(synth.get_config(name))
    return _WEIGHTS[name]
