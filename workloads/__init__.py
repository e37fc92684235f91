"""Seeded synthetic workloads shared by the tests, the benchmark and the oracle's checks."""
from .synth import *  # noqa: F401,F403
from .synth import CONFIGS, ALIASES, LayerConfig, LayerWeights, Requests  # noqa: F401
