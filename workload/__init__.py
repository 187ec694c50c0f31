"""Seeded synthetic inputs shared by the oracle and the GPU path (no method arithmetic)."""
from .configs import CONFIGS, Config, tiny  # noqa: F401
from .generate import Workload, build_tree, keyed_rng, setup_ops  # noqa: F401
