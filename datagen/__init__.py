"""Seeded synthetic input generators shared by the tests, the bench and the
oracle harness.  Nothing here computes any part of the selective-transfer
method; it only draws inputs of the paper's workload shapes."""
from . import configs, inputs, rng  # noqa: F401
from .configs import CONFIGS, ORDER, Config, budget_k, extras_count, get  # noqa: F401
