"""Seeded synthetic rollouts shared by the tests, the smoke check and the benchmark."""
from .rollouts import CONFIGS, Config, Structure, make_structure, make_batch, make_fused_batch  # noqa: F401
