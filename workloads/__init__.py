"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke check."""
from .generators import CONFIGS, Workload, batch, config, custom, sample  # noqa: F401
