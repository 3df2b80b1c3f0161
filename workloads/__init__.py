"""Seeded synthetic inputs shared by the oracle and the GPU path (no method arithmetic)."""
from .generator import CONFIGS, Config  # noqa: F401
