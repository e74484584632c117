"""Seeded synthetic inputs and per-head configs (no arithmetic of the method)."""
from . import config, generate, workloads  # noqa: F401
