"""Shared workload structure (specs) and seeded synthetic inputs (synth)."""
from . import specs, synth  # noqa: F401
