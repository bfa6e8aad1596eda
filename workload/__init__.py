"""Seeded synthetic inputs shared by the HIP path's tests/bench and the oracle."""
from .synth import CONFIGS, DESCRIPTIONS, Workload, base_chunks, make_workload, random_encoder, random_index  # noqa: F401
