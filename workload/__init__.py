"""Seeded synthetic inputs for the eviction path (shared by the tests and the benchmark; no method code)."""
from .gen import CONFIGS, LLAMA8B, LLAMA8B_LAZY, QWEN, SCOREFREE128K, TINY, Config, Workload, raw_numpy  # noqa: F401
