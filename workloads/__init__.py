"""Seeded synthetic workloads for the Lethe hot path.

Input synthesis only: this package draws keys, values, queries and score
vectors with the shapes and attention structure of the paper's decoding
workloads (DeepSeek-R1-Distill Llama-8B / Qwen-7B shapes, long reasoning
traces).  It holds none of the method's arithmetic and imports neither the
HIP binding nor the oracle; both sides receive the same arrays from here.
"""
from .configs import CONFIGS, WorkloadConfig  # noqa: F401
