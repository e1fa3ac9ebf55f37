"""Seeded synthetic inputs shared by the oracle (oracle/) and the GPU path.

This package holds no arithmetic of the decoding method.
"""
from .configs import BF16, F32, ModelShape, Request, Workload, workload, TINY, TINY_BF16, QWEN3B, QWEN7B, QWEN05B
from . import gen
