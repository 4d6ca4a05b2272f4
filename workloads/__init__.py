"""Seeded synthetic inputs shaped like the paper's GPT-2 / DistilGPT2 workloads.

This package is shared by the fp64 oracle tests, the GPU parity tests and the
benchmark. It only draws and encodes input arrays; it computes nothing of the
DP-SGD method itself (no norms, clip factors, sums or noise).
"""
from .gen import *  # noqa: F401,F403
