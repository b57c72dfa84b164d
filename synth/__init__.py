"""Seeded synthetic inputs shaped like RoleSub's OpenVLA-OFT-7B workloads.

This package only draws and rounds input numbers. It holds none of the
method's arithmetic, so both the float64 oracle and the HIP path can consume
its output without sharing any computation.
"""
from .workloads import *  # noqa: F401,F403
