"""Seeded synthetic inputs for the FlashLoop per-loop attention step.

This package only draws random inputs (loop-1 states and lazy per-loop deltas, stored as bf16 bit
patterns) and describes the five workload shapes. It holds none of the method's arithmetic: token
scoring, top-k, the residual codec and attention live separately in the GPU library and in the CPU
oracle, which both consume what this package produces.
"""
from .configs import CONFIGS, Workload, get, scaled
from .gen import LoopStates, make_layer

__all__ = ["CONFIGS", "Workload", "get", "scaled", "LoopStates", "make_layer"]
