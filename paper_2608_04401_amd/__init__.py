"""Elbow-routed MoE layer for MI355X (gfx950): HIP kernels behind a C ABI.

The GPU library (libelbow_moe.so, built from csrc/) is loaded on first use by the binding
module; importing this package loads nothing.
"""
__all__ = ["binding", "synth", "stats"]
