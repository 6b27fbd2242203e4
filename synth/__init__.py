"""Seeded synthetic workloads for the sparse spiking BPTT path.

This package draws input spike tensors, weights and labels. It holds none of
the method's arithmetic (no LIF update, no surrogate, no gradient): both the
CPU oracle's tests and the GPU path's tests and benchmark take their inputs
from here, so the two sides see identical arrays.
"""
from .inputs import CONFIGS, Config, make_inputs, rng_for  # noqa: F401
