"""Seeded synthetic inputs shaped like the paper's trainer workloads.

This package is shared by the float64 oracle tests, the GPU parity tests and
the benchmark.  It only draws random numbers and lays them out; it computes
none of the trainer-step arithmetic (no log-softmax, advantage, loss or
gradient).  See ``gen.synth`` for the recipe.
"""
from .synth import CONFIGS, Config, config, make_batch, Batch  # noqa: F401
