"""Seeded synthetic workloads shared by the oracle tests and the HIP path.

This package holds the configuration table and the seeded input
generators (weights, latents, text context, keep masks).  It contains none
of the method's arithmetic: no block forward, no attention, no
normalisation.  Both sides consume what it produces; neither side's code
lives here.
"""
from .configs import CONFIGS, Config, get_config  # noqa: F401
