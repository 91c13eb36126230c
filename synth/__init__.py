"""Seeded synthetic inputs for the verification path.

This module owns every random *input* the tests and the benchmark feed to both
the CPU oracle and the GPU library: weights, prefix and draft token ids, drafter
confidences, KV-cache contents, synthetic logits and draft distributions.  It
holds none of the method's arithmetic (no forward pass, no acceptance rule, no
length selection), so sharing it does not couple the oracle to the GPU path.
"""
from .configs import MODELS, WORKLOADS, ModelShape, Workload  # noqa: F401
