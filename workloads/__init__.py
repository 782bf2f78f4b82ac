"""Seeded synthetic inputs for the MosaicKV hot path.

This module holds no arithmetic of the method itself: it draws dense K, V and
q tensors with the shapes and value distributions of the five workloads, and
derives the per-window rotation matrices from the drawn keys and values (the
caller-side SVD step whose result the compression pass takes as an input).
Both the HIP path and the CPU oracle receive exactly these tensors.
"""
from .gen import CONFIGS, WorkloadSpec, make_layer, make_queries, make_appends, spec  # noqa: F401
