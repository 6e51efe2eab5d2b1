"""Seeded synthetic workloads for tree verification.

This package only produces inputs: model shapes, random-init weights, prefix
tokens, prefix KV caches, draft trees and the planting of given token paths
into those trees.  It contains none of the arithmetic of the verification pass
itself, so that both the HIP path and the fp64 oracle can consume its outputs
without sharing any of the computation they are compared on.
"""

from .configs import ModelShape, Workload, WORKLOADS, get_workload  # noqa: F401
