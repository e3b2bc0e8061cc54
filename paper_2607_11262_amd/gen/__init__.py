"""Seeded synthetic inputs: tile graphs (workloads) and hardware records.

Importing this subpackage never loads the native library."""
from . import graph, hw, rng, workloads  # noqa: F401
from .graph import GraphBuilder, TileGraph, empty_graph, validate  # noqa: F401
