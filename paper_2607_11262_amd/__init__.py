"""MI355X-native batched tile-graph simulation (GTSim backend, arXiv 2607.11262).

``paper_2607_11262_amd.gen`` builds seeded graphs and hardware records;
``paper_2607_11262_amd.api`` wraps the C ABI of libgts.so (loaded lazily on
first use, and never replaced by a CPU path)."""
__all__ = ["gen", "api"]
